"""Benchmark: GASLoC rounds on one MI355X through libgasloc.so.

One step = one whole round of the hot path on resident synthetic replicas:
H_i masked local AdamW steps, the fused gossip round (pseudo-gradient, outer
Nesterov step, neighbour mix, consensus momentum, consensus-error partials),
its fp64 finalize and the consensus-error readback.  `value` is
replica-param updates per second, n * P / (seconds per round).

Prints ONE JSON line.  Per-kernel durations come from HIP events recorded on
the library's stream around every call inside the timed region.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, AMD specification
METRIC = "replica-param updates/s per gossip round; achieved HBM GB/s vs peak"
DEFAULT_WORKLOAD = "onepeer-exp-n16-p350m"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


CSRC = os.path.join(ROOT, "paper_2606_11081_amd", "csrc")
# the sources each kernel family is compiled and launched from: a committed
# counter summary stays valid while its family's sources are unchanged
KERNEL_FAMILIES = {
    "adamw": ("device_common.h", "internal.h", "adamw.hip", "runtime.cpp"),
    "phase": ("device_common.h", "internal.h", "round_phase.hip", "reductions.hip", "runtime.cpp"),
    "planned": ("device_common.h", "internal.h", "round_planned.hip", "reductions.hip", "runtime.cpp", "plan.cpp"),
}


def kernel_family(kernel, n):
    """Family of the kernel behind a profiled role: AdamW, or the gossip
    kernel the library picks for n workers (the planned kernel beyond 16,
    unless GASLOC_GOSSIP_KERNEL forces one)."""
    if kernel == "k_local_adamw":
        return "adamw"
    forced = os.environ.get("GASLOC_GOSSIP_KERNEL", "")
    if forced in ("phase", "planned"):
        return forced
    return "planned" if n > 16 else "phase"


def kernels_sha(family):
    h = hashlib.sha256()
    for name in KERNEL_FAMILIES[family]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def param_bytes(dtype):
    return 2 if dtype == "bf16" else 4


def adamw_bytes_per_rp(sp):
    # read y (or x), g, m, v; write y, m, v
    return 2 * sp + 20


FORMS = ("eq", "alg1", "dadam", "local_dadam")


def gossip_bytes_per_rp(sp, gamma, stepped=True, with_u=True, form="eq"):
    """Algorithmic bytes of one round per replica-parameter.
    eq:          read x, y (stepped workers), u, zp (gamma); write x, u, zp (gamma)
    alg1:        read x, y (x again for a worker that did not step), u; write x, u
    dadam:       read x, y (stepped workers); write x (no outer momentum)
    local_dadam: read x, y (stepped workers), u; write x, u"""
    b = sp + sp  # x read + x write
    if stepped or form == "alg1":
        b += sp
    if with_u and form != "dadam":
        b += 8
    if gamma != 0.0 and form == "eq":
        b += 8
    return b


def fused_bytes_per_rp(sp, gamma, active, stepped, with_u=True, form="eq"):
    """Fused last local step + round (EQ and ALG1), per worker: an active
    worker also reads g, m, v and writes m, v; its new iterate is never
    stored."""
    b = gossip_bytes_per_rp(sp, gamma, stepped=stepped, with_u=with_u, form=form)
    if active:
        b += 4 + 8 + 8
    return b


def read_traffic(kernel, workload, n):
    """HBM bytes per dispatch from a committed rocprofv3 --pmc summary, or None
    if absent or taken on other sources of the kernel's family."""
    path = os.path.join(ROOT, "profiles", "%s_%s_pmc.md" % (kernel, workload))  # kernel: a kernel or role name
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"traffic_bytes_per_dispatch:\s*([0-9.eE+]+)\s+kernels_sha:\s*([0-9a-f]+)", text)
    if not m or m.group(2) != kernels_sha(kernel_family(kernel, n)):
        return None
    return float(m.group(1))


def _oracle_sample(w, columns, form, seed):
    """An oracle on `columns` columns of the workload, with its x0 and one
    gradient batch (host arrays, made before any timing)."""
    import numpy as np

    import gasloc_inputs as gi
    import oracle

    hp = oracle.OracleHParams(beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY,
                              outer_lr=gi.OUTER_LR, outer_momentum=gi.OUTER_MOMENTUM,
                              nesterov=True, consensus_momentum=w.gamma if form == "eq" else 0.0, form=form)
    o = oracle.Oracle(w.n, columns, hp, topology=w.topology, seed=gi.SEED_TOPOLOGY, degree=w.degree,
                      precision="f32", param_dtype=w.param_dtype)
    rng = np.random.default_rng(seed)
    o.set_params((rng.standard_normal(columns) * 0.02).astype(np.float32))
    g = (rng.standard_normal((w.n, columns)) + gi.worker_means(w.n)[:, None]).astype(np.float32)
    return o, g


def _oracle_round(o, g, H_i):
    """One full round on the oracle: every local step, the round, the
    consensus error."""
    import numpy as np

    import gasloc_inputs as gi

    for h in range(int(H_i.max())):
        o.local_step(g, gi.LOCAL_LR, (H_i > h).astype(np.uint8))
    o.gossip_round(0)
    o.consensus_error()


def cpu_baseline(w, H_i, columns, form="eq"):
    """The oracle as it stands, single-threaded, on `columns` columns of the
    same workload: one full round (all local steps, gossip, consensus error)
    in the same round form."""
    o, g = _oracle_sample(w, columns, form, 0)
    t0 = time.perf_counter()
    _oracle_round(o, g, H_i)
    dt = time.perf_counter() - t0
    return {"value": w.n * columns / dt, "unit": "replica-param updates/s", "cores": 1, "kind": "oracle",
            "sample": "%d of %d columns x %d workers, one round (%d local steps + %s round + CE), "
                      "plain C oracle (fp32 build, -O2, single thread on %s, %d host threads visible): %.2f s"
                      % (columns, w.P, w.n, int(H_i.max()), form.upper() if form == "eq" else form, host_cpu(),
                         os.cpu_count() or 0, dt)}


def host_threads():
    """Host threads this process may use: its CPU affinity, capped by
    OMP_NUM_THREADS when that is set."""
    try:
        t = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        t = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        t = min(t, int(env))
    return max(1, t)


def cpu_baseline_parallel(w, H_i, columns, form="eq", threads=None):
    """The same oracle on all host threads: the sample's columns split into
    one contiguous slice per thread, each slice an oracle of its own (every
    stored value depends only on its own column, so the slices are
    independent), run concurrently.  The oracle's C calls release the GIL."""
    import threading

    threads = threads or host_threads()
    threads = max(1, min(threads, columns))
    bounds = [columns * k // threads for k in range(threads + 1)]
    parts = [_oracle_sample(w, bounds[k + 1] - bounds[k], form, 100 + k) for k in range(threads)]
    start = threading.Barrier(threads + 1)
    errors = []

    def run(k):
        start.wait()
        try:
            _oracle_round(parts[k][0], parts[k][1], H_i)
        except Exception as e:  # reported after the join
            errors.append(e)

    pool = [threading.Thread(target=run, args=(k,)) for k in range(threads)]
    for t in pool:
        t.start()
    start.wait()
    t0 = time.perf_counter()
    for t in pool:
        t.join()
    dt = time.perf_counter() - t0
    if errors:
        raise errors[0]
    return {"value": w.n * columns / dt, "unit": "replica-param updates/s", "cores": threads, "kind": "oracle",
            "sample": "%d of %d columns x %d workers, one round (%d local steps + %s round + CE), "
                      "plain C oracle (fp32 build, -O2) on %d threads of %s, one contiguous column slice "
                      "per thread: %.2f s"
                      % (columns, w.P, w.n, int(H_i.max()), form.upper() if form == "eq" else form, threads,
                         host_cpu(), dt)}


# Oracle work units (one worker-column through one local step or one gossip
# round) in the default CPU sample: about 12 s on one core of the MI355X host,
# 30M columns of the n=16, H=10 workload.
CPU_SAMPLE_UNITS = 30_000_000 * 16 * 11


def cpu_sample_columns(w, H_i):
    """Columns of the oracle's sample: a fixed amount of work whatever the
    workload's worker count and local steps, at most the whole row."""
    per_column = w.n * (float(H_i.mean()) + 1.0)
    return int(max(1, min(w.P, CPU_SAMPLE_UNITS // per_column)))


def host_cpu():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cpu-columns", type=int, default=0,
                    help="columns of the oracle's sample (0: sized to about 12 s of single-core work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-gb", type=float, default=8.0, help="size of the copy probe (GB read)")
    ap.add_argument("--no-fuse", dest="fuse", action="store_false",
                    help="run the last local step and the round as two calls")
    ap.add_argument("--form", choices=FORMS, default="eq",
                    help="round form (non-EQ forms run with gamma = 0; DAdam forms without the fused step)")
    args = ap.parse_args()
    if args.form in ("dadam", "local_dadam"):
        args.fuse = False

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: every replica of the round lives on a single MI355X; "
              "multi-GPU runs (%d requested) are not supported" % max(args.gpus, 1), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import gasloc_inputs as gi
    import paper_2606_11081_amd as g

    w = gi.WORKLOADS[args.workload]
    gamma = w.gamma if args.form == "eq" else 0.0  # the consensus momentum exists in EQ only
    # profiles and the JSON name the workload with its round form when not EQ
    wname = w.name if args.form == "eq" else "%s-%s" % (w.name, args.form)
    H_i = gi.local_steps(w)
    masks = gi.active_masks(H_i)
    sp = param_bytes(w.param_dtype)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("bench: %s  (n=%d P=%d %s H=%s gamma=%g)" % (wname, w.n, w.P, w.param_dtype,
                                                    "U{%d..%d}" % w.hetero_H if w.hetero_H else w.H, gamma))

    lib = g.GASLoC(w.n, w.P, topology=w.topology, seed=gi.SEED_TOPOLOGY, degree=w.degree,
                   param_dtype=w.param_dtype, beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS,
                   weight_decay=gi.WEIGHT_DECAY, outer_lr=gi.OUTER_LR, outer_momentum=gi.OUTER_MOMENTUM,
                   outer_nesterov=True, consensus_momentum=gamma, round_form=args.form)
    lib.set_params(gi.make_x0(w.P, device=dev))
    # one resident gradient batch (stand-in for backpropagated gradients)
    grads = torch.empty((w.n, lib.ld), dtype=torch.float32, device=dev)
    gi.fill_grads(grads, gi.worker_means(w.n), 0)
    stream = lib.stream
    torch.cuda.synchronize()

    def rec(ev, key, extra=None):
        pair = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True), extra)
        ev[key].append(pair)
        pair[0].record(stream)
        return pair

    def one_round(t, ev=None):
        """H_i local steps and the round; the last step is fused into the round."""
        last = len(masks) - 1 if args.fuse else len(masks)
        for h in range(last):
            e = rec(ev, "adam", int(masks[h].sum())) if ev is not None else None
            lib.local_step(grads, gi.LOCAL_LR, masks[h])
            if e:
                e[1].record(stream)
        if args.fuse:
            e = rec(ev, "round", masks[-1]) if ev is not None else None
            lib.local_step_gossip_round(grads, gi.LOCAL_LR, t, masks[-1])
        else:
            e = rec(ev, "round", None) if ev is not None else None
            lib.gossip_round(t)
        if e:
            e[1].record(stream)
        return lib.consensus_error()

    for t in range(args.warmup):
        one_round(t)
    torch.cuda.synchronize()

    ev = {"adam": [], "round": []}
    ces = []
    torch.cuda.synchronize()
    wall = []  # per round: each round ends with the blocking consensus-error readback
    t0 = time.perf_counter()
    for s in range(args.steps):
        r0 = time.perf_counter()
        ces.append(one_round(args.warmup + s, ev))
        wall.append((time.perf_counter() - r0) * 1e3)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = elapsed / args.steps * 1e3

    adam_ms = [a.elapsed_time(b) for a, b, _ in ev["adam"]]
    adam_rp = [k * w.P for _, _, k in ev["adam"]]
    round_ms = [a.elapsed_time(b) for a, b, _ in ev["round"]]
    adam_bytes = adamw_bytes_per_rp(sp)
    if args.fuse:
        act_last = masks[-1]
        # a worker read y in the fused call if it took a local step earlier this round
        stepped_before = np.minimum(H_i, len(masks) - 1) > 0
        round_bytes = sum(fused_bytes_per_rp(sp, gamma, bool(act_last[i]), bool(stepped_before[i]), form=args.form)
                          for i in range(w.n)) * w.P
    else:
        round_bytes = w.n * w.P * gossip_bytes_per_rp(sp, gamma, form=args.form)
    adam_gbps = sum(r * adam_bytes for r in adam_rp) / (sum(adam_ms) * 1e-3) / 1e9 if adam_ms else 0.0
    round_gbps = round_bytes / (np.mean(round_ms) * 1e-3) / 1e9
    adam_total, round_total = sum(adam_ms), sum(round_ms)

    # the standalone gossip kernel (no fused step), timed after the rounds
    g_ms = []
    for s in range(5):
        lib.local_step(grads, gi.LOCAL_LR)
        e = rec({"g": []}, "g")
        lib.gossip_round(args.warmup + args.steps + s)
        e[1].record(stream)
        torch.cuda.synchronize()
        g_ms.append(e[0].elapsed_time(e[1]))
    gossip_bytes = gossip_bytes_per_rp(sp, gamma, form=args.form)
    gossip_ms = float(np.median(g_ms))
    gossip_gbps = w.n * w.P * gossip_bytes / (gossip_ms * 1e-3) / 1e9

    # copy probe: a plain device copy of known size, same run
    copy_elems = int(args.copy_gb * 1e9 / 4)
    src = torch.empty(copy_elems, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(5):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * copy_elems * 4 * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst

    if adam_total >= round_total and adam_ms:
        dom, dom_bytes = "k_local_adamw", float(np.mean([r * adam_bytes for r in adam_rp]))
        dom_ms = float(np.mean(adam_ms))
    else:
        dom = "fused_round" if args.fuse else "gossip_round"
        dom_bytes, dom_ms = round_bytes, float(np.mean(round_ms))
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                "traffic": read_traffic(dom, wname, w.n),
                "algorithmic_bytes_per_launch": int(dom_bytes), "avg_launch_ms": round(dom_ms, 4)}
    out = {
        "metric": METRIC,
        "value": w.n * w.P / (ms_step * 1e-3),
        "unit": "replica-param updates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "round_ms_p10_p50_p90": [round(float(np.percentile(wall, q)), 3) for q in (10, 50, 90)],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        # the arithmetic of every kernel is fp32 (reductions fp64), whatever the
        # parameters are stored in; the storage type is config.param_dtype
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": wname, "n": w.n, "P": w.P, "topology": w.topology, "round_form": args.form,
                   "local_steps": "U{%d..%d}" % w.hetero_H if w.hetero_H else w.H,
                   "gamma": gamma, "param_dtype": w.param_dtype, "state_dtype": "f32",
                   "last_local_step_fused": bool(args.fuse)},
        "roofline": roofline,
        "gossip_round": {"role": "gossip round alone (library-chosen gossip kernel + CSR/plan upload + finalize)",
                         "rp_updates_per_s": w.n * w.P / (gossip_ms * 1e-3),
                         "ms": round(gossip_ms, 4), "GBps": round(gossip_gbps, 1),
                         "frac_of_peak": round(gossip_gbps / PEAK_HBM_GBPS, 4), "bytes_per_rp": gossip_bytes,
                         "traffic": read_traffic("gossip_round", wname, w.n)},
        "round_kernel": {"role": "fused_round" if args.fuse else "gossip_round",
                         "ms": round(float(np.mean(round_ms)), 4), "GBps": round(round_gbps, 1),
                         "frac_of_peak": round(round_gbps / PEAK_HBM_GBPS, 4),
                         "bytes_per_launch": int(round_bytes)},
        "local_adamw": {"ms_per_launch": round(float(np.mean(adam_ms)), 4) if adam_ms else None,
                        "GBps": round(adam_gbps, 1), "frac_of_peak": round(adam_gbps / PEAK_HBM_GBPS, 4),
                        "bytes_per_rp": adam_bytes, "launches_per_round": len(adam_ms) // max(args.steps, 1)},
        "copy_probe_GBps": round(copy_gbps, 1),
        "consensus_error_last": ces[-1],
    }
    lib.close()
    del grads
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        columns = min(args.cpu_columns, w.P) if args.cpu_columns > 0 else cpu_sample_columns(w, H_i)
        log("bench: timing the oracle on %d columns" % columns)
        out["cpu_baseline"] = cpu_baseline(w, H_i, columns, args.form)
        log("bench: timing the oracle on %d host threads" % host_threads())
        out["cpu_baseline_all_threads"] = cpu_baseline_parallel(w, H_i, columns, args.form)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

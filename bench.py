"""Benchmark: GASLoC rounds on one MI355X through libgasloc.so.

One step = one whole round of the hot path on resident synthetic replicas:
H_i masked local AdamW steps, the fused gossip round (pseudo-gradient, outer
Nesterov step, neighbour mix, consensus momentum, consensus-error partials),
its fp64 finalize and the consensus-error readback.  `value` is
replica-param updates per second, n * P / (seconds per round), on the
headline workload (n=16, P=350M by default).

After the headline workload, the other workloads of the benchmark run one
after another in the same process (each one's buffers freed before the
next), each with its own rounds, standalone gossip round, streaming-probe
mixes and oracle baselines, reported under "workloads".

Gradients: one resident [n, ld] fp32 batch per workload, drawn once before
timing (seed 2); every local step reads it from HBM, so each step moves the
bytes of a fresh gradient batch (the stand-in for backpropagation, which is
not part of the round).

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
INFINITY_CACHE_BYTES = 256e6  # MI355X last-level cache
METRIC = "replica-param updates/s per gossip round; achieved HBM GB/s vs peak"
DEFAULT_WORKLOAD = "onepeer-exp-n16-p350m"
# the benchmark's five configurations by name
CONFIGS = {"C1": "ring-n4-p1m", "C2": "exp-n8-p124m", "C3": "onepeer-exp-n16-p350m",
           "C4": "regular3-n32-p150m-bf16", "C5": "matching-n64-p50m-hetH"}


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


def pmc_profile(kernel, workload):
    return os.path.join("profiles", "%s_%s_pmc.md" % (kernel, workload))  # kernel: a kernel or role name


def read_traffic(kernel, workload, n):
    """HBM bytes per dispatch from a committed rocprofv3 --pmc summary, or None
    if absent or taken on other sources of the kernel's family."""
    path = os.path.join(ROOT, pmc_profile(kernel, workload))
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"traffic_bytes_per_dispatch:\s*([0-9.eE+]+)\s+kernels_sha:\s*([0-9a-f]+)", text)
    if not m or m.group(2) != kernels_sha(kernel_family(kernel, n)):
        return None
    return float(m.group(1))


def traffic_source(kernel, workload, n):
    """Where a reported traffic figure comes from (None when there is none):
    not measured in this run, but read from a committed counter summary whose
    kernel sources are the ones built now."""
    if read_traffic(kernel, workload, n) is None:
        return None
    return {"profile": pmc_profile(kernel, workload), "kernels_sha": kernels_sha(kernel_family(kernel, n)),
            "method": "rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE, per dispatch, each scaled by the same "
                      "counter of the streaming probe's copy of known size (in that profile's process)"}


def _oracle_sample(w, columns, form, seed, topo_seed=0):
    """An oracle on `columns` columns of the workload, with its x0 and one
    gradient batch (host arrays, made before any timing); topo_seed is added
    to the schedule's seed, as the benchmark's --seed does."""
    import numpy as np

    import gasloc_inputs as gi
    import oracle

    hp = oracle.OracleHParams(beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY,
                              outer_lr=gi.OUTER_LR, outer_momentum=gi.OUTER_MOMENTUM,
                              nesterov=True, consensus_momentum=w.gamma if form == "eq" else 0.0, form=form)
    o = oracle.Oracle(w.n, columns, hp, topology=w.topology, seed=gi.SEED_TOPOLOGY + topo_seed, degree=w.degree,
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


def cpu_baseline(w, H_i, columns, form="eq", topo_seed=0):
    """The oracle as it stands, single-threaded, on `columns` columns of the
    same workload: one full round (all local steps, gossip, consensus error)
    in the same round form."""
    o, g = _oracle_sample(w, columns, form, 0, topo_seed)
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


def cpu_baseline_parallel(w, H_i, columns, form="eq", threads=None, topo_seed=0):
    """The same oracle on all host threads: the sample's columns split into
    one contiguous slice per thread, each slice an oracle of its own (every
    stored value depends only on its own column, so the slices are
    independent), run concurrently.  The oracle's C calls release the GIL."""
    import threading

    threads = threads or host_threads()
    threads = max(1, min(threads, columns))
    bounds = [columns * k // threads for k in range(threads + 1)]
    parts = [_oracle_sample(w, bounds[k + 1] - bounds[k], form, 100 + k, topo_seed) for k in range(threads)]
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


# Streaming-probe mixes (include/gasloc_probe.h): (fp32 reads, bf16 reads,
# fp32 writes, bf16 writes), destinations in place of the first sources.
PROBE_MIXES = {
    "read": (4, 0, 0, 0), "write": (0, 0, 3, 0), "copy": (1, 0, 1, 0),
    "r16w12_f32": (4, 0, 3, 0),          # AdamW fp32; EQ round fp32, gamma != 0
    "r12w8_f32": (3, 0, 2, 0),           # EQ round fp32, gamma = 0
    "adamw_bf16": (3, 1, 2, 1), "round_bf16": (2, 2, 2, 1),
    "fused_f32": (7, 0, 5, 0), "fused_f32_g0": (6, 0, 4, 0), "fused_bf16": (5, 2, 4, 1),
}
PROBE_COUNT = 1 << 28  # elements per stream: 1 GiB per fp32 stream


def probe_mix_bytes(mix, count=PROBE_COUNT):
    r32, r16, w32, w16 = mix
    return count * (4 * (r32 + w32) + 2 * (r16 + w16))


def kernel_mixes(param_dtype, gamma):
    """The probe mix whose bytes per element match each kernel (EQ form)."""
    if param_dtype == "bf16":
        return {"adamw": "adamw_bf16", "round": "round_bf16", "fused": "fused_bf16"}
    if gamma != 0.0:
        return {"adamw": "r16w12_f32", "round": "r16w12_f32", "fused": "fused_f32"}
    return {"adamw": "r16w12_f32", "round": "r12w8_f32", "fused": "fused_f32_g0"}


PROBE_THREADS = (256, 64)  # workgroup sizes timed per mix; the faster one is the probe's figure


def stream_probe(names, dev, reps=5):
    """GB/s of the hand-written streaming kernel on each named mix, in this
    process: for each workgroup size in PROBE_THREADS one warm-up and `reps`
    timed launches (median); the mix's figure is the faster size's."""
    import numpy as np
    import torch

    import paper_2606_11081_amd as g

    need32 = max(max(PROBE_MIXES[k][0], PROBE_MIXES[k][2]) for k in names)
    need16 = max(max(PROBE_MIXES[k][1], PROBE_MIXES[k][3]) for k in names)
    f32 = [torch.ones(PROBE_COUNT, dtype=torch.float32, device=dev) for _ in range(need32)]
    b16 = [torch.ones(PROBE_COUNT, dtype=torch.bfloat16, device=dev) for _ in range(need16)]
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    out = {}
    for name in names:
        r32, r16, w32, w16 = mix = PROBE_MIXES[name]
        src, dst = f32[:r32] + b16[:r16], f32[:w32] + b16[:w16]
        by_threads = {}
        for threads in PROBE_THREADS:
            ms = []
            for k in range(reps + 1):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                g.gasloc.gasloc_stream_probe(r32, r16, w32, w16, src, dst, PROBE_COUNT, sink, stream, threads)
                b.record(stream)
                torch.cuda.synchronize()
                if k:
                    ms.append(a.elapsed_time(b))
            by_threads[threads] = float(np.median(ms))
        best = min(by_threads, key=by_threads.get)
        t = by_threads[best]
        nbytes = probe_mix_bytes(mix)
        out[name] = {"mix": list(mix), "bytes": nbytes, "ms": round(t, 4),
                     "GBps": round(nbytes / (t * 1e-3) / 1e9, 1), "threads": best,
                     "GBps_by_threads": {str(k): round(nbytes / (v * 1e-3) / 1e9, 1) for k, v in by_threads.items()}}
    del f32, b16, sink
    torch.cuda.empty_cache()
    return out


def run_workload(w, form, steps, warmup, fuse, dev, log_prefix="bench", seed=0):
    """Whole rounds of one workload on the GPU: `warmup` untimed rounds, then
    `steps` timed rounds, then 5 standalone gossip rounds.  `seed` shifts the
    schedule's seed and picks the gradient batch.  Returns the measurements;
    frees the workload's buffers before returning."""
    import numpy as np
    import torch

    import gasloc_inputs as gi
    import paper_2606_11081_amd as g

    gamma = w.gamma if form == "eq" else 0.0  # the consensus momentum exists in EQ only
    H_i = gi.local_steps(w)
    masks = gi.active_masks(H_i)
    sp = param_bytes(w.param_dtype)
    log("%s: %s%s  (n=%d P=%d %s H=%s gamma=%g)" % (log_prefix, w.name, "" if form == "eq" else " " + form, w.n,
                                                   w.P, w.param_dtype,
                                                   "U{%d..%d}" % w.hetero_H if w.hetero_H else w.H, gamma))
    lib = g.GASLoC(w.n, w.P, topology=w.topology, seed=gi.SEED_TOPOLOGY + seed, degree=w.degree,
                   param_dtype=w.param_dtype, beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS,
                   weight_decay=gi.WEIGHT_DECAY, outer_lr=gi.OUTER_LR, outer_momentum=gi.OUTER_MOMENTUM,
                   outer_nesterov=True, consensus_momentum=gamma, round_form=form)
    lib.set_params(gi.make_x0(w.P, device=dev))
    grads = torch.empty((w.n, lib.ld), dtype=torch.float32, device=dev)
    gi.fill_grads(grads, gi.worker_means(w.n), seed)
    stream = lib.stream
    torch.cuda.synchronize()

    def rec(ev, key, extra=None):
        pair = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True), extra)
        ev[key].append(pair)
        pair[0].record(stream)
        return pair

    def one_round(t, ev=None):
        """H_i local steps and the round; the last step is fused into the round."""
        last = len(masks) - 1 if fuse else len(masks)
        for h in range(last):
            e = rec(ev, "adam", int(masks[h].sum())) if ev is not None else None
            lib.local_step(grads, gi.LOCAL_LR, masks[h])
            if e:
                e[1].record(stream)
        if fuse:
            e = rec(ev, "round", masks[-1]) if ev is not None else None
            lib.local_step_gossip_round(grads, gi.LOCAL_LR, t, masks[-1])
        else:
            e = rec(ev, "round", None) if ev is not None else None
            lib.gossip_round(t)
        if e:
            e[1].record(stream)
        return lib.consensus_error()

    for t in range(warmup):
        one_round(t)
    torch.cuda.synchronize()

    ev = {"adam": [], "round": []}
    ces = []
    wall = []  # per round: each round ends with the blocking consensus-error readback
    t0 = time.perf_counter()
    for s in range(steps):
        r0 = time.perf_counter()
        ces.append(one_round(warmup + s, ev))
        wall.append((time.perf_counter() - r0) * 1e3)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) / steps * 1e3

    adam_ms = [a.elapsed_time(b) for a, b, _ in ev["adam"]]
    adam_rp = [k * w.P for _, _, k in ev["adam"]]
    round_ms = [a.elapsed_time(b) for a, b, _ in ev["round"]]
    adam_bytes = adamw_bytes_per_rp(sp)
    if fuse:
        act_last = masks[-1]
        # a worker read y in the fused call if it took a local step earlier this round
        stepped_before = np.minimum(H_i, len(masks) - 1) > 0
        round_bytes = sum(fused_bytes_per_rp(sp, gamma, bool(act_last[i]), bool(stepped_before[i]), form=form)
                          for i in range(w.n)) * w.P
    else:
        round_bytes = w.n * w.P * gossip_bytes_per_rp(sp, gamma, form=form)
    adam_gbps = sum(r * adam_bytes for r in adam_rp) / (sum(adam_ms) * 1e-3) / 1e9 if adam_ms else 0.0
    round_gbps = round_bytes / (np.mean(round_ms) * 1e-3) / 1e9

    # the standalone gossip kernel (no fused step), timed after the rounds
    g_ms = []
    for s in range(5):
        lib.local_step(grads, gi.LOCAL_LR)
        e = rec({"g": []}, "g")
        lib.gossip_round(warmup + steps + s)
        e[1].record(stream)
        torch.cuda.synchronize()
        g_ms.append(e[0].elapsed_time(e[1]))
    gossip_bytes = gossip_bytes_per_rp(sp, gamma, form=form)
    gossip_ms = float(np.median(g_ms))
    gossip_gbps = w.n * w.P * gossip_bytes / (gossip_ms * 1e-3) / 1e9
    lib.close()
    del lib, grads
    torch.cuda.empty_cache()
    return {
        "H_i": H_i, "gamma": gamma, "ms_per_step": ms_step, "wall": wall, "ces": ces,
        "adam_ms": adam_ms, "adam_rp": adam_rp, "adam_bytes": adam_bytes, "adam_gbps": adam_gbps,
        "round_ms": round_ms, "round_bytes": round_bytes, "round_gbps": round_gbps,
        "gossip_ms": gossip_ms, "gossip_bytes": gossip_bytes, "gossip_gbps": gossip_gbps,
    }


def build_record():
    """The loaded library's build record and whether its sources are this tree's."""
    import paper_2606_11081_amd as g
    from paper_2606_11081_amd import build as lib_build

    info = g.gasloc.gasloc_build_info()
    sha = lib_build.sources_sha()
    return {"library": info, "tree_sources_sha": sha, "matches_tree": info.startswith("sources %s;" % sha)}


def frac(x, ref):
    return round(x / ref, 4) if ref else None


def kernel_records(w, form, fuse, r, probe):
    """The per-kernel records of one workload: time, GB/s, fraction of peak and
    of the matching streaming-probe mix."""
    import numpy as np

    mixes = kernel_mixes(w.param_dtype, r["gamma"]) if form == "eq" else {}
    pg = lambda role: probe.get(mixes.get(role), {}).get("GBps")  # noqa: E731
    round_role = "fused" if fuse else "round"
    return {
        "gossip_round": {"role": "gossip round alone (library-chosen gossip kernel + CSR/plan upload + finalize)",
                         "rp_updates_per_s": w.n * w.P / (r["gossip_ms"] * 1e-3),
                         "ms": round(r["gossip_ms"], 4), "GBps": round(r["gossip_gbps"], 1),
                         "frac_of_peak": frac(r["gossip_gbps"], PEAK_HBM_GBPS), "bytes_per_rp": r["gossip_bytes"],
                         "probe_mix": mixes.get("round"), "frac_of_probe": frac(r["gossip_gbps"], pg("round"))},
        "round_kernel": {"role": "fused_round" if fuse else "gossip_round",
                         "ms": round(float(np.mean(r["round_ms"])), 4), "GBps": round(r["round_gbps"], 1),
                         "frac_of_peak": frac(r["round_gbps"], PEAK_HBM_GBPS),
                         "bytes_per_launch": int(r["round_bytes"]), "probe_mix": mixes.get(round_role),
                         "frac_of_probe": frac(r["round_gbps"], pg(round_role))},
        "local_adamw": {"ms_per_launch": round(float(np.mean(r["adam_ms"])), 4) if r["adam_ms"] else None,
                        "GBps": round(r["adam_gbps"], 1), "frac_of_peak": frac(r["adam_gbps"], PEAK_HBM_GBPS),
                        "bytes_per_rp": r["adam_bytes"],
                        "launches_per_round": len(r["adam_ms"]) // max(len(r["wall"]), 1),
                        "probe_mix": mixes.get("adamw") if r["adam_ms"] else None,
                        "frac_of_probe": frac(r["adam_gbps"], pg("adamw")) if r["adam_ms"] else None},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--config", choices=sorted(CONFIGS), help="the workload by its configuration name (C1..C5)")
    ap.add_argument("--rounds", type=int, default=None, help="the same as --steps")
    ap.add_argument("--seed", type=int, default=0,
                    help="added to the schedule's seed; also selects the gradient batch (default 0)")
    ap.add_argument("--workloads", default="auto",
                    help="other workloads timed after the headline one: 'auto' (all the others when the headline is "
                         "the default workload in the EQ form, else none), 'none', or a comma-separated list")
    ap.add_argument("--workload-steps", type=int, default=5, help="timed rounds of each other workload")
    ap.add_argument("--cpu-columns", type=int, default=0,
                    help="columns of the oracle's sample (0: sized to about 12 s of single-core work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probe", dest="probe", action="store_false", help="skip the streaming-probe mixes")
    ap.add_argument("--no-fuse", dest="fuse", action="store_false",
                    help="run the last local step and the round as two calls")
    ap.add_argument("--form", choices=FORMS, default="eq",
                    help="round form (non-EQ forms run with gamma = 0; DAdam forms without the fused step)")
    args = ap.parse_args()
    if args.form in ("dadam", "local_dadam"):
        args.fuse = False
    if args.config:
        args.workload = CONFIGS[args.config]
    if args.rounds is not None:
        args.steps = args.rounds

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: every replica of the round lives on a single MI355X; "
              "multi-GPU runs (%d requested) are not supported" % max(args.gpus, 1), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import gasloc_inputs as gi

    w = gi.WORKLOADS[args.workload]
    # profiles and the JSON name the workload with its round form when not EQ
    wname = w.name if args.form == "eq" else "%s-%s" % (w.name, args.form)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    r = run_workload(w, args.form, args.steps, args.warmup, args.fuse, dev, seed=args.seed)
    gamma, H_i = r["gamma"], r["H_i"]
    probe = {}
    if args.probe:
        names = ["read", "write", "copy"] + sorted(set(kernel_mixes(w.param_dtype, gamma).values()))
        log("bench: streaming probe, mixes %s" % ", ".join(names))
        probe = stream_probe(names, dev)
    recs = kernel_records(w, args.form, args.fuse, r, probe)

    adam_total, round_total = sum(r["adam_ms"]), sum(r["round_ms"])
    if adam_total >= round_total and r["adam_ms"]:
        dom = "k_local_adamw"
        dom_bytes = float(np.mean([k * r["adam_bytes"] for k in r["adam_rp"]]))
        dom_ms = float(np.mean(r["adam_ms"]))
    else:
        dom = "fused_round" if args.fuse else "gossip_round"
        dom_bytes, dom_ms = r["round_bytes"], float(np.mean(r["round_ms"]))
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                "traffic": read_traffic(dom, wname, w.n), "traffic_source": traffic_source(dom, wname, w.n),
                "algorithmic_bytes_per_launch": int(dom_bytes), "avg_launch_ms": round(dom_ms, 4)}
    recs["gossip_round"]["traffic"] = read_traffic("gossip_round", wname, w.n)
    recs["gossip_round"]["traffic_source"] = traffic_source("gossip_round", wname, w.n)
    out = {
        "metric": METRIC,
        "value": w.n * w.P / (r["ms_per_step"] * 1e-3),
        "unit": "replica-param updates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 3),
        "round_ms_p10_p50_p90": [round(float(np.percentile(r["wall"], q)), 3) for q in (10, 50, 90)],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        # the arithmetic of every kernel is fp32 (reductions fp64), whatever the
        # parameters are stored in; the storage type is config.param_dtype
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": wname, "n": w.n, "P": w.P, "topology": w.topology, "round_form": args.form,
                   "local_steps": "U{%d..%d}" % w.hetero_H if w.hetero_H else w.H,
                   "gamma": gamma, "param_dtype": w.param_dtype, "state_dtype": "f32",
                   "last_local_step_fused": bool(args.fuse),
                   "seed": args.seed,
                   "gradients": "one resident [n, ld] fp32 batch, drawn once (seed %d), read by every local step"
                                % (gi.SEED_GRAD_BASE + args.seed)},
        "roofline": roofline,
    }
    out.update(recs)
    out["stream_probe"] = probe
    out["build"] = build_record()
    out["consensus_error_last"] = r["ces"][-1]
    if not args.no_cpu_baseline:
        columns = min(args.cpu_columns, w.P) if args.cpu_columns > 0 else cpu_sample_columns(w, H_i)
        log("bench: timing the oracle on %d columns" % columns)
        out["cpu_baseline"] = cpu_baseline(w, H_i, columns, args.form, args.seed)
        log("bench: timing the oracle on %d host threads" % host_threads())
        out["cpu_baseline_all_threads"] = cpu_baseline_parallel(w, H_i, columns, args.form, topo_seed=args.seed)

    if args.workloads == "auto":
        others = [k for k in gi.WORKLOADS if k != w.name] if (w.name == DEFAULT_WORKLOAD and args.form == "eq") else []
    elif args.workloads == "none":
        others = []
    else:
        others = [k for k in args.workloads.split(",") if k]
    if others:
        out["workloads"] = {}
    for name in others:
        wo = gi.WORKLOADS[name]
        ro = run_workload(wo, "eq", args.workload_steps, 2, True, dev, log_prefix="bench (workloads)", seed=args.seed)
        po = {}
        # a workload whose round fits the 256 MB Infinity Cache is not an HBM
        # stream: no probe fraction for it
        if args.probe and wo.n * wo.P * ro["gossip_bytes"] > INFINITY_CACHE_BYTES:
            po = stream_probe(sorted(set(kernel_mixes(wo.param_dtype, ro["gamma"]).values())), dev)
        rec = {"n": wo.n, "P": wo.P, "topology": wo.topology, "param_dtype": wo.param_dtype, "gamma": ro["gamma"],
               "local_steps": "U{%d..%d}" % wo.hetero_H if wo.hetero_H else wo.H,
               "steps": args.workload_steps, "warmup": 2, "ms_per_step": round(ro["ms_per_step"], 3),
               "value": wo.n * wo.P / (ro["ms_per_step"] * 1e-3)}
        rec.update(kernel_records(wo, "eq", True, ro, po))
        rec["stream_probe"] = po
        if not args.no_cpu_baseline:
            Hw = ro["H_i"]
            columns = max(1, cpu_sample_columns(wo, Hw) // 3)  # about 4 s of single-core work
            log("bench (workloads): timing the oracle on %d columns of %s" % (columns, name))
            rec["cpu_baseline"] = cpu_baseline(wo, Hw, columns, topo_seed=args.seed)
            rec["cpu_baseline_all_threads"] = cpu_baseline_parallel(wo, Hw, columns, topo_seed=args.seed)
        out["workloads"][name] = rec
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

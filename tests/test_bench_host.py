"""Host-side logic of bench.py, on the CPU: the algorithmic byte counts that
price every kernel against the HBM roofline, the one-GPU guard, the parser of
the committed PMC summaries and the oracle-timing leg."""
import importlib.util
import os
import re
import subprocess
import sys

import numpy as np
import pytest

import gasloc_inputs as gi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def moved(reads, writes):
    return sum(reads.values()) + sum(writes.values())


@pytest.mark.parametrize("sp", [4, 2])
def test_adamw_bytes_are_the_buffers_it_streams(bench, sp):
    # one local step (Sec. 2, the inner AdamW update): params, grads and both
    # moments are read; params and moments written back; grads stay fp32
    assert bench.adamw_bytes_per_rp(sp) == moved({"y": sp, "g": 4, "m": 4, "v": 4},
                                                  {"y": sp, "m": 4, "v": 4})


@pytest.mark.parametrize("sp", [4, 2])
@pytest.mark.parametrize("gamma", [0.0, 0.1])
@pytest.mark.parametrize("stepped", [True, False])
@pytest.mark.parametrize("with_u", [True, False])
def test_gossip_bytes_are_the_buffers_it_streams(bench, sp, gamma, stepped, with_u):
    # Eq. 1 / Eq. 2: x, the local iterate y (only if the worker stepped),
    # the outer momentum u (mu != 0) and the previous z (gamma != 0) are read;
    # x, u and the stored z are written
    reads = {"x": sp}
    writes = {"x": sp}
    if stepped:
        reads["y"] = sp
    if with_u:
        reads["u"] = writes["u"] = 4
    if gamma:
        reads["zp"] = writes["zp"] = 4
    assert bench.gossip_bytes_per_rp(sp, gamma, stepped=stepped, with_u=with_u) == moved(reads, writes)


@pytest.mark.parametrize("sp", [4, 2])
def test_fused_bytes_add_the_last_step_without_its_iterate(bench, sp):
    # the fused last step reads g, m, v and writes m, v; its new iterate only
    # feeds the pseudo-gradient, so it is neither stored nor re-read
    for gamma in (0.0, 0.1):
        for stepped in (True, False):
            base = bench.gossip_bytes_per_rp(sp, gamma, stepped=stepped)
            assert bench.fused_bytes_per_rp(sp, gamma, True, stepped) == base + 4 + 8 + 8
            assert bench.fused_bytes_per_rp(sp, gamma, False, stepped) == base


@pytest.mark.parametrize("name, gossip_gb, adamw_gb", [
    ("exp-n8-p124m", 27.776, 27.776),
    ("onepeer-exp-n16-p350m", 156.8, 156.8),
    ("regular3-n32-p150m-bf16", 105.6, 115.2),
    ("matching-n64-p50m-hetH", 64.0, 89.6),
])
def test_bytes_per_round_of_the_workloads(bench, name, gossip_gb, adamw_gb):
    w = gi.WORKLOADS[name]
    sp = bench.param_bytes(w.param_dtype)
    assert w.n * w.P * bench.gossip_bytes_per_rp(sp, w.gamma) == pytest.approx(gossip_gb * 1e9, rel=1e-12)
    assert w.n * w.P * bench.adamw_bytes_per_rp(sp) == pytest.approx(adamw_gb * 1e9, rel=1e-12)


def test_default_workload_is_the_n16_p350m_configuration(bench):
    w = gi.WORKLOADS[bench.DEFAULT_WORKLOAD]
    assert (w.n, w.P, w.topology, w.param_dtype, w.H, w.gamma) == (16, 350_000_000, "one_peer_exp", "f32", 10, 0.1)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and "2 requested" in r.stderr
    assert r.stdout == ""


def test_committed_pmc_summaries_parse(bench):
    names = [f for f in os.listdir(os.path.join(ROOT, "profiles")) if f.endswith("_pmc.md")]
    assert names
    for f in names:
        text = open(os.path.join(ROOT, "profiles", f)).read()
        m = re.search(r"traffic_bytes_per_dispatch:\s*([0-9.eE+]+)\s+kernels_sha:\s*([0-9a-f]{16})\b", text)
        assert m, f
        assert float(m.group(1)) > 0
        assert "rocprofv3 --pmc FETCH_SIZE" in text and "rocprofv3 --pmc WRITE_SIZE" in text, f


def test_traffic_is_withheld_for_another_kernel_source(bench, tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "k_local_adamw_w_pmc.md").write_text("traffic_bytes_per_dispatch: 1.5e+11 kernels_sha: 0123456789abcdef\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernels_sha", lambda family: "0123456789abcdef")
    assert bench.read_traffic("k_local_adamw", "w", 16) == 1.5e11
    monkeypatch.setattr(bench, "kernels_sha", lambda family: "fedcba9876543210")
    assert bench.read_traffic("k_local_adamw", "w", 16) is None
    assert bench.read_traffic("missing", "w", 16) is None


def test_kernel_families_hash_their_own_sources(bench, tmp_path, monkeypatch):
    import shutil

    monkeypatch.delenv("GASLOC_GOSSIP_KERNEL", raising=False)
    assert bench.kernel_family("k_local_adamw", 64) == "adamw"
    assert bench.kernel_family("gossip_round", 16) == "phase"
    assert bench.kernel_family("fused_round", 17) == "planned"
    monkeypatch.setenv("GASLOC_GOSSIP_KERNEL", "planned")
    assert bench.kernel_family("gossip_round", 8) == "planned"
    names = sorted({f for files in bench.KERNEL_FAMILIES.values() for f in files})
    for f in names:
        shutil.copy(os.path.join(bench.CSRC, f), tmp_path / f)
    monkeypatch.setattr(bench, "CSRC", str(tmp_path))
    before = {fam: bench.kernels_sha(fam) for fam in bench.KERNEL_FAMILIES}
    with open(tmp_path / "round_planned.hip", "a") as fh:
        fh.write("// edited\n")
    after = {fam: bench.kernels_sha(fam) for fam in bench.KERNEL_FAMILIES}
    assert after["planned"] != before["planned"]
    assert after["adamw"] == before["adamw"] and after["phase"] == before["phase"]


def test_cpu_baseline_times_the_oracle_on_a_sample(bench):
    w = gi.WORKLOADS[bench.DEFAULT_WORKLOAD]
    out = bench.cpu_baseline(w, gi.local_steps(w), 2000)
    assert out["kind"] == "oracle" and out["cores"] == 1
    assert out["unit"] == "replica-param updates/s" and out["value"] > 0
    assert "2000 of 350000000 columns x 16 workers, one round (10 local steps + EQ round + CE)" in out["sample"]
    alt = bench.cpu_baseline(w, gi.local_steps(w), 500, "local_dadam")
    assert "local_dadam round" in alt["sample"] and alt["value"] > 0


def test_cpu_baseline_on_all_threads_splits_the_sample(bench):
    w = gi.WORKLOADS[bench.DEFAULT_WORKLOAD]
    out = bench.cpu_baseline_parallel(w, gi.local_steps(w), 2001, threads=3)
    assert out["kind"] == "oracle" and out["cores"] == 3
    assert out["unit"] == "replica-param updates/s" and out["value"] > 0
    assert "2001 of 350000000 columns x 16 workers" in out["sample"] and "on 3 threads" in out["sample"]
    assert bench.cpu_baseline_parallel(w, gi.local_steps(w), 2, threads=8)["cores"] == 2
    assert bench.host_threads() >= 1


def test_oracle_column_slices_are_independent(bench):
    """The all-threads baseline runs the oracle on column slices; a round on
    each slice gives exactly the columns of a round on the whole row."""
    import oracle

    w = gi.WORKLOADS["regular3-n32-p150m-bf16"]
    H_i = np.array([1 + (i % 3) for i in range(w.n)])
    P = 3001
    full, g = bench._oracle_sample(w, P, "eq", 7)
    x0 = full.x[0].copy()
    bench._oracle_round(full, g, H_i)
    bench._oracle_round(full, g, H_i)  # the second round applies the consensus momentum
    cuts = [0, 1000, 1001, P]
    for a, b in zip(cuts[:-1], cuts[1:]):
        part, _ = bench._oracle_sample(w, b - a, "eq", 7)
        part.set_params(x0[a:b])
        gs = np.ascontiguousarray(g[:, a:b])
        bench._oracle_round(part, gs, H_i)
        bench._oracle_round(part, gs, H_i)
        for name in ("x", "y", "m", "v", "u", "zp"):
            assert np.array_equal(getattr(part, name), getattr(full, name)[:, a:b]), name
    assert isinstance(full, oracle.Oracle)


def test_cpu_sample_is_a_fixed_amount_of_work(bench):
    sizes = {}
    for name, w in gi.WORKLOADS.items():
        H_i = gi.local_steps(w)
        cols = bench.cpu_sample_columns(w, H_i)
        assert 1 <= cols <= w.P
        sizes[name] = cols
        if cols < w.P:  # work = columns x workers x (local steps + the round)
            work = cols * w.n * (H_i.mean() + 1)
            assert abs(work - bench.CPU_SAMPLE_UNITS) <= w.n * (H_i.mean() + 1)
    assert sizes["onepeer-exp-n16-p350m"] == 30_000_000
    assert sizes["ring-n4-p1m"] == 1_048_576  # the whole row


@pytest.mark.parametrize("sp", [4, 2])
@pytest.mark.parametrize("stepped", [True, False])
def test_round_form_bytes_are_the_buffers_they_stream(bench, sp, stepped):
    # Algorithm 1: the slot holds y_j (x_j for a worker that did not step),
    # each row reads x_i and u_i and writes x_i and u_i
    assert bench.gossip_bytes_per_rp(sp, 0.0, stepped=stepped, form="alg1") == moved(
        {"x": sp, "y or x": sp, "u": 4}, {"x": sp, "u": 4})
    # DAdam (App. C): x_j in the slot, y_i for a worker that stepped, x written
    dadam_reads = {"x": sp, "y": sp} if stepped else {"x": sp}
    assert bench.gossip_bytes_per_rp(sp, 0.0, stepped=stepped, form="dadam") == moved(dadam_reads, {"x": sp})
    # Local-DAdam: as DAdam plus the outer momentum u read and written
    assert bench.gossip_bytes_per_rp(sp, 0.0, stepped=stepped, form="local_dadam") == moved(
        dict(dadam_reads, u=4), {"x": sp, "u": 4})
    # consensus momentum exists in EQ only
    for form in ("alg1", "dadam", "local_dadam"):
        assert bench.gossip_bytes_per_rp(sp, 0.1, stepped=stepped, form=form) == \
            bench.gossip_bytes_per_rp(sp, 0.0, stepped=stepped, form=form)
    # the fused last step adds g, m, v read and m, v written to an active worker
    assert bench.fused_bytes_per_rp(sp, 0.0, True, stepped, form="alg1") == \
        bench.gossip_bytes_per_rp(sp, 0.0, stepped=stepped, form="alg1") + 20


def test_scripts_use_no_unbound_names():
    """Every name the benchmark and the entry points read is bound somewhere
    in the file or is a builtin (main() itself needs a GPU to run)."""
    import ast
    import builtins

    for script in ("bench.py", "__graft_entry__.py"):
        tree = ast.parse(open(os.path.join(ROOT, script)).read())
        bound = set(dir(builtins)) | {"__file__", "__name__"}
        for node in ast.walk(tree):
            if isinstance(node, (ast.FunctionDef, ast.AsyncFunctionDef, ast.ClassDef)):
                bound.add(node.name)
            elif isinstance(node, ast.arg):
                bound.add(node.arg)
            elif isinstance(node, ast.Name) and isinstance(node.ctx, (ast.Store, ast.Del)):
                bound.add(node.id)
            elif isinstance(node, (ast.Import, ast.ImportFrom)):
                bound.update((a.asname or a.name).split(".")[0] for a in node.names)
            elif isinstance(node, ast.ExceptHandler) and node.name:
                bound.add(node.name)
        unbound = sorted({n.id for n in ast.walk(tree) if isinstance(n, ast.Name) and isinstance(n.ctx, ast.Load)}
                         - bound)
        assert not unbound, (script, unbound)


def test_configurations_name_the_workloads(bench):
    assert set(bench.CONFIGS.values()) == set(gi.WORKLOADS)
    assert bench.CONFIGS["C3"] == bench.DEFAULT_WORKLOAD
    for name, wl in bench.CONFIGS.items():
        w = gi.WORKLOADS[wl]
        assert (name, w.n) in {("C1", 4), ("C2", 8), ("C3", 16), ("C4", 32), ("C5", 64)}


def test_probe_mixes_match_the_kernel_bytes(bench):
    # every kernel's probe mix moves that kernel's bytes per element (EQ form)
    for wl in gi.WORKLOADS.values():
        sp = bench.param_bytes(wl.param_dtype)
        mixes = bench.kernel_mixes(wl.param_dtype, wl.gamma)
        per = lambda m: bench.probe_mix_bytes(bench.PROBE_MIXES[m], 1)  # noqa: E731
        assert per(mixes["adamw"]) == bench.adamw_bytes_per_rp(sp)
        assert per(mixes["round"]) == bench.gossip_bytes_per_rp(sp, wl.gamma)
        assert per(mixes["fused"]) == bench.fused_bytes_per_rp(sp, wl.gamma, True, True)

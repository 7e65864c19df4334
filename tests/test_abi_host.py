"""Host-side tests of libgasloc.so (no GPU): exported symbols, bit-exact
round schedules against the oracle, CSR validation and argument checks that
fail before any device call."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2606_11081_amd as g

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KINDS = ["ring", "complete", "exponential", "one_peer_exp", "one_peer", "two_peer", "random_regular"]


def header_functions():
    """Every function declared by a header under include/."""
    names = set()
    inc = os.path.join(ROOT, "include")
    for h in sorted(os.listdir(inc)):
        if h.endswith(".h"):
            text = re.sub(r"/\*.*?\*/", "", open(os.path.join(inc, h)).read(), flags=re.S)
            names.update(re.findall(r"\b(gasloc_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    lib = g.library()
    names = header_functions()
    assert len(names) >= 13
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(g.gasloc._SIGNATURES)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 8, 16, 32, 33, 64])
def test_schedule_bit_exact_with_oracle(kind, n):
    if kind == "random_regular" and (n <= 3 or (3 * n) % 2):
        pytest.skip("3-regular graph needs n > 3 and 3n even")
    topo = g.make_topology_struct(kind, seed=3, degree=3)
    rounds = 200 if n <= 16 else 40
    for t in range(rounds):
        rp, col, val = g.gasloc_make_topology(topo, n, t)
        orp, ocol, oval = oracle.topology_csr(kind, n, 3, t, 3)
        assert np.array_equal(rp, orp), (kind, n, t)
        assert np.array_equal(col, ocol), (kind, n, t)
        assert np.array_equal(val.view(np.uint32), oval.view(np.uint32)), (kind, n, t)


@pytest.mark.parametrize("kind,n,degree", [("random_regular", 10, 4), ("random_regular", 12, 5),
                                           ("random_regular", 9, 0), ("two_peer", 64, 3)])
def test_schedule_bit_exact_other_degrees_and_seeds(kind, n, degree):
    for seed in (0, 1, 2 ** 63 + 5):
        topo = g.make_topology_struct(kind, seed=seed, degree=degree)
        for t in (0, 1, 17, 2 ** 40 + 3):
            got = g.gasloc_make_topology(topo, n, t)
            exp = oracle.topology_csr(kind, n, seed, t, degree)
            for a, b in zip(got, exp):
                assert np.array_equal(a, b)


def test_schedule_long_horizon_matching_n64():
    topo = g.make_topology_struct("one_peer", seed=3)
    for t in range(0, 1000, 7):
        got = g.gasloc_make_topology(topo, 64, t)
        exp = oracle.topology_csr("one_peer", 64, 3, t)
        for a, b in zip(got, exp):
            assert np.array_equal(a, b)


def test_make_topology_rejects_bad_arguments():
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_make_topology(g.make_topology_struct("random_regular", degree=3), 5, 0)  # 3*5 odd
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_make_topology(g.make_topology_struct("random_regular", degree=4), 4, 0)  # degree >= n
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_make_topology(g.make_topology_struct(99), 4, 0)
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_make_topology(g.make_topology_struct("explicit"), 4, 0)
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_make_topology(g.make_topology_struct("ring"), 65, 0)
    # capacity too small
    lib = g.library()
    rp = np.zeros(9, np.int32)
    col = np.zeros(4, np.int32)
    val = np.zeros(4, np.float32)
    nnz = ctypes.c_int32()
    topo = g.make_topology_struct("complete")
    st = lib.gasloc_make_topology(ctypes.byref(topo), 8, 0, rp.ctypes.data, col.ctypes.data,
                                  val.ctypes.data, 4, ctypes.byref(nnz))
    assert st == g.GASLOC_EINVAL
    assert "capacity" in g.gasloc_last_error()


def _ring4():
    return oracle.topology_csr("ring", 4, 0, 0)


def test_validate_csr_accepts_generated_graphs():
    for kind in KINDS:
        n = 8
        W = oracle.topology_csr(kind, n, 3, 5, 3)
        g.gasloc_validate_csr(W, n)


@pytest.mark.parametrize("case", ["n_mismatch", "unsorted", "duplicate", "out_of_range", "negative_col",
                                  "row_sum", "nan", "rowptr_start", "rowptr_nonmono", "rowptr_end"])
def test_validate_csr_rejects(case):
    rp, col, val = (a.copy() for a in _ring4())
    n = 4
    if case == "n_mismatch":
        n = 5
    elif case == "unsorted":
        col[0], col[1] = col[1], col[0]
    elif case == "duplicate":
        col[1] = col[0]
    elif case == "out_of_range":
        col[2] = 4
    elif case == "negative_col":
        col[0] = -1
    elif case == "row_sum":
        val[0] = 0.5
    elif case == "nan":
        val[3] = np.nan
    elif case == "rowptr_start":
        rp[0] = 1
    elif case == "rowptr_nonmono":
        rp[2] = rp[1] - 1
    elif case == "rowptr_end":
        rp[-1] -= 1
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_validate_csr((rp, col, val), n)


def _csr_is_valid(rp, col, val, n):
    """The documented acceptance rule of a caller's CSR (include/gasloc.h), restated."""
    if len(rp) - 1 != n:
        return False
    nnz = len(col)
    if nnz < n or nnz > n * n or rp[0] != 0 or rp[n] != nnz:
        return False
    for i in range(n):
        b, e = int(rp[i]), int(rp[i + 1])
        if e < b or b < 0 or e > nnz:
            return False
        total = 0.0
        for k in range(b, e):
            c = int(col[k])
            if c < 0 or c >= n or (k > b and c <= int(col[k - 1])) or not np.isfinite(val[k]):
                return False
            total += float(val[k])  # fp64 sum of the fp32 weights, in CSR order
        if abs(total - 1.0) > 1e-6:
            return False
    return True


def test_validate_csr_agrees_with_its_rule_on_random_graphs():
    # random row-stochastic CSRs, half of them with one random defect (or a
    # weight nudged across the 1e-6 row-sum tolerance): the library accepts
    # exactly those the documented rule accepts
    rng = np.random.default_rng(2024)
    decisions = {True: 0, False: 0}
    for case in range(1500):
        n = int(rng.integers(1, 13))
        rows_c, rows_v = [], []
        for i in range(n):
            k = int(rng.integers(1, n + 1))
            c = np.sort(rng.choice(n, size=k, replace=False)).astype(np.int32)
            w = rng.random(k) + 0.05
            w = (w / w.sum()).astype(np.float32)
            w[-1] = np.float32(1.0 - float(np.sum(w[:-1], dtype=np.float64)))  # row sum close to 1 in fp64
            rows_c.append(c)
            rows_v.append(w)
        rp = np.zeros(n + 1, np.int32)
        rp[1:] = np.cumsum([len(c) for c in rows_c])
        col = np.concatenate(rows_c).astype(np.int32)
        val = np.concatenate(rows_v).astype(np.float32)
        nv = n
        if rng.random() < 0.5:
            kind = int(rng.integers(0, 9))
            k = int(rng.integers(0, len(col)))
            if kind == 0 and len(col) > 1:
                col[k], col[(k + 1) % len(col)] = col[(k + 1) % len(col)], col[k]
            elif kind == 1:
                col[k] = n + int(rng.integers(0, 3))
            elif kind == 2:
                col[k] = -1 - int(rng.integers(0, 3))
            elif kind == 3:
                val[k] = np.float32(val[k] + rng.choice([5e-7, -5e-7, 2e-6, -2e-6, 0.25]))
            elif kind == 4:
                val[k] = rng.choice([np.nan, np.inf, -np.inf])
            elif kind == 5 and n > 1:
                j = int(rng.integers(1, n))
                rp[j] = rp[j] + int(rng.choice([-2, -1, 1, 2]))
            elif kind == 6:
                rp[-1] += int(rng.choice([-1, 1]))
            elif kind == 7:
                nv = n + 1 if n < 64 else n - 1
            elif kind == 8 and len(col) > 1:
                col[k] = col[k - 1] if k > 0 else col[1]
        want = _csr_is_valid(rp, col, val, nv)
        decisions[want] += 1
        if want:
            g.gasloc_validate_csr((rp, col, val), nv)
        else:
            with pytest.raises(g.GaslocError, match="EINVAL"):
                g.gasloc_validate_csr((rp, col, val), nv)
    assert decisions[True] > 300 and decisions[False] > 300, decisions


def test_row_sum_tolerance_is_1e6_in_fp64():
    rp = np.array([0, 1], np.int32)
    col = np.array([0], np.int32)
    g.gasloc_validate_csr((rp, col, np.array([1.0 + 9e-7], np.float32)), 1)
    with pytest.raises(g.GaslocError):
        g.gasloc_validate_csr((rp, col, np.array([1.0 + 2e-6], np.float32)), 1)


# --- gasloc_init argument checks that fail before any HIP call -------------

FAKE = 1 << 20  # a 16-byte aligned address that is never dereferenced


def _init(n=4, P=1024, ld=None, hp=None, topo=None, x=FAKE, y=FAKE, m=FAKE, v=FAKE, u=FAKE, zp=FAKE):
    hp = hp or g.make_hparams()
    topo = topo or g.make_topology_struct("ring")
    return g.gasloc_init(n, P, topo, hp, x, y, m, v, u, zp, ld if ld is not None else P)


@pytest.mark.parametrize("kwargs,msg", [
    (dict(n=0), "n=0"),
    (dict(n=65), "n=65"),
    (dict(P=0), "P=0"),
    (dict(P=2 ** 31), "P="),
    (dict(P=1024, ld=1000), "ld must be"),
    (dict(P=1023, ld=1023), "multiple of 16"),
    (dict(x=None), "must not be NULL"),
    (dict(m=FAKE + 4), "16-byte aligned"),
    (dict(u=None), "u may be NULL"),
    (dict(zp=None), "zp may be NULL"),
    (dict(hp=g.make_hparams(beta1=1.0)), "beta1"),
    (dict(hp=g.make_hparams(beta2=-0.1)), "beta2"),
    (dict(hp=g.make_hparams(eps=0.0)), "eps"),
    (dict(hp=g.make_hparams(outer_lr=0.0)), "outer_lr"),
    (dict(hp=g.make_hparams(outer_momentum=1.0)), "outer_momentum"),
    (dict(hp=g.make_hparams(consensus_momentum=1.5)), "consensus_momentum"),
    (dict(hp=g.make_hparams(weight_decay=float("nan"))), "weight_decay"),
    (dict(topo=g.make_topology_struct(42)), "topology kind"),
    (dict(n=5, topo=g.make_topology_struct("random_regular", degree=3)), "topology"),
])
def test_init_rejects_bad_arguments(kwargs, msg):
    with pytest.raises(g.GaslocError, match="EINVAL") as ei:
        _init(**kwargs)
    assert msg in str(ei.value)


def test_null_context_is_rejected():
    lib = g.library()
    assert lib.gasloc_local_step(None, FAKE, 4, None, 0.1) == g.GASLOC_EINVAL
    assert lib.gasloc_gossip_round(None, None, 0) == g.GASLOC_EINVAL
    out = ctypes.c_double()
    assert lib.gasloc_consensus_error(None, ctypes.byref(out)) == g.GASLOC_EINVAL
    lib.gasloc_destroy(None)  # ignored


@pytest.mark.parametrize("total", [1, 9, 10, 100, 1000, 2569, 100_000])
@pytest.mark.parametrize("fracs", [(0.1, 0.01, 0.0), (0.05, 0.1, 0.1), (0.0, 0.01, 0.0), (1.0, 0.01, 0.0)])
def test_lr_schedule_bit_exact_with_oracle(total, fracs):
    f32 = lambda v: float(np.float32(v))  # noqa: E731
    peak = f32(4e-3)
    w, s, f = (f32(v) for v in fracs)
    steps = sorted(set(list(range(0, min(total, 300) + 1)) + [total // 2, total - 1, total, total + 3, -1]))
    for step in steps:
        got = g.gasloc_lr_schedule(peak, step, total, w, s, f)
        exp = oracle.lr_schedule(peak, step, total, w, s, f)
        assert np.float32(got).view(np.uint32) == np.float32(exp).view(np.uint32), (step, got, exp)


def _adjacency(n, p, seed):
    rng = np.random.default_rng(seed)
    A = np.triu((rng.random((n, n)) < p).astype(np.uint8), 1)
    return (A + A.T).astype(np.uint8)


@pytest.mark.parametrize("kind", ["one_peer", "two_peer"])
@pytest.mark.parametrize("n,p", [(8, 0.5), (16, 0.3), (64, 0.1), (5, 1.0)])
def test_restricted_schedule_bit_exact_with_oracle(kind, n, p):
    A = _adjacency(n, p, n)
    topo = g.make_topology_struct(kind, seed=3, admissible=A)
    for t in range(60):
        got = g.gasloc_make_topology(topo, n, t)
        exp = oracle.topology_csr(kind, n, 3, t, admissible=A)
        for a, b in zip(got, exp):
            assert np.array_equal(a.view(np.uint32) if a.dtype == np.float32 else a,
                                  b.view(np.uint32) if b.dtype == np.float32 else b)


def test_admissible_only_for_random_peer_kinds():
    with pytest.raises(g.GaslocError, match="admissible"):
        g.gasloc_make_topology(g.make_topology_struct("ring", admissible=np.ones((4, 4))), 4, 0)
    asym = np.zeros((4, 4), np.uint8)
    asym[0, 1] = 1
    with pytest.raises(g.GaslocError, match="symmetric"):
        g.gasloc_init(4, 1024, g.make_topology_struct("one_peer", admissible=asym), g.make_hparams(), FAKE, FAKE,
                      FAKE, FAKE, FAKE, FAKE, 1024)


@pytest.mark.parametrize("kind", KINDS)
def test_skip_exchanges_bit_exact_with_oracle(kind):
    n = 12
    rng = np.random.default_rng(11)
    for t in range(20):
        W = oracle.topology_csr(kind, n, 3, t, 3)
        alive = (rng.random(n) > 0.25).astype(np.uint8)
        link = (rng.random((n, n)) > 0.2).astype(np.uint8)
        for al, lk in ((alive, None), (None, link), (alive, link), (None, None)):
            got = g.gasloc_skip_exchanges(W, n, al, lk)
            exp = oracle.skip_exchanges(W, n, al, lk)
            assert np.array_equal(got[0], exp[0]) and np.array_equal(got[1], exp[1])
            assert np.array_equal(got[2].view(np.uint32), exp[2].view(np.uint32))


def test_skip_exchanges_on_a_csr_without_diagonal():
    # a row without its own entry gets one only if weight is moved to it
    rp = np.array([0, 2, 4, 6], np.int32)
    col = np.array([1, 2, 0, 2, 0, 1], np.int32)
    val = np.full(6, 0.5, np.float32)
    alive = np.array([1, 1, 0], np.uint8)
    got = g.gasloc_skip_exchanges((rp, col, val), 3, alive)
    exp = oracle.skip_exchanges((rp, col, val), 3, alive)
    for a, b in zip(got, exp):
        assert np.array_equal(a, b)
    assert list(got[0]) == [0, 2, 4, 5]


@pytest.mark.parametrize("mix,count,threads,msg", [
    ((1, 1, 1, 1), 1024, 256, "unsupported mix"),
    ((4, 0, 3, 1), 1024, 256, "unsupported mix"),
    ((-1, 0, 1, 0), 1024, 256, "unsupported mix"),
    ((1, 0, 1, 0), 0, 256, "count outside"),
    ((1, 0, 1, 0), 1 << 31, 256, "count outside"),
    ((1, 0, 1, 0), 1024, 0, "threads must be"),
    ((1, 0, 1, 0), 1024, 32, "threads must be"),
    ((1, 0, 1, 0), 1024, 512, "threads must be"),
])
def test_stream_probe_rejects_bad_arguments(mix, count, threads, msg):
    # every case fails before any device work
    lib = g.library()
    st = lib.gasloc_stream_probe(*mix, None, None, count, threads, None, None)
    assert st == g.gasloc.GASLOC_EINVAL
    assert msg in g.gasloc.gasloc_last_error(None)


def test_stream_probe_rejects_null_and_misaligned_streams():
    lib = g.library()
    src = (ctypes.c_void_p * 1)(None)
    dst = (ctypes.c_void_p * 1)(0x1000)
    assert lib.gasloc_stream_probe(1, 0, 1, 0, src, dst, 64, 256, None, None) == g.gasloc.GASLOC_EINVAL
    assert "source" in g.gasloc.gasloc_last_error(None)
    src = (ctypes.c_void_p * 1)(0x1008)
    assert lib.gasloc_stream_probe(1, 0, 1, 0, src, dst, 64, 256, None, None) == g.gasloc.GASLOC_EINVAL
    assert "misaligned" in g.gasloc.gasloc_last_error(None)
    src = (ctypes.c_void_p * 4)(0x1000, 0x2000, 0x3000, 0x4000)
    assert lib.gasloc_stream_probe(4, 0, 0, 0, src, None, 64, 256, None, None) == g.gasloc.GASLOC_EINVAL
    assert "sink" in g.gasloc.gasloc_last_error(None)


@pytest.mark.parametrize("args,msg", [
    ((None, 0, 4, 1024, 0, 1024), "x must be"),
    ((0x1008, 0, 4, 1024, 0, 1024), "x must be"),
    ((0x1000, 2, 4, 1024, 0, 1024), "param_dtype"),
    ((0x1000, 0, 0, 1024, 0, 1024), "n outside"),
    ((0x1000, 0, 65, 1024, 0, 1024), "n outside"),
    ((0x1000, 0, 4, 1026, 0, 1024), "multiple of 16"),
    ((0x1000, 1, 4, 1028, 0, 1024), "multiple of 16"),
    ((0x1000, 0, 4, 1024, 5, 4), "p_begin"),
    ((0x1000, 0, 4, 1024, 0, 1028), "p_begin"),
    ((0x1000, 0, 1, 1 << 31, 0, 1 << 31), "p_begin"),
    # the scratch bound: 2^16 workgroups of 8 x 256 groups of 4 fp32 / 8 bf16 columns
    ((0x1000, 0, 1, 1 << 30, 0, (1 << 29) + 1), "at most 536870912 columns"),
    ((0x1000, 1, 1, 1 << 30, 4, (1 << 30) + 1), "p_begin"),
    ((0x1000, 1, 1, (1 << 31) - 8, 0, (1 << 30) + 8), "at most 1073741824 columns"),
])
def test_noalloc_consensus_error_rejects_bad_arguments(args, msg):
    # every case fails on the host, before the scratch lookup or any launch
    out = 0x2000
    st = g.library().gasloc_consensus_error_cols_noalloc(*args, out, None)
    assert st == g.gasloc.GASLOC_EINVAL
    assert msg in g.gasloc.gasloc_last_error(None)


def test_noalloc_consensus_error_rejects_bad_output():
    lib = g.library()
    assert lib.gasloc_consensus_error_cols_noalloc(0x1000, 0, 4, 1024, 0, 1024, None, None) == g.gasloc.GASLOC_EINVAL
    assert lib.gasloc_consensus_error_cols_noalloc(0x1000, 0, 4, 1024, 0, 1024, 0x2004, None) == g.gasloc.GASLOC_EINVAL
    assert "out must be" in g.gasloc.gasloc_last_error(None)


def test_library_was_built_from_this_tree():
    # gasloc_build_info carries the hash of the sources the library was
    # compiled from; a library left over from other sources fails here
    from paper_2606_11081_amd import build as lib_build

    info = g.gasloc.gasloc_build_info()
    assert info == lib_build.build_info(), (info, lib_build.build_info())
    assert "gfx950" in info and "packed-fp32" in info

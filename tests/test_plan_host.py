"""Host tests of the visit planner of the slot-reusing gossip kernel
(paper_2606_11081_amd/csrc/plan.cpp), no GPU.

The planner reorders a round's independent work: each worker's slot value is
computed once into an LDS slot before its first reader and the slot is
reused after its last reader; with reuse allowed, a row whose CSR entries
equal those of the row summed just before it takes that sum.  Here every
plan is replayed numerically the way the kernel consumes it (slots as an
array, rows summed in the order the plan lists their entries, a reusing row
taking the last sum) and must reproduce sum_k W_ik z_k in CSR order bit for
bit, with every row emitted once; tampered plans must be rejected by the
planner's own verifier.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_11081_amd", "csrc")
CXX = "/opt/rocm/llvm/bin/clang++"


@pytest.fixture(scope="module")
def shim(tmp_path_factory):
    if not os.path.exists(CXX):
        pytest.skip("no host C++ compiler at " + CXX)
    out = str(tmp_path_factory.mktemp("plan") / "libplan_shim.so")
    cmd = [CXX, "-O1", "-std=c++17", "-shared", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, os.path.join(ROOT, "tests", "plan_shim.cpp"),
           os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "topology.cpp"), "-o", out]
    subprocess.run(cmd, check=True, capture_output=True)
    lib = ctypes.CDLL(out)
    P = ctypes.POINTER
    lib.plan_shim_plan.argtypes = [ctypes.c_int, P(ctypes.c_int32), P(ctypes.c_int32), P(ctypes.c_float),
                                   ctypes.c_int, P(ctypes.c_int32), ctypes.c_int, P(ctypes.c_int), ctypes.c_char_p,
                                   ctypes.c_int]
    lib.plan_shim_verify.argtypes = [ctypes.c_int, P(ctypes.c_int32), P(ctypes.c_int32), P(ctypes.c_float),
                                     ctypes.c_int, P(ctypes.c_int32), ctypes.c_int, ctypes.c_int]
    lib.plan_shim_words_max.restype = ctypes.c_int64
    lib.plan_shim_scale.argtypes = [P(ctypes.c_int32), ctypes.c_int, ctypes.c_int32]
    return lib


def _ptr(a, t):
    return a.ctypes.data_as(ctypes.POINTER(t))


def plan(lib, n, rp, col, val, reuse=False):
    rp, col, val = (np.ascontiguousarray(rp, np.int32), np.ascontiguousarray(col, np.int32),
                    np.ascontiguousarray(val, np.float32))
    cap = int(lib.plan_shim_words_max(n))
    out = np.zeros(cap, np.int32)
    slots = ctypes.c_int(0)
    err = ctypes.create_string_buffer(256)
    k = lib.plan_shim_plan(n, _ptr(rp, ctypes.c_int32), _ptr(col, ctypes.c_int32), _ptr(val, ctypes.c_float),
                           int(reuse), _ptr(out, ctypes.c_int32), cap, ctypes.byref(slots), err, 256)
    assert k > 0, err.value.decode()
    return out[:k].copy(), slots.value


def verify(lib, n, rp, col, val, ops, slots, reuse=False):
    rp, col, val = (np.ascontiguousarray(rp, np.int32), np.ascontiguousarray(col, np.int32),
                    np.ascontiguousarray(val, np.float32))
    ops = np.ascontiguousarray(ops, np.int32)
    return lib.plan_shim_verify(n, _ptr(rp, ctypes.c_int32), _ptr(col, ctypes.c_int32), _ptr(val, ctypes.c_float),
                                int(reuse), _ptr(ops, ctypes.c_int32), len(ops), slots) == 1


def replay(lib, n, rp, col, val, ops, slots, z, reuse=False):
    """Runs the plan on slot values z (float32 [n]) as the kernel does and
    returns the row sums and the rows that took the previous sum; asserts
    the plan's structural limits on the way."""
    batch, rows_max, reuse_code = lib.plan_shim_batch(), lib.plan_shim_rows(), lib.plan_shim_reuse_code()
    reused = []
    last = None  # (row, sum) of the last row that summed its entries
    S = int(ops[0])
    assert 1 <= S <= 2 * n
    lds = np.full(slots, np.nan, np.float32)
    holder = np.full(slots, -1)
    out = np.full(n, np.nan, np.float32)
    done = np.zeros(n, bool)
    computed = np.zeros(n, bool)
    pc = 1 + S
    for s in range(S):
        assert ops[1 + s] == pc
        npre, nrows = int(ops[pc]), int(ops[pc + 1])
        pc += 2
        assert 0 <= npre <= batch and 0 <= nrows <= rows_max and npre + nrows > 0
        for _ in range(npre):
            j, sl = int(ops[pc]), int(ops[pc + 1])
            pc += 2
            assert not computed[j]
            computed[j] = True
            lds[sl], holder[sl] = z[j], j
        ids = [int(r) for r in ops[pc:pc + nrows]]
        pc += nrows
        for r in ids:
            nent, own = int(ops[pc]), int(ops[pc + 1])
            pc += 2
            assert holder[own] == r, "own slot of row %d" % r
            assert not done[r]
            done[r] = True
            if nent == reuse_code:
                assert reuse and last is not None
                lr = last[0]
                assert np.array_equal(col[rp[r]:rp[r + 1]], col[rp[lr]:rp[lr + 1]])
                assert np.array_equal(np.asarray(val[rp[r]:rp[r + 1]], np.float32).view(np.uint32),
                                      np.asarray(val[rp[lr]:rp[lr + 1]], np.float32).view(np.uint32))
                out[r] = last[1]
                reused.append(r)
                continue
            assert nent == rp[r + 1] - rp[r]
            acc = np.float32(0.0)
            for k in range(nent):
                sl, bits = int(ops[pc]), int(ops[pc + 1])
                pc += 2
                w = np.array([bits], np.int32).view(np.float32)[0]
                assert holder[sl] == col[rp[r] + k] and w == val[rp[r] + k]
                acc = np.float32(acc + np.float32(w * lds[sl]))
            out[r] = acc
            last = (r, acc)
    assert pc == len(ops) and done.all()
    return out, reused


def dense_order_sums(n, rp, col, val, z):
    out = np.zeros(n, np.float32)
    for i in range(n):
        acc = np.float32(0.0)
        for k in range(rp[i], rp[i + 1]):
            acc = np.float32(acc + np.float32(np.float32(val[k]) * z[col[k]]))
        out[i] = acc
    return out


def check(lib, n, rp, col, val, seed=0, reuse=False):
    ops, slots = plan(lib, n, rp, col, val, reuse)
    assert 1 <= slots <= n
    assert len(ops) <= lib.plan_shim_words_max(n)
    z = np.random.default_rng(seed).standard_normal(n).astype(np.float32)
    got, reused = replay(lib, n, rp, col, val, ops, slots, z, reuse)
    assert np.array_equal(got.view(np.uint32), dense_order_sums(n, rp, col, val, z).view(np.uint32))
    assert verify(lib, n, rp, col, val, ops, slots, reuse)
    if reused:
        assert not verify(lib, n, rp, col, val, ops, slots, False)
    return ops, slots, sorted(reused)


KINDS = ["ring", "complete", "exponential", "one_peer_exp", "one_peer", "two_peer", "random_regular"]


def rows_with_an_equal_earlier_row(n, rp, col, val):
    seen, count = set(), 0
    for i in range(n):
        key = (tuple(col[rp[i]:rp[i + 1]]), np.asarray(val[rp[i]:rp[i + 1]], np.float32).tobytes())
        count += key in seen
        seen.add(key)
    return count


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("n", [1, 2, 5, 16, 17, 32, 33, 64])
def test_generated_graphs_replay_exactly(shim, kind, n, reuse):
    if kind == "random_regular" and (n <= 3 or (3 * n) % 2):
        pytest.skip("3-regular graph needs n > 3 and 3n even")
    for t in range(6):
        rp, col, val = oracle.topology_csr(kind, n, 3, t, 3)
        ops, slots, reused = check(shim, n, rp, col, val, seed=t, reuse=reuse)
        if kind in ("one_peer", "ring") and n >= 16:
            assert slots <= 8, (kind, n, slots)  # sparse graphs reuse slots
        # the generated graphs carry every self-loop, so every row equal to an
        # earlier one can take its sum: all but one row of the complete graph,
        # one row of each 1-Peer pair
        assert len(reused) == (rows_with_an_equal_earlier_row(n, rp, col, val) if reuse else 0)
        if reuse and kind == "complete":
            assert len(reused) == n - 1
        if reuse and kind == "one_peer":
            assert len(reused) == n // 2


@pytest.mark.parametrize("reuse", [False, True])
def test_random_csrs_with_dense_rows_and_missing_diagonals(shim, reuse):
    rng = np.random.default_rng(11)
    for trial in range(300):
        n = int(rng.integers(1, 65))
        dens = float(rng.random())
        rows = []
        for i in range(n):
            cs = np.nonzero(rng.random(n) < dens)[0]
            if cs.size == 0:
                cs = np.array([int(rng.integers(n))])
            rows.append(cs)
        rp = np.concatenate([[0], np.cumsum([len(c) for c in rows])]).astype(np.int32)
        col = np.concatenate(rows).astype(np.int32)
        val = np.concatenate([np.full(len(c), 1.0 / len(c)) for c in rows]).astype(np.float32)
        check(shim, n, rp, col, val, seed=trial, reuse=reuse)


def test_equal_rows_without_their_own_column_sum_their_entries(shim):
    # four equal rows reading workers 2 and 3: rows 0 and 1 cannot take an
    # earlier row's sum (their own values are not among those columns, so
    # they may not be live), rows 2 and 3 follow whichever row sums first
    rp = np.array([0, 2, 4, 6, 8], np.int32)
    col = np.array([2, 3, 2, 3, 2, 3, 2, 3], np.int32)
    val = np.full(8, 0.5, np.float32)
    ops, slots, reused = check(shim, 4, rp, col, val, reuse=True)
    assert reused == [2, 3]


@pytest.mark.parametrize("kind, reuse", [("two_peer", False), ("one_peer", True), ("complete", True)])
def test_tampered_plans_are_rejected(shim, kind, reuse):
    n = 12
    rp, col, val = oracle.topology_csr(kind, n, 5, 2)
    ops, slots, reused = check(shim, n, rp, col, val, reuse=reuse)
    assert bool(reused) == reuse
    rejected = 0
    for k in range(len(ops)):
        for d in (-1, 1, 1000):
            bad = ops.copy()
            bad[k] += d
            rejected += not verify(shim, n, rp, col, val, bad, slots, reuse)
    assert rejected == 3 * len(ops)
    assert not verify(shim, n, rp, col, val, ops[:-1], slots, reuse)
    assert not verify(shim, n, rp, col, val, ops, slots - 1, reuse)


def test_reused_sum_needs_equal_entries(shim):
    n = 6
    rp, col, val = oracle.topology_csr("complete", n, 0, 0)
    ops, slots, reused = check(shim, n, rp, col, val, reuse=True)
    assert len(reused) == n - 1
    # the same plan against a CSR whose later rows differ in one weight bit
    for r in range(n):
        other = np.asarray(val, np.float32).copy()
        k = rp[r] + r % (rp[r + 1] - rp[r])
        other[k] = np.nextafter(other[k], np.float32(1.0))
        assert not verify(shim, n, rp, col, other, ops, slots, True), r



def slot_word_positions(ops):
    """Indices of the words of a plan that name a slot, read off the encoding
    independently of the library: each new value's slot, each row's own slot
    and each entry's slot."""
    reuse_code = -1
    pos = []
    S = int(ops[0])
    for s in range(S):
        pc = int(ops[1 + s])
        npre, nrows = int(ops[pc]), int(ops[pc + 1])
        pc += 2
        for _ in range(npre):
            pos.append(pc + 1)
            pc += 2
        pc += nrows
        for _ in range(nrows):
            nent = int(ops[pc])
            pos.append(pc + 1)
            pc += 2
            if nent == reuse_code:
                continue
            for _ in range(nent):
                pos.append(pc)
                pc += 2
    return pos


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("unit", [1, 4 * 64, 4 * 256 * 2, 4 * 256 * 4])
def test_scaled_plans_hold_byte_offsets_of_the_same_slots(shim, kind, unit):
    # the kernel reads slot words as byte offsets (slot * threads * V * 4):
    # scaling multiplies exactly those words, and dividing them back gives a
    # plan that replays bit for bit like the original
    assert shim.plan_shim_reuse_code() == -1
    n = 32
    for t in range(3):
        rp, col, val = oracle.topology_csr(kind, n, 3, t, 3)
        for reuse in (False, True):
            ops, slots = plan(shim, n, rp, col, val, reuse)
            scaled = np.ascontiguousarray(ops.copy(), np.int32)
            assert shim.plan_shim_scale(_ptr(scaled, ctypes.c_int32), len(scaled), unit) == 1
            pos = slot_word_positions(ops)
            other = np.setdiff1d(np.arange(len(ops)), pos)
            assert np.array_equal(scaled[other], ops[other])
            assert np.array_equal(scaled[pos], ops[pos] * unit)
            back = scaled.copy()
            back[pos] //= unit
            z = np.random.default_rng(t).standard_normal(n).astype(np.float32)
            got, _ = replay(shim, n, rp, col, val, back, slots, z, reuse)
            assert np.array_equal(got.view(np.uint32), dense_order_sums(n, rp, col, val, z).view(np.uint32))


def test_scaling_rejects_offsets_beyond_range(shim):
    rp, col, val = oracle.topology_csr("complete", 64, 0, 0)
    ops, slots = plan(shim, 64, rp, col, val, False)
    assert slots == 64
    big = np.ascontiguousarray(ops.copy(), np.int32)
    assert shim.plan_shim_scale(_ptr(big, ctypes.c_int32), len(big), 1 << 25) == 0

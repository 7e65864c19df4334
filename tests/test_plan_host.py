"""Host tests of the visit planner of the slot-reusing gossip kernel
(paper_2606_11081_amd/csrc/plan.cpp), no GPU.

The planner reorders a round's independent work: each worker's slot value is
computed once into an LDS slot before its first reader and the slot is
reused after its last reader.  Here every plan is replayed numerically the
way the kernel consumes it (slots as an array, rows summed in the order the
plan lists their entries) and must reproduce sum_k W_ik z_k in CSR order
bit for bit, with every row emitted once; tampered plans must be rejected
by the planner's own verifier.
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
                                   P(ctypes.c_int32), ctypes.c_int, P(ctypes.c_int), ctypes.c_char_p, ctypes.c_int]
    lib.plan_shim_verify.argtypes = [ctypes.c_int, P(ctypes.c_int32), P(ctypes.c_int32), P(ctypes.c_float),
                                     P(ctypes.c_int32), ctypes.c_int, ctypes.c_int]
    lib.plan_shim_words_max.restype = ctypes.c_int64
    return lib


def _ptr(a, t):
    return a.ctypes.data_as(ctypes.POINTER(t))


def plan(lib, n, rp, col, val):
    rp, col, val = (np.ascontiguousarray(rp, np.int32), np.ascontiguousarray(col, np.int32),
                    np.ascontiguousarray(val, np.float32))
    cap = int(lib.plan_shim_words_max(n))
    out = np.zeros(cap, np.int32)
    slots = ctypes.c_int(0)
    err = ctypes.create_string_buffer(256)
    k = lib.plan_shim_plan(n, _ptr(rp, ctypes.c_int32), _ptr(col, ctypes.c_int32), _ptr(val, ctypes.c_float),
                           _ptr(out, ctypes.c_int32), cap, ctypes.byref(slots), err, 256)
    assert k > 0, err.value.decode()
    return out[:k].copy(), slots.value


def verify(lib, n, rp, col, val, ops, slots):
    rp, col, val = (np.ascontiguousarray(rp, np.int32), np.ascontiguousarray(col, np.int32),
                    np.ascontiguousarray(val, np.float32))
    ops = np.ascontiguousarray(ops, np.int32)
    return lib.plan_shim_verify(n, _ptr(rp, ctypes.c_int32), _ptr(col, ctypes.c_int32), _ptr(val, ctypes.c_float),
                                _ptr(ops, ctypes.c_int32), len(ops), slots) == 1


def replay(lib, n, rp, col, val, ops, slots, z):
    """Runs the plan on slot values z (float32 [n]) as the kernel does and
    returns the row sums; asserts the plan's structural limits on the way."""
    batch, rows_max = lib.plan_shim_batch(), lib.plan_shim_rows()
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
            acc = np.float32(0.0)
            for k in range(nent):
                sl, bits = int(ops[pc]), int(ops[pc + 1])
                pc += 2
                w = np.array([bits], np.int32).view(np.float32)[0]
                assert holder[sl] == col[rp[r] + k] and w == val[rp[r] + k]
                acc = np.float32(acc + np.float32(w * lds[sl]))
            assert not done[r]
            done[r] = True
            out[r] = acc
    assert pc == len(ops) and done.all()
    return out


def dense_order_sums(n, rp, col, val, z):
    out = np.zeros(n, np.float32)
    for i in range(n):
        acc = np.float32(0.0)
        for k in range(rp[i], rp[i + 1]):
            acc = np.float32(acc + np.float32(np.float32(val[k]) * z[col[k]]))
        out[i] = acc
    return out


def check(lib, n, rp, col, val, seed=0):
    ops, slots = plan(lib, n, rp, col, val)
    assert 1 <= slots <= n
    assert len(ops) <= lib.plan_shim_words_max(n)
    z = np.random.default_rng(seed).standard_normal(n).astype(np.float32)
    got = replay(lib, n, rp, col, val, ops, slots, z)
    assert np.array_equal(got.view(np.uint32), dense_order_sums(n, rp, col, val, z).view(np.uint32))
    assert verify(lib, n, rp, col, val, ops, slots)
    return ops, slots


KINDS = ["ring", "complete", "exponential", "one_peer_exp", "one_peer", "two_peer", "random_regular"]


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("n", [1, 2, 5, 16, 17, 32, 33, 64])
def test_generated_graphs_replay_exactly(shim, kind, n):
    if kind == "random_regular" and (n <= 3 or (3 * n) % 2):
        pytest.skip("3-regular graph needs n > 3 and 3n even")
    for t in range(6):
        rp, col, val = oracle.topology_csr(kind, n, 3, t, 3)
        ops, slots = check(shim, n, rp, col, val, seed=t)
        if kind in ("one_peer", "ring") and n >= 16:
            assert slots <= 8, (kind, n, slots)  # sparse graphs reuse slots


def test_random_csrs_with_dense_rows_and_missing_diagonals(shim):
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
        check(shim, n, rp, col, val, seed=trial)


def test_tampered_plans_are_rejected(shim):
    n = 12
    rp, col, val = oracle.topology_csr("two_peer", n, 5, 2)
    ops, slots = check(shim, n, rp, col, val)
    rejected = 0
    for k in range(len(ops)):
        for d in (-1, 1, 1000):
            bad = ops.copy()
            bad[k] += d
            rejected += not verify(shim, n, rp, col, val, bad, slots)
    assert rejected == 3 * len(ops)
    assert not verify(shim, n, rp, col, val, ops[:-1], slots)
    assert not verify(shim, n, rp, col, val, ops, slots - 1)


"""Oracle pins: communication graphs against the paper's definitions (host, no GPU).

Every mixing matrix is checked against an independent construction from the
Laplacian form of section 3.1 (W = I - alpha * Lambda) or the graph's own
definition, and the random schedules against Proposition 1 (section 3.2)
and the edge probabilities of its proof (App. A).
"""
import math

import numpy as np
import pytest

import oracle
from tests.bruteforce import laplacian

KINDS = ["ring", "complete", "exponential", "one_peer_exp", "one_peer", "two_peer", "random_regular"]


def dense(kind, n, seed, t, degree=3):
    return oracle.csr_to_dense(*oracle.topology_csr(kind, n, seed, t, degree), n)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 8, 16, 33, 64])
def test_csr_invariants(kind, n):
    if kind == "random_regular" and (n <= 3 or (n * 3) % 2):
        pytest.skip("3-regular graph needs n > 3 and 3n even")
    for t in range(4):
        row_ptr, col, val = oracle.topology_csr(kind, n, 3, t)
        assert row_ptr[0] == 0 and row_ptr[-1] == len(col)
        for i in range(n):
            cols = col[row_ptr[i]:row_ptr[i + 1]]
            assert list(cols) == sorted(set(cols.tolist())), "ascending, no duplicates"
            assert i in cols, "the node itself is always a neighbour"
            assert np.all(val[row_ptr[i]:row_ptr[i + 1]] > 0)
            assert abs(float(np.sum(val[row_ptr[i]:row_ptr[i + 1]].astype(np.float64))) - 1.0) <= 1e-6


@pytest.mark.parametrize("kind", KINDS)
def test_schedule_is_a_function_of_seed_and_round(kind):
    n = 16
    a = [dense(kind, n, 3, t) for t in range(6)]
    b = [dense(kind, n, 3, t) for t in range(6)]
    for wa, wb in zip(a, b):
        assert np.array_equal(wa, wb)
    if kind in ("one_peer", "two_peer", "random_regular"):
        assert any(not np.array_equal(a[0], w) for w in a[1:]), "a fresh graph every round"
        assert not np.array_equal(dense(kind, n, 3, 0), dense(kind, n, 4, 0))


@pytest.mark.parametrize("n", [4, 6, 7, 16])
def test_one_peer_is_I_minus_Lambda1(n):
    # Lambda1_sigma = 1/2 sum_k (e_{s(2k)} - e_{s(2k+1)})(...)^T (section 3.2), alpha = 1
    for t in range(5):
        sigma = oracle.shuffled_identity(oracle.round_state(3, t), n)
        pairs = [(sigma[2 * k], sigma[2 * k + 1]) for k in range(n // 2)]
        L1 = laplacian(n, pairs, [1.0] * len(pairs))
        np.testing.assert_allclose(dense("one_peer", n, 3, t), np.eye(n) - L1, rtol=0, atol=1e-7)
        np.testing.assert_allclose(L1 @ L1, L1, atol=1e-12)  # idempotent (App. A)


@pytest.mark.parametrize("n", [3, 4, 5, 16])
def test_two_peer_is_I_minus_four_thirds_Lambda2(n):
    # Lambda2_sigma = 1/2 sum_i 1/2 (e_{s(i)} - e_{s(i+1)})(...)^T (section 3.2).
    # Uniform 1/|N_i| = 1/3 weights correspond to alpha = 4/3.
    for t in range(5):
        sigma = oracle.shuffled_identity(oracle.round_state(3, t), n)
        edges = [(sigma[i], sigma[(i + 1) % n]) for i in range(n)]
        L2 = laplacian(n, edges, [0.5] * n)
        np.testing.assert_allclose(dense("two_peer", n, 3, t), np.eye(n) - 4.0 / 3.0 * L2, atol=1e-7)


@pytest.mark.parametrize("n", [3, 4, 9])
def test_ring_is_identity_cycle(n):
    edges = [(i, (i + 1) % n) for i in range(n)]
    L = laplacian(n, edges, [0.5] * n)
    np.testing.assert_allclose(dense("ring", n, 0, 0), np.eye(n) - 4.0 / 3.0 * L, atol=1e-7)


def test_ring_n4_spectrum_matches_golden(golden_dir):
    with open(golden_dir + "/ring_n4_spectrum.txt") as f:
        line = [ln for ln in f if ln.strip() and not ln.startswith("#")][0]
    expected = [float(eval(tok)) for tok in line.split()]  # "2/3" style fractions
    W = dense("ring", 4, 0, 0)
    got = np.sort(np.linalg.eigvalsh(np.eye(4) - (W + W.T) / 2))
    np.testing.assert_allclose(got, expected, atol=1e-6)


@pytest.mark.parametrize("n", [1, 2, 5, 16])
def test_complete_is_I_minus_pi(n):
    pi = np.eye(n) - np.ones((n, n)) / n
    np.testing.assert_allclose(dense("complete", n, 0, 0), np.eye(n) - pi, atol=1e-7)


@pytest.mark.parametrize("n", [5, 8, 16])
def test_exponential_is_circulant_hops(n):
    hops = []
    h = 1
    while h < n:
        hops.append(h)
        h *= 2
    W = np.zeros((n, n))
    for i in range(n):
        nb = {i} | {(i + h) % n for h in hops}
        for j in nb:
            W[i, j] = 1.0 / len(nb)
    np.testing.assert_allclose(dense("exponential", n, 0, 0), W, atol=1e-7)
    np.testing.assert_allclose(W.sum(axis=0), 1.0, atol=1e-7)  # doubly stochastic


def test_one_peer_exp_cycles_hops_n16():
    n = 16
    for t in range(10):
        hop = 2 ** (t % 4)
        W = np.eye(n) * 0.5
        for i in range(n):
            W[i, (i + hop) % n] += 0.5
        np.testing.assert_allclose(dense("one_peer_exp", n, 3, t), W, atol=0)


@pytest.mark.parametrize("n", [4, 8, 32])
def test_random_regular_simple_and_metropolis(n):
    for t in range(6):
        W = dense("random_regular", n, 3, t)
        A = (W > 0) & ~np.eye(n, dtype=bool)
        assert np.array_equal(A, A.T)
        assert np.all(A.sum(axis=1) == 3)
        L = np.diag(A.sum(axis=1)) - A.astype(float)
        np.testing.assert_allclose(W, np.eye(n) - L / 4.0, atol=1e-7)  # Metropolis 1/(1+3)


def _edge_frequency(kind, n, rounds, seed=3):
    counts = np.zeros((n, n))
    for t in range(rounds):
        W = dense(kind, n, seed, t)
        counts += (W > 0) & ~np.eye(n, dtype=bool)
    return counts / rounds


@pytest.mark.parametrize("kind,num", [("one_peer", 1.0), ("two_peer", 2.0), ("random_regular", 3.0)])
def test_edge_probabilities(kind, num):
    # matching 1/(n-1), cycle 2/(n-1) (App. A, proof of Proposition 1); d-regular d/(n-1)
    n, rounds = 8, 6000
    freq = _edge_frequency(kind, n, rounds)
    p = num / (n - 1)
    off = freq[~np.eye(n, dtype=bool)]
    se = math.sqrt(p * (1 - p) / rounds)
    assert np.all(np.abs(off - p) < 5 * se)


def _prop1_coeffs(golden_dir):
    out = {}
    with open(golden_dir + "/proposition1.txt") as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                name, num, den = line.split()
                out[name] = (float(num), den)
    return out


@pytest.mark.parametrize("n", [4, 6, 8])
def test_proposition1_expectations(n, golden_dir):
    coeffs = _prop1_coeffs(golden_dir)

    def coeff(name):
        num, den = coeffs[name]
        scale = {"2(n-1)": 2 * (n - 1), "8(n-1)": 8 * (n - 1), "(n-1)": n - 1}[den]
        return num * n / scale if den != "(n-1)" else num / scale

    pi = np.eye(n) - np.ones((n, n)) / n
    rounds = 20000
    acc = {k: np.zeros((n, n)) for k in ("L1", "L1sq", "L2", "L2sq")}
    for t in range(rounds):
        L1 = np.eye(n) - dense("one_peer", n, 9, t)  # alpha = 1
        L2 = (np.eye(n) - dense("two_peer", n, 9, t)) * 0.75  # alpha = 4/3
        acc["L1"] += L1
        acc["L1sq"] += L1 @ L1
        acc["L2"] += L2
        acc["L2sq"] += L2 @ L2
    for key, name in (("L1", "E_L1"), ("L1sq", "E_L1sq"), ("L2", "E_L2"), ("L2sq", "E_L2sq")):
        np.testing.assert_allclose(acc[key] / rounds, coeff(name) * pi, atol=0.02)
    assert coeff("P_edge_matching") == pytest.approx(1 / (n - 1))

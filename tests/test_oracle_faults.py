"""Oracle pins for fault tolerance and restricted peer selection (host).

* Section 3.2 "Fault tolerance": a failed exchange is skipped.  Each endpoint
  keeps the weight it would have sent: W stays row stochastic, a symmetric W
  stays doubly stochastic (so the mean is preserved, App. A), a dead worker
  only keeps itself and nobody reads it.
* App. B.1: the randomized 1-/2-Peer selections restricted to the edges of an
  admissible graph; with the complete graph admissible nothing changes.
"""
import math

import numpy as np
import pytest

import oracle
from tests.test_oracle_round import HP, close, grads_fn


def dense(W, n):
    return oracle.csr_to_dense(*W, n)


def ring_adjacency(n):
    A = np.zeros((n, n), np.uint8)
    for i in range(n):
        A[i, (i + 1) % n] = A[(i + 1) % n, i] = 1
    return A


def random_adjacency(n, p, seed):
    rng = np.random.default_rng(seed)
    A = (rng.random((n, n)) < p).astype(np.uint8)
    A = np.triu(A, 1)
    return (A + A.T).astype(np.uint8)


def metropolis(adj):
    n = adj.shape[0]
    off = adj.astype(bool) & ~np.eye(n, dtype=bool)
    deg = off.sum(axis=1)
    W = np.zeros((n, n))
    for i in range(n):
        for j in np.nonzero(off[i])[0]:
            W[i, j] = 1.0 / (1 + max(deg[i], deg[j]))
        W[i, i] = 1.0 - W[i].sum()
    return W


@pytest.mark.parametrize("kind", ["one_peer", "two_peer"])
@pytest.mark.parametrize("n", [4, 7, 16])
def test_complete_admissible_graph_changes_nothing(kind, n):
    full = np.ones((n, n), np.uint8)
    for t in range(30):
        a = oracle.topology_csr(kind, n, 3, t)
        b = oracle.topology_csr(kind, n, 3, t, admissible=full)
        for u, v in zip(a, b):
            assert np.array_equal(u, v)


@pytest.mark.parametrize("kind", ["one_peer", "two_peer"])
@pytest.mark.parametrize("adj_name", ["ring", "random"])
def test_restricted_selection_matches_its_definition(kind, adj_name):
    n = 12
    A = ring_adjacency(n) if adj_name == "ring" else random_adjacency(n, 0.4, 5)
    for t in range(40):
        sigma = oracle.shuffled_identity(oracle.round_state(3, t), n)
        if kind == "one_peer":
            pairs = [(sigma[2 * k], sigma[2 * k + 1]) for k in range(n // 2)]
        else:
            pairs = [(sigma[k], sigma[(k + 1) % n]) for k in range(n)]
        sel = np.eye(n, dtype=np.uint8)
        for a, b in pairs:
            if A[a, b]:
                sel[a, b] = sel[b, a] = 1
        W = dense(oracle.topology_csr(kind, n, 3, t, admissible=A), n)
        np.testing.assert_allclose(W, metropolis(sel), atol=1e-7)
        off = (W > 0) & ~np.eye(n, dtype=bool)
        assert np.all(A[off] == 1), "only admissible edges are used"
        np.testing.assert_allclose(W, W.T, atol=0)
        np.testing.assert_allclose(W.sum(axis=0), 1.0, atol=1e-6)


def test_restricted_matching_edge_probability():
    # the matching is still uniform: an admissible pair is active w.p. 1/(n-1)
    n, rounds = 8, 8000
    A = random_adjacency(n, 0.5, 6)
    freq = np.zeros((n, n))
    for t in range(rounds):
        W = dense(oracle.topology_csr("one_peer", n, 9, t, admissible=A), n)
        freq += (W > 0) & ~np.eye(n, dtype=bool)
    freq /= rounds
    p = 1.0 / (n - 1)
    se = math.sqrt(p * (1 - p) / rounds)
    adm = A.astype(bool) & ~np.eye(n, dtype=bool)
    assert np.all(np.abs(freq[adm] - p) < 5 * se)
    assert np.all(freq[~adm & ~np.eye(n, dtype=bool)] == 0)


def _skip_reference(W, alive, link_ok):
    n = W.shape[0]
    R = W.copy()
    for i in range(n):
        for j in range(n):
            if i == j or W[i, j] == 0:
                continue
            dead = alive is not None and (not alive[i] or not alive[j])
            broken = link_ok is not None and (not link_ok[i, j] or not link_ok[j, i])
            if dead or broken:
                R[i, i] += R[i, j]
                R[i, j] = 0.0
    return R


@pytest.mark.parametrize("kind", ["ring", "exponential", "one_peer", "two_peer", "random_regular", "complete"])
def test_skip_exchanges_definition(kind):
    n = 10
    rng = np.random.default_rng(7)
    for t in range(8):
        W = oracle.topology_csr(kind, n, 3, t, 3)
        Wd = dense(W, n)
        alive = (rng.random(n) > 0.2).astype(np.uint8)
        link = (rng.random((n, n)) > 0.3).astype(np.uint8)
        out = dense(oracle.skip_exchanges(W, n, alive, link), n)
        np.testing.assert_allclose(out, _skip_reference(Wd, alive, link), atol=1e-7)
        np.testing.assert_allclose(out.sum(axis=1), 1.0, atol=1e-6)
        for k in np.nonzero(alive == 0)[0]:
            e = np.zeros(n)
            e[k] = 1
            np.testing.assert_array_equal(out[k], e)  # a dead worker keeps only itself
            assert np.all(out[np.arange(n) != k, k] == 0)  # and nobody reads it
        if np.allclose(Wd, Wd.T):
            np.testing.assert_allclose(out, out.T, atol=0)
            np.testing.assert_allclose(out.sum(axis=0), 1.0, atol=1e-6)
    same = oracle.skip_exchanges(W, n)
    for a, b in zip(same, W):
        assert np.array_equal(a, b)


def test_skipped_exchanges_preserve_the_mean_and_isolate_dead_workers():
    n, P = 8, 32
    hp = oracle.OracleHParams(beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"], weight_decay=HP["wd"],
                              outer_lr=0.7, outer_momentum=0.0, nesterov=True, consensus_momentum=0.0)
    o = oracle.Oracle(n, P, hp, topology="two_peer", seed=3, precision="f64")
    x0 = np.random.default_rng(8).standard_normal((n, P)) * 0.02
    o.x[...] = x0
    o.y[...] = x0
    alive = np.ones(n, np.uint8)
    alive[3] = 0
    g = grads_fn(n, P, seed=400)
    for t in range(4):
        xbar = o.x.mean(axis=0).copy()
        x_dead = o.x[3].copy()
        act = alive.copy()
        o.local_step(g(t), HP["lr"], act)
        gbar = (o.y - o.x).mean(axis=0)
        o.gossip_round(t, csr=oracle.skip_exchanges(o.csr(t), n, alive, precision="f64"))
        close(o.x.mean(axis=0), xbar + 0.7 * gbar, 1e-12)  # App. A mean dynamics
        np.testing.assert_array_equal(o.x[3], x_dead)  # no steps, no neighbours, no momentum

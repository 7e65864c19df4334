"""GPU parity: the HIP library against the oracle on identical seeded inputs.

Every test calls the library through its C ABI (ctypes binding) on cuda:0.
"""
import numpy as np
import pytest

import gasloc_inputs as gi
import oracle
from tests.gpu_harness import Pair, log, reduction_close, within

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_11081_amd as g

    g.library()  # fail loudly if the HIP library is missing
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _run(pair, rounds, H_i, check_every_round=True, tag=""):
    H_i = np.asarray(H_i)
    n = pair.n
    for t in range(rounds):
        for h in range(int(H_i.max()) if H_i.size else 0):
            pair.local_step(active=(H_i > h).astype(np.uint8))
        stepped = np.nonzero(H_i > 0)[0]
        if t == rounds - 1:
            pair.check_state(names=("m", "v"), y_rows=stepped, tag="%s round %d pre-gossip" % (tag, t))
        pair.gossip_round(t)
        if check_every_round or t == rounds - 1:
            ce = pair.gpu.consensus_error()
            o32 = pair.oracles["f32"]
            ce_ref = o32.consensus_error()
            reduction_close(ce, ce_ref, "%s round %d consensus error" % (tag, t))
            if "f64" in pair.oracles:
                # fp64-state drift check (loose); for identical replicas the
                # oracle's two-pass fp64 mean leaves a residue of at most about
                # 3e-34 per element (n <= 64), far under the 1e-24 floor
                ce64 = pair.oracles["f64"].consensus_error()
                assert abs(ce - ce64) <= 1e-3 * abs(ce64) + 1e-24 * n * pair.P, (ce, ce64)
    assert n == pair.n
    return pair.check_state(tag=tag)


def test_ring_n4_p1m_full_state_ten_rounds():
    w = gi.WORKLOADS["ring-n4-p1m"]
    log("case %s: n=%d P=%d" % (w.name, w.n, w.P))
    pair = Pair(w.n, w.P, w.topology, w.param_dtype, gamma=w.gamma)
    stats = _run(pair, w.rounds, gi.local_steps(w), tag=w.name)
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    # the kernels follow the oracle's op order: identical bits are expected
    assert min(stats.values()) == 1.0
    # network average (Algorithm 1 output)
    import torch

    out = torch.empty(w.P, dtype=torch.float32, device="cuda")
    pair.gpu.replica_mean(out)
    torch.cuda.synchronize()
    ref = pair.oracles["f32"].replica_mean()
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("n,P,topology,dtype", [(5, 9_999, "two_peer", "bf16"), (37, 5_003, "one_peer", "f32"),
                                                  (64, 2_051, "complete", "bf16"), (16, 1, "ring", "f32")])
def test_replica_mean_matches_the_oracle(n, P, topology, dtype):
    # the network average (Algorithm 1's output) after rounds that leave the
    # replicas apart: fp32 bits, or bf16 bits rounded from the fp32 mean, as
    # the fp32 oracle stores them; ragged P, odd n, and a single column
    import torch

    log("case replica mean n=%d P=%d %s %s" % (n, P, topology, dtype))
    pair = Pair(n, P, topology, dtype, gamma=0.1)
    for t in range(2):
        pair.local_step()
        pair.gossip_round(t)
    out = torch.empty(P, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")
    pair.gpu.replica_mean(out)
    torch.cuda.synchronize()
    ref = pair.oracles["f32"].replica_mean()
    if dtype == "bf16":
        got = out.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, np.asarray(ref).view(np.uint16))
    else:
        assert np.array_equal(out.cpu().numpy().view(np.uint32), np.asarray(ref).view(np.uint32))


SMALL = [
    # n, P, topology, dtype, H, gamma, mu, nesterov
    (1, 1000, "ring", "f32", 2, 0.1, 0.9, True),
    (2, 4099, "ring", "f32", 1, 0.1, 0.9, True),
    (3, 777, "two_peer", "f32", 2, 0.2, 0.9, True),
    (5, 4097, "one_peer", "f32", 3, 0.0, 0.9, True),
    (8, 10007, "exponential", "f32", 1, 0.1, 0.9, False),
    (16, 8191, "one_peer_exp", "f32", 2, 0.1, 0.0, False),
    (32, 3001, "random_regular", "bf16", 2, 0.1, 0.9, True),
    # fp32 rows of four entries (3-regular graph with its self-loop) take the
    # planned kernel's branch-free sum at 2 columns per thread; ragged P
    (32, 4097, "random_regular", "f32", 2, 0.1, 0.9, True),
    (33, 515, "two_peer", "f32", 1, 0.3, 0.5, True),
    (64, 2053, "complete", "f32", 1, 0.0, 0.9, True),
    (64, 4099, "one_peer", "bf16", 2, 0.0, 0.9, True),
    # n > 16, rows sharing one neighbour sum, with the consensus-momentum term
    (40, 3333, "complete", "f32", 2, 0.1, 0.9, True),
    (34, 2049, "one_peer", "bf16", 1, 0.2, 0.5, False),
    (7, 3, "ring", "f32", 1, 0.1, 0.9, True),
    (4, 1, "complete", "bf16", 1, 0.1, 0.9, True),
]


@pytest.mark.parametrize("n,P,topology,dtype,H,gamma,mu,nesterov", SMALL)
def test_small_cases(n, P, topology, dtype, H, gamma, mu, nesterov):
    log("case n=%d P=%d %s %s H=%d gamma=%g mu=%g nesterov=%s" % (n, P, topology, dtype, H, gamma, mu,
                                                                   nesterov))
    pair = Pair(n, P, topology, dtype, gamma=gamma, mu=mu, nesterov=nesterov)
    H_i = np.full(n, H)
    if n >= 5:
        H_i[1] = 0  # a worker that skips its local steps this round (H_i = 0)
        H_i[-1] = max(1, H - 1)
    stats = _run(pair, 3, H_i, tag="small")
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    if topology == "complete" and gamma == 0.0:
        x = pair.gather("x")
        assert np.all(x == x[0]), "complete graph keeps replicas bit-identical"
        assert pair.gpu.consensus_error() == 0.0


FUSED = [
    # n, P, topology, dtype, H, gamma
    (4, 1_048_576, "ring", "f32", 1, 0.1),
    (16, 100_003, "one_peer_exp", "f32", 3, 0.1),
    (8, 65_537, "exponential", "bf16", 2, 0.1),
    (64, 20_011, "one_peer", "f32", 2, 0.0),
    (33, 9_999, "two_peer", "bf16", 1, 0.2),
    (40, 7_001, "complete", "bf16", 2, 0.1),
]


@pytest.mark.parametrize("n,P,topology,dtype,H,gamma", FUSED)
def test_fused_last_step_matches_two_calls_and_oracle(n, P, topology, dtype, H, gamma):
    import torch

    log("case fused n=%d P=%d %s %s H=%d gamma=%g" % (n, P, topology, dtype, H, gamma))
    H_i = np.full(n, H)
    if n >= 5:
        H_i[2] = 0
        H_i[3] = max(1, H - 1)
    fused = Pair(n, P, topology, dtype, gamma=gamma, precisions=("f32",))
    split = Pair(n, P, topology, dtype, gamma=gamma, precisions=())
    for t in range(3):
        for h in range(int(H_i.max())):
            act = (H_i > h).astype(np.uint8)
            split.local_step(active=act)
            if h == int(H_i.max()) - 1:
                fused.local_step_gossip_round(t, active=act)
            else:
                fused.local_step(active=act)
        split.gossip_round(t)
        ce_f, ce_s = fused.gpu.consensus_error(), split.gpu.consensus_error()
        # the two launches may give a thread a different number of columns, which
        # regroups the fp64 partial sums: equal up to the last bits
        assert abs(ce_f - ce_s) <= 1e-12 * abs(ce_s)
        reduction_close(ce_f, fused.oracles["f32"].consensus_error(), "fused CE round %d" % t)
    torch.cuda.synchronize()
    for name in ("x", "m", "v", "u", "zp"):
        a, b = getattr(fused.gpu, name), getattr(split.gpu, name)
        if a is None:
            continue
        assert torch.equal(a[:, :P], b[:, :P]), name
    assert all(np.array_equal(u, v) for u, v in zip(fused.gpu.counters(), split.gpu.counters()))
    stats = fused.check_state(tag="fused")
    log("bit-exact fraction vs fp32 oracle: %s" % stats)


FORMS = [
    # form, n, P, topology, dtype, H, mu, nesterov
    ("alg1", 8, 40_003, "exponential", "f32", 2, 0.9, True),
    ("alg1", 16, 10_001, "one_peer_exp", "bf16", 1, 0.9, False),
    ("alg1", 5, 777, "complete", "f32", 2, 0.0, True),
    ("dadam", 8, 30_011, "two_peer", "f32", 1, 0.9, True),
    ("dadam", 32, 4_099, "random_regular", "bf16", 2, 0.9, True),
    ("local_dadam", 16, 20_000, "one_peer", "f32", 3, 0.9, True),
    ("local_dadam", 7, 5_001, "ring", "bf16", 1, 0.5, False),
    ("local_dadam", 64, 1_003, "one_peer", "f32", 2, 0.0, True),
    # n > 16 on sparse graphs: the slot-reusing kernel
    ("alg1", 40, 12_345, "two_peer", "f32", 2, 0.9, True),
    ("alg1", 24, 9_001, "random_regular", "bf16", 1, 0.9, False),
    ("dadam", 48, 7_777, "one_peer_exp", "f32", 2, 0.9, True),
    ("local_dadam", 33, 6_007, "exponential", "bf16", 2, 0.9, True),
    # complete graph beyond 16 workers: shared sums (DAdam) and n live slots
    # without them (ALG1, the DiLoCo reduction)
    ("dadam", 40, 5_003, "complete", "bf16", 2, 0.9, True),
    ("alg1", 40, 4_001, "complete", "f32", 2, 0.0, True),
]


@pytest.mark.parametrize("form,n,P,topology,dtype,H,mu,nesterov", FORMS)
def test_round_forms(form, n, P, topology, dtype, H, mu, nesterov):
    log("case form=%s n=%d P=%d %s %s H=%d mu=%g nesterov=%s" % (form, n, P, topology, dtype, H, mu, nesterov))
    pair = Pair(n, P, topology, dtype, gamma=0.0, mu=mu, nesterov=nesterov, form=form)
    H_i = np.full(n, H)
    if n >= 5:
        H_i[1] = 0
    stats = _run(pair, 3, H_i, tag=form)
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    if form == "alg1" and topology == "complete":
        x = pair.gather("x")
        assert np.all(x == x[0]) and pair.gpu.consensus_error() == 0.0


@pytest.mark.parametrize("n,P,topology", [(8, 33_333, "two_peer"), (40, 10_007, "one_peer")])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused_last_step_alg1(dtype, n, P, topology):
    import torch

    log("case fused alg1 n=%d P=%d %s %s" % (n, P, topology, dtype))
    fused = Pair(n, P, topology, dtype, gamma=0.0, form="alg1", precisions=("f32",))
    split = Pair(n, P, topology, dtype, gamma=0.0, form="alg1", precisions=())
    for t in range(3):
        for h in range(2):
            split.local_step()
            if h == 1:
                fused.local_step_gossip_round(t)
            else:
                fused.local_step()
        split.gossip_round(t)
        ce_f, ce_s = fused.gpu.consensus_error(), split.gpu.consensus_error()
        assert abs(ce_f - ce_s) <= 1e-12 * abs(ce_s)  # launches may regroup the fp64 partials
    torch.cuda.synchronize()
    for name in ("x", "m", "v", "u"):
        assert torch.equal(getattr(fused.gpu, name)[:, :P], getattr(split.gpu, name)[:, :P]), name
    fused.check_state(tag="fused alg1")


def test_form_arguments_are_checked():
    import paper_2606_11081_amd as g

    with pytest.raises(g.GaslocError, match="consensus_momentum must be 0"):
        g.GASLoC(4, 256, round_form="alg1", consensus_momentum=0.1)
    d = g.GASLoC(4, 256, round_form="dadam", consensus_momentum=0.0)
    grads = d.x.new_zeros((4, d.ld), dtype=d.m.dtype)
    with pytest.raises(g.GaslocError, match="EQ and ALG1"):
        d.local_step_gossip_round(grads, 0.01, 0)


def test_dead_workers_match_the_oracle_with_skipped_exchanges():
    import paper_2606_11081_amd as g

    n, P = 16, 50_001
    alive = np.ones(n, np.uint8)
    alive[[2, 9]] = 0
    # the library applies the mask itself; the oracle is given the masked W
    # and the masked local steps explicitly
    pair2 = Pair(n, P, "two_peer", "f32", gamma=0.1)
    pair2.gpu.set_alive(alive)
    for t in range(3):
        gi.fill_grads(pair2.grads, pair2.mu_i, pair2.step)
        g_host = pair2.grads[:, pair2.cols_dev].cpu().numpy()
        pair2.gpu.local_step(pair2.grads, pair2.lr)  # active = all, dead ones skipped
        for o in pair2.oracles.values():
            o.local_step(g_host, pair2.lr, alive)
        pair2.step += 1
        pair2.gpu.gossip_round(t)
        for o in pair2.oracles.values():
            o.gossip_round(t, csr=oracle.skip_exchanges(o.csr(t), n, alive, precision=o.precision))
        reduction_close(pair2.gpu.consensus_error(), pair2.oracles["f32"].consensus_error(), "CE round %d" % t)
    k, _, _ = pair2.gpu.counters()
    assert list(k[[2, 9]]) == [0, 0] and all(k[alive == 1] == 3)
    pair2.check_state(tag="dead workers")


def test_nan_gradient_spreads_only_along_the_round_edges():
    import torch

    n, P = 8, 4_096
    pair = Pair(n, P, "one_peer", "f32", gamma=0.0, precisions=("f32",))
    gi.fill_grads(pair.grads, pair.mu_i, 0)
    bad = 5
    pair.grads[bad, 100] = float("nan")
    pair.gpu.local_step(pair.grads, pair.lr)
    pair.gpu.gossip_round(0)
    torch.cuda.synchronize()
    x = pair.gpu.x[:, :P].cpu().numpy()
    W = oracle.csr_to_dense(*oracle.topology_csr("one_peer", n, gi.SEED_TOPOLOGY, 0), n)
    poisoned = np.isnan(x[:, 100])
    assert np.array_equal(poisoned, W[:, bad] != 0), "NaN reaches exactly the workers that read worker %d" % bad
    assert not np.isnan(np.delete(x, 100, axis=1)).any(), "other columns stay finite"
    assert np.isnan(pair.gpu.consensus_error())
    assert np.isnan(pair.gpu.pseudo_gradient_sq())


def test_restricted_schedule_on_device():
    import paper_2606_11081_amd as g

    n, P = 16, 10_007
    rng = np.random.default_rng(5)
    A = np.triu((rng.random((n, n)) < 0.3).astype(np.uint8), 1)
    A = A + A.T
    pair = Pair(n, P, "two_peer", "f32", gamma=0.1)
    gpu2 = g.GASLoC(n, P, topology="two_peer", seed=gi.SEED_TOPOLOGY, admissible=A)
    for t in range(4):
        got = g.gasloc_topology_csr(gpu2.ctx, t, n)
        exp = oracle.topology_csr("two_peer", n, gi.SEED_TOPOLOGY, t, admissible=A)
        for a, b in zip(got, exp):
            assert np.array_equal(a, b)
        pair.local_step()
        pair.gossip_round(t, W=exp)
    pair.check_state(tag="restricted")


def test_explicit_nonsymmetric_csr_and_identity():
    n, P = 6, 5003
    rng = np.random.default_rng(3)
    pair = Pair(n, P, "ring", "f32", gamma=0.2)
    for t in range(3):
        pair.local_step()
        dense = rng.random((n, n)) * (rng.random((n, n)) < 0.5) + np.eye(n)
        dense /= dense.sum(axis=1, keepdims=True)
        rp = np.zeros(n + 1, np.int32)
        cols, vals = [], []
        for i in range(n):
            nz = np.nonzero(dense[i])[0]
            cols += nz.tolist()
            vals += dense[i, nz].tolist()
            rp[i + 1] = len(cols)
        val = np.array(vals, np.float32)
        # renormalise in fp32 so each row sums to 1 within the validator's 1e-6
        W = (rp, np.array(cols, np.int32), val)
        pair.gossip_round(t, W=W)
        reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "explicit CE")
    pair.check_state(tag="explicit")


@pytest.mark.parametrize("density", [0.05, 0.2, 0.6])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_explicit_random_csr_large_n(density, dtype):
    # unstructured graphs at n = 40 (the slot-reusing kernel when the plan
    # reuses slots), some rows without their own entry
    n, P = 40, 20_011
    rng = np.random.default_rng(int(density * 100) + (dtype == "bf16"))
    pair = Pair(n, P, "ring", dtype, gamma=0.1)
    for t in range(3):
        pair.local_step()
        dense = rng.random((n, n)) * (rng.random((n, n)) < density)
        dense[np.arange(n), np.arange(n)] = (rng.random(n) < 0.8) * rng.random(n)
        dense[dense.sum(axis=1) == 0, 0] = 1.0
        dense /= dense.sum(axis=1, keepdims=True)
        rp = np.zeros(n + 1, np.int32)
        cols, vals = [], []
        for i in range(n):
            nz = np.nonzero(dense[i])[0]
            cols += nz.tolist()
            vals += dense[i, nz].tolist()
            rp[i + 1] = len(cols)
        pair.gossip_round(t, W=(rp, np.array(cols, np.int32), np.array(vals, np.float32)))
        reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "CE round %d" % t)
    pair.check_state(tag="explicit n=40 density %g" % density)


def _csr_from_rows(rows):
    rp = np.zeros(len(rows) + 1, np.int32)
    cols, vals = [], []
    for i, (c, w) in enumerate(rows):
        cols += list(c)
        vals += list(w)
        rp[i + 1] = len(cols)
    return rp, np.array(cols, np.int32), np.array(vals, np.float32)


@pytest.mark.parametrize("form,dtype", [("eq", "f32"), ("eq", "bf16"), ("dadam", "f32")])
def test_explicit_csr_with_equal_rows(form, dtype):
    # groups of rows with equal entries at n = 24: rows 0-5 all read workers
    # 0-5 (each holds its own column: five of them take the first one's sum);
    # rows 6-9 all read workers 8 and 9 (rows 6 and 7 lack their own column,
    # so only rows 8 and 9 may take another row's sum); the rest are distinct
    n, P = 24, 12_007
    rng = np.random.default_rng(5 + (dtype == "bf16") + 2 * (form == "dadam"))
    pair = Pair(n, P, "ring", dtype, gamma=0.1 if form == "eq" else 0.0, form=form)
    for t in range(3):
        pair.local_step()
        w6 = rng.random(6) + 0.1
        w2 = rng.random(2) + 0.1
        rows = [(range(6), w6 / w6.sum())] * 6 + [((8, 9), w2 / w2.sum())] * 4
        for i in range(10, n):
            c = sorted({i, (i + 1 + t) % n, (i + 5) % n})
            w = rng.random(len(c)) + 0.1
            rows.append((c, w / w.sum()))
        pair.gossip_round(t, W=_csr_from_rows(rows))
        reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "CE round %d" % t)
    pair.check_state(tag="equal rows %s %s" % (form, dtype))


@pytest.mark.parametrize("n,dtype,fused", [(3, "f32", False), (12, "bf16", True), (24, "bf16", False),
                                           (33, "f32", True), (40, "bf16", False), (64, "f32", True),
                                           (64, "bf16", True), (20, "bf16", True)])
def test_rows_all_equal_share_one_running_sum(n, dtype, fused):
    # every row holds the same entries (the complete graph, DiLoCo's average):
    # the EQ round keeps one running sum per column and each row's own gamma
    # term.  Shared rows that skip most workers (so most rows lack their own
    # column), hold an explicit zero weight, or name every worker; the gamma
    # term from the second round on; fused and standalone rounds (the fused
    # bf16 round at 17-32 workers runs the planned kernel)
    P = 5_003
    log("case all rows equal n=%d %s fused=%s" % (n, dtype, fused))
    rng = np.random.default_rng(n + 100 * (dtype == "bf16"))
    pair = Pair(n, P, "ring", dtype, gamma=0.1)
    for t in range(4):
        if t == 0:
            cols = list(range(n))
            w = np.full(n, 1.0 / n)
        elif t == 1:
            cols = [0, min(1, n - 1)] if n > 1 else [0]
            cols = sorted(set(cols))
            w = np.full(len(cols), 1.0 / len(cols))
        elif t == 2:
            cols = sorted(set([0, n // 2, n - 1]))
            w = np.zeros(len(cols))
            w[0] = 0.5
            w[-1] += 0.5  # the middle entry has weight 0 (an explicit zero)
        else:
            cols = sorted(rng.choice(n, size=max(1, n // 3), replace=False).tolist())
            w = rng.random(len(cols)) + 0.1
            w = w / w.sum()
        W = _csr_from_rows([(cols, w)] * n)
        if fused:
            pair.local_step()
            pair.local_step_gossip_round(t, W=W)
        else:
            pair.local_step()
            pair.gossip_round(t, W=W)
        reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "CE round %d" % t)
    stats = pair.check_state(tag="all rows equal n=%d %s" % (n, dtype))
    assert min(stats.values()) == 1.0, stats


@pytest.mark.parametrize("n,P,dtype", [(16, 4_099, "f32"), (32, 1, "bf16"), (32, 2_051, "f32"), (17, 777, "bf16")])
def test_rows_all_equal_with_partial_activity(n, P, dtype):
    # the shared-row kernel at its register-array boundaries (16 and 32
    # workers), a single column, and heterogeneous activity: some workers
    # skip the fused step, one takes no local step at all (its y is its x)
    log("case all rows equal, partial activity n=%d P=%d %s" % (n, P, dtype))
    pair = Pair(n, P, "ring", dtype, gamma=0.1)
    rng = np.random.default_rng(7 * n + P)
    W = _csr_from_rows([(list(range(n)), np.full(n, 1.0 / n))] * n)
    for t in range(3):
        first = np.ones(n, np.uint8)
        first[n // 3] = 0  # no local step this round
        pair.local_step(active=first)
        last = (rng.random(n) < 0.6).astype(np.uint8)
        last[n // 3] = 0
        if t % 2 == 0:
            pair.local_step_gossip_round(t, active=last, W=W)
        else:
            pair.local_step(active=last)
            pair.gossip_round(t, W=W)
        reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "CE round %d" % t)
    stats = pair.check_state(tag="all rows equal, partial activity n=%d %s" % (n, dtype))
    assert min(stats.values()) == 1.0, stats


def _bf16_edge_pairs(rng, P):
    """Two rows of bf16 bit patterns whose fp32 midpoints meet the rounding
    cases: adjacent values (exact ties, both parities of the lower one), random
    finite values, subnormals, signed zeros and the largest finite values."""
    finite = lambda k: rng.integers(0, 0x7F80, k).astype(np.uint16) | (rng.integers(0, 2, k).astype(np.uint16) << 15)
    a = finite(P)
    b = finite(P)
    q = P // 5
    b[:q] = a[:q] + 1  # the next bf16 value of the same sign: the midpoint is a tie
    fix = (a[:q] & 0x7FFF) == 0x7F7F  # the next one after the largest finite is infinity
    b[:q][fix] = a[:q][fix] - 1
    sub = slice(q, 2 * q)  # subnormals (exponent field 0), either sign
    a[sub] = (a[sub] & 0x807F)
    b[sub] = (b[sub] & 0x807F)
    z = 2 * q
    a[z:z + 4] = [0x0000, 0x8000, 0x0000, 0x8000]  # +0, -0 in every combination
    b[z:z + 4] = [0x0000, 0x0000, 0x8000, 0x8000]
    a[z + 4:z + 8] = [0x7F7F, 0xFF7F, 0x7F7F, 0x7F7E]  # the largest finite values
    b[z + 4:z + 8] = [0x7F7F, 0xFF7F, 0x7F7E, 0x7F7F]
    return a, b


@pytest.mark.parametrize("n", [2, 18])
def test_bf16_rounding_edge_cases(n):
    """bf16 stores round to nearest, ties to even, keep subnormals and signed
    zeros, as the oracle does and as an independent rounding (torch's CPU
    conversion) of the same fp32 sums does.  With no local steps, mu = gamma =
    0 and rows averaging pairs of workers with weights 1/2, each stored value
    is the rounding of (0 + z_a/2) + z_b/2, with z = x: the exact midpoint of
    two stored values.  n = 2 runs the phase kernel, n = 18 the planned one."""
    import torch

    import paper_2606_11081_amd as g

    P = 4099
    rng = np.random.default_rng(21 + n)
    bits = np.empty((n, P), np.uint16)
    for k in range(0, n, 2):
        bits[k], bits[k + 1] = _bf16_edge_pairs(rng, P)
    log("case bf16 rounding: n=%d P=%d" % (n, P))
    gpu = g.GASLoC(n, P, topology="ring", param_dtype="bf16", outer_momentum=0.0, consensus_momentum=0.0,
                   outer_lr=0.7)
    gpu.x[:, :P].view(torch.int16).copy_(torch.from_numpy(bits.view(np.int16)).cuda())
    hp = oracle.OracleHParams(beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY,
                              outer_lr=0.7, outer_momentum=0.0, nesterov=True, consensus_momentum=0.0)
    o = oracle.Oracle(n, P, hp, param_dtype="bf16")
    o.x[...] = bits
    o.y[...] = bits  # no local steps: y is x
    W = _csr_from_rows([((k - k % 2, k - k % 2 + 1), (0.5, 0.5)) for k in range(n)])
    gpu.gossip_round(0, W)
    o.gossip_round(0, csr=W)
    torch.cuda.synchronize()
    got = gpu.x[:, :P].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, o.x), "bf16 stores differ from the oracle"
    # independent of both: fp32 sums in the same order, rounded by torch on the CPU
    f = oracle.bf16_bits_to_f32(bits)
    half = np.float32(0.5)
    ref = np.empty_like(bits)
    for k in range(n):
        lo = k - k % 2
        mid = (np.float32(0.0) + half * f[lo]) + half * f[lo + 1]
        ref[k] = torch.from_numpy(mid).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref), "bf16 stores differ from round-to-nearest-even"
    # the first fifth of each pair of rows are neighbours: every midpoint is a tie
    assert np.all(got[:, : P // 5] % 2 == 0), "a tie did not go to the even neighbour"
    gpu.close()


def test_all_inactive_step_changes_nothing():
    import torch

    n, P = 4, 1024
    pair = Pair(n, P, "ring", "f32")
    before = {k: getattr(pair.gpu, k).clone() for k in ("x", "m", "v")}
    pair.local_step(active=np.zeros(n, np.uint8))
    torch.cuda.synchronize()
    for k, t in before.items():
        assert torch.equal(t, getattr(pair.gpu, k))
    k, stepped, rounds = pair.gpu.counters()
    assert list(k) == [0] * n and list(stepped) == [0] * n and rounds == 0


def test_runs_are_bit_identical():
    import torch

    outs = []
    for _ in range(2):
        pair = Pair(16, 100_003, "one_peer_exp", "f32", precisions=("f32",))
        for t in range(2):
            pair.local_step()
            pair.local_step()
            pair.gossip_round(t)
        ce = pair.gpu.consensus_error()
        torch.cuda.synchronize()
        P = pair.P  # columns beyond P (row padding) are never touched by the library
        outs.append((pair.gpu.x[:, :P].clone(), pair.gpu.u[:, :P].clone(), pair.gpu.zp[:, :P].clone(), ce))
    for a, b in zip(outs[0][:3], outs[1][:3]):
        assert torch.equal(a, b)
    assert outs[0][3] == outs[1][3]


def test_checkpoint_resume_is_bit_exact():
    import torch

    import paper_2606_11081_amd as g

    n, P = 8, 20_001
    full = Pair(n, P, "two_peer", "f32", precisions=("f32",))
    for t in range(2):
        full.local_step()
        full.gossip_round(t)
    torch.cuda.synchronize()
    saved = {k: getattr(full.gpu, k).clone() for k in ("x", "y", "m", "v", "u", "zp")}
    k, stepped, rounds = full.gpu.counters()
    step = full.step
    for t in range(2, 4):
        full.local_step()
        full.gossip_round(t)
    torch.cuda.synchronize()

    resumed = Pair(n, P, "two_peer", "f32", precisions=())  # compared with `full`, not an oracle
    torch.cuda.synchronize()
    for name, t_ in saved.items():
        getattr(resumed.gpu, name).copy_(t_)
    resumed.gpu.set_counters(k, stepped, rounds)
    resumed.step = step
    for t in range(2, 4):
        resumed.local_step()
        resumed.gossip_round(t)
    torch.cuda.synchronize()
    for name in ("x", "m", "v", "u", "zp"):
        assert torch.equal(getattr(full.gpu, name)[:, :P], getattr(resumed.gpu, name)[:, :P]), name
    assert full.gpu.consensus_error() == resumed.gpu.consensus_error()
    assert full.gpu.pseudo_gradient_sq() == resumed.gpu.pseudo_gradient_sq()


@pytest.mark.parametrize("n,topology", [(8, "ring"), (40, "one_peer")])
def test_pseudo_gradient_statistic_zero_cases(n, topology):
    # 0 before any round, and for a round without local steps (y = x)
    pair = Pair(n, 10_007, topology, "f32", gamma=0.1, precisions=("f32",))
    assert pair.gpu.pseudo_gradient_sq() == 0.0
    pair.local_step()
    pair.gossip_round(0)  # checked against the oracle inside
    assert pair.gpu.pseudo_gradient_sq() > 0.0
    pair.gossip_round(1)
    assert pair.gpu.pseudo_gradient_sq() == 0.0


@pytest.mark.parametrize("n,topology,dtype", [(16, "one_peer_exp", "f32"), (32, "random_regular", "bf16")])
def test_consensus_error_columns_and_closed_form(n, topology, dtype):
    # the standalone reduction over column ranges that start and end off the
    # 16-byte column groups (4 fp32 or 8 bf16 columns), against the oracle
    import torch

    P = 1_000_003
    log("case consensus error columns n=%d %s %s" % (n, topology, dtype))
    pair = Pair(n, P, topology, dtype, precisions=("f32",))
    pair.local_step()
    pair.gossip_round(0)
    fused = pair.gpu.consensus_error()
    total = pair.gpu.consensus_error_cols(0, P)
    reduction_close(total, fused, "standalone vs fused")
    o = pair.oracles["f32"]
    for a, b in [(0, 1), (0, 4097), (5, 70_001), (3, 11), (P - 999, P), (P - 5, P), (123_456, 123_456)]:
        got = pair.gpu.consensus_error_cols(a, b)
        reduction_close(got, o.consensus_error(slice(a, b)) if b > a else 0.0, "cols [%d,%d)" % (a, b))
    # closed form: x_i = c_i on every column -> CE = P * sum_i (c_i - cbar)^2 exactly
    c = torch.arange(1, n + 1, dtype=torch.float32, device="cuda").view(n, 1)  # exact in bf16 too
    pair.gpu.x[:, :P].copy_(c.expand(n, P).to(pair.gpu.x.dtype))
    expect = P * float(((np.arange(1, n + 1) - (n + 1) / 2.0) ** 2).sum())
    assert pair.gpu.consensus_error_cols(0, P) == expect


def test_error_paths_on_device():
    import torch

    import paper_2606_11081_amd as g

    pair = Pair(4, 1024, "ring", "f32", precisions=("f32",))
    ctx = pair.gpu.ctx
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_local_step(ctx, pair.grads.data_ptr() + 4, pair.gpu.ld, None, 0.1)  # misaligned
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_local_step(ctx, pair.grads, pair.gpu.ld, None, float("nan"))
    bad = (np.array([0, 1, 2, 3, 4], np.int32), np.array([0, 1, 2, 4], np.int32),
           np.ones(4, np.float32))
    with pytest.raises(g.GaslocError, match="out of range"):
        g.gasloc_gossip_round(ctx, bad, 0)
    with pytest.raises(g.GaslocError, match="EINVAL"):
        g.gasloc_consensus_error_cols(ctx, 5, 4)
    # the context keeps working after argument errors
    pair.local_step()
    pair.gossip_round(0)
    reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "after errors")
    # explicit topology needs W every round
    gexp = g.GASLoC(4, 256, topology="explicit")
    with pytest.raises(g.GaslocError, match="EXPLICIT"):
        g.gasloc_gossip_round(gexp.ctx, None, 0)
    torch.cuda.synchronize()


def test_topology_csr_from_context_matches_oracle():
    import paper_2606_11081_amd as g

    gpu = g.GASLoC(32, 256, topology="random_regular", seed=3, degree=3)
    for t in range(20):
        got = gpu.topology_csr(t)
        exp = oracle.topology_csr("random_regular", 32, 3, t, 3)
        for a, b in zip(got, exp):
            assert np.array_equal(a, b)


# ---------------------------------------------------------------------------
# full-size workloads: sampled columns (first/last 64 plus uniform picks)
# ---------------------------------------------------------------------------

FULL = [
    # workload, sampled columns, rounds (each workload's own H_i)
    ("exp-n8-p124m", 1 << 18, 10),
    ("onepeer-exp-n16-p350m", 1 << 20, 5),
    ("regular3-n32-p150m-bf16", 1 << 16, 3),
    ("matching-n64-p50m-hetH", 1 << 16, 3),
]


def test_maximum_row_length_64bit_offsets():
    # P = 2^31 - 1, the largest the ABI accepts: worker 1's row starts beyond
    # element 2^31, so every kernel's element offsets exceed 32 bits, and the
    # ragged last group of each row (P % 4 = 3) is exercised at the far end.
    import torch

    n, P = 2, (1 << 31) - 1
    log("case max row length n=%d P=%d" % (n, P))
    cols = gi.sample_columns(P, 1 << 12)
    pair = Pair(n, P, "ring", "f32", gamma=0.1, cols=cols)
    for t in range(2):
        pair.local_step()
        pair.local_step()
        pair.gossip_round(t)
        # the round's own consensus error: 2^21 steps of 1024 columns, two per
        # workgroup, 2^20 partials summed in segments; the standalone reduction
        # of the same x groups the fp64 sums differently
        fused = pair.gpu.consensus_error()
        whole = pair.gpu.consensus_error_cols(0, P)
        assert abs(fused - whole) <= 1e-12 * abs(whole), (fused, whole)
        tail = pair.gpu.consensus_error_cols(P - 64, P)
        reduction_close(tail, pair.oracles["f32"].consensus_error(slice(len(cols) - 64, len(cols))), "tail CE")
    pair.check_state(tag="max row length")
    del pair
    torch.cuda.empty_cache()


def host_consensus_error(x, n, P, param_dtype, chunk=1 << 23):
    """The oracle's two-pass fp64 consensus error of the whole stored x,
    downloaded column chunk by column chunk (the sum is additive over columns)."""
    import ctypes

    import torch

    L = oracle.lib("f32")
    code = oracle.PARAM_BF16 if param_dtype == "bf16" else oracle.PARAM_NATIVE
    total = 0.0
    for c0 in range(0, P, chunk):
        c1 = min(P, c0 + chunk)
        part = x[:, c0:c1].contiguous()
        host = (part.view(torch.int16).cpu().numpy().view(np.uint16) if param_dtype == "bf16"
                else part.cpu().numpy())
        host = np.ascontiguousarray(host)
        total += L.orc_consensus_error(n, c1 - c0, c1 - c0, code, host.ctypes.data_as(ctypes.c_void_p))
    return total


@pytest.mark.parametrize("name,sample,rounds", FULL)
def test_full_size_sampled(name, sample, rounds):
    import torch

    w = gi.WORKLOADS[name]
    log("case %s (sampled %d columns, %d rounds)" % (name, sample, rounds))
    cols = gi.sample_columns(w.P, sample)
    pair = Pair(w.n, w.P, w.topology, w.param_dtype, gamma=w.gamma, degree=w.degree, cols=cols,
                precisions=("f32",) if w.param_dtype == "bf16" else ("f32", "f64"))
    H_i = gi.local_steps(w)
    for t in range(rounds):
        # as the benchmark runs a round: the last local step fused into the round
        last = int(H_i.max()) - 1
        for h in range(last):
            pair.local_step(active=(H_i > h).astype(np.uint8))
        pair.local_step_gossip_round(t, active=(H_i > last).astype(np.uint8))
        fused = pair.gpu.consensus_error()
        assert np.isfinite(fused) and fused >= 0.0
        # the full-size CE from the round kernel against the standalone reduction
        # kernel over all P columns (other kernel, other summation order)
        whole = pair.gpu.consensus_error_cols(0, w.P)
        assert abs(whole - fused) <= 1e-10 * fused, (whole, fused)
        # edge slices of the row are contiguous in both index spaces
        head = pair.gpu.consensus_error_cols(0, 64)
        tail = pair.gpu.consensus_error_cols(w.P - 64, w.P)
        o = pair.oracles["f32"]
        reduction_close(head, o.consensus_error(slice(0, 64)), "%s round %d CE head" % (name, t))
        reduction_close(tail, o.consensus_error(slice(len(cols) - 64, len(cols))), "%s CE tail" % name)
        log("round %d: CE %.6e" % (t, fused))
    # the fused full-size CE of the last round against the oracle's definition
    # over the whole downloaded state
    whole_host = host_consensus_error(pair.gpu.x, w.n, w.P, w.param_dtype)
    assert abs(whole_host - fused) <= 1e-9 * whole_host, (whole_host, fused)
    stats = pair.check_state(tag=name)
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    del pair
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n,P,dtype", [(16, 350_000_000, "f32"), (64, 50_000_000, "f32"), (32, 150_000_000, "bf16")])
def test_full_size_sampled_two_peer(n, P, dtype):
    # the paper's randomized 2-Peer cycle (section 3.2) at the workloads'
    # sizes: H = 3, the last step fused, gamma = 0.1; 2^16 sampled columns
    import torch

    log("case two_peer n=%d P=%d %s (sampled 65536 columns, 3 rounds)" % (n, P, dtype))
    cols = gi.sample_columns(P, 1 << 16)
    pair = Pair(n, P, "two_peer", dtype, gamma=0.1, cols=cols,
                precisions=("f32",) if dtype == "bf16" else ("f32", "f64"))
    for t in range(3):
        for _ in range(2):
            pair.local_step()
        pair.local_step_gossip_round(t)
        ce = pair.gpu.consensus_error()
        whole = pair.gpu.consensus_error_cols(0, P)
        assert abs(whole - ce) <= 1e-10 * ce, (whole, ce)
        o = pair.oracles["f32"]
        reduction_close(pair.gpu.consensus_error_cols(P - 64, P),
                        o.consensus_error(slice(len(cols) - 64, len(cols))), "CE tail")
    stats = pair.check_state(tag="two_peer n=%d %s" % (n, dtype))
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    del pair
    torch.cuda.empty_cache()


@pytest.mark.parametrize("form", ["alg1", "dadam", "local_dadam"])
def test_full_size_sampled_round_forms(form):
    # the other round forms at the n=64, P=50M matching workload's full size,
    # as the benchmark runs them (gamma = 0; Algorithm 1 with the last local
    # step fused into the round, the DAdam forms as separate calls): 2^16
    # sampled columns against both oracles, the full-size CE two ways
    import torch

    w = gi.WORKLOADS["matching-n64-p50m-hetH"]
    log("case %s %s (sampled 65536 columns, 2 rounds)" % (w.name, form))
    cols = gi.sample_columns(w.P, 1 << 16)
    pair = Pair(w.n, w.P, w.topology, w.param_dtype, gamma=0.0, degree=w.degree, cols=cols, form=form)
    H_i = gi.local_steps(w)
    fuse = form == "alg1"
    for t in range(2):
        last = int(H_i.max()) - (1 if fuse else 0)
        for h in range(last):
            pair.local_step(active=(H_i > h).astype(np.uint8))
        if fuse:
            pair.local_step_gossip_round(t, active=(H_i > last).astype(np.uint8))
        else:
            pair.gossip_round(t)
        ce = pair.gpu.consensus_error()
        assert np.isfinite(ce) and ce >= 0.0
        whole = pair.gpu.consensus_error_cols(0, w.P)
        assert abs(whole - ce) <= 1e-10 * ce, (whole, ce)
        o = pair.oracles["f32"]
        reduction_close(pair.gpu.consensus_error_cols(0, 64), o.consensus_error(slice(0, 64)), "CE head")
        reduction_close(pair.gpu.consensus_error_cols(w.P - 64, w.P),
                        o.consensus_error(slice(len(cols) - 64, len(cols))), "CE tail")
        log("round %d: CE %.6e" % (t, ce))
    stats = pair.check_state(tag="%s %s" % (w.name, form))
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    del pair
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_extreme_gradients_bit_exact(dtype):
    # IEEE behaviour the op order relies on: subnormal squares (g ~ 1e-20 gives
    # g*g ~ 1e-40), squares that overflow to inf (|g| >= 2e19), exact zeros and
    # signed tiny values must round exactly as the oracle's do
    import torch

    n, P = 4, 4096
    pair = Pair(n, P, "ring", dtype, gamma=0.1, precisions=("f32",))
    rng = np.random.default_rng(21)
    specials = np.array([0.0, -0.0, 1e-20, -3e-21, 1e-38, 3e-39, -7e-45, 1e19, -2e19, 3e20, 1e-3, -5.0],
                        dtype=np.float32)
    for t in range(2):
        for h in range(2):
            g = rng.standard_normal((n, P)).astype(np.float32)
            idx = rng.integers(0, P, size=(n, 600))
            for i in range(n):
                g[i, idx[i]] = rng.choice(specials, size=600)
            pair.grads[:, :P].copy_(torch.from_numpy(g).to("cuda"))
            pair.gpu.local_step(pair.grads, pair.lr)
            for o in pair.oracles.values():
                o.local_step(g, pair.lr)
        pair.gossip_round(t)
    stats = pair.check_state(tag="extreme gradients")
    log("bit-exact fraction vs fp32 oracle: %s" % stats)
    assert np.isfinite(pair.params_f64(pair.gather("x"))).all()


def test_two_contexts_interleaved_stay_independent():
    # two contexts on the same device, different graphs, dtypes and kernels
    # (n=8 phase kernel, n=40 slot-reusing kernel), rounds interleaved
    a = Pair(8, 9_001, "exponential", "f32", gamma=0.1, precisions=("f32",))
    b = Pair(40, 7_003, "one_peer", "bf16", gamma=0.2, precisions=("f32",))
    for t in range(3):
        a.local_step()
        b.local_step()
        b.local_step()
        a.gossip_round(t)
        b.local_step_gossip_round(t)
        reduction_close(a.gpu.consensus_error(), a.oracles["f32"].consensus_error(), "context a round %d" % t)
        reduction_close(b.gpu.consensus_error(), b.oracles["f32"].consensus_error(), "context b round %d" % t)
    a.check_state(tag="context a")
    b.check_state(tag="context b")


def test_context_on_a_side_stream_matches_the_oracle():
    # every call enqueues on the context's stream: a context made on a side
    # stream (default priority) and fed from that stream gives the oracle's bits
    import torch

    import paper_2606_11081_amd as g

    n, P = 6, 5_003
    side = torch.cuda.Stream()
    gpu = g.GASLoC(n, P, topology="two_peer", seed=gi.SEED_TOPOLOGY, stream=side, beta1=gi.BETA1,
                   beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY, outer_lr=gi.OUTER_LR,
                   outer_momentum=gi.OUTER_MOMENTUM, consensus_momentum=0.1)
    hp = oracle.OracleHParams(beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY,
                              outer_lr=gi.OUTER_LR, outer_momentum=gi.OUTER_MOMENTUM, consensus_momentum=0.1)
    ref = oracle.Oracle(n, P, hp, topology="two_peer", seed=gi.SEED_TOPOLOGY, precision="f32")
    x0 = gi.make_x0(P, device="cuda")  # made on the current stream
    gpu.set_params(x0)
    ref.set_params(x0.cpu().numpy())
    grads = torch.empty((n, gpu.ld), dtype=torch.float32, device="cuda")
    mu = gi.worker_means(n)
    for t in range(3):
        with torch.cuda.stream(side):
            gi.fill_grads(grads, mu, t)
            gpu.local_step(grads, gi.LOCAL_LR)
            if t == 2:
                gpu.local_step_gossip_round(grads, gi.LOCAL_LR, t)
            else:
                gpu.gossip_round(t)
        side.synchronize()
        g_host = grads[:, :P].cpu().numpy()
        ref.local_step(g_host, gi.LOCAL_LR)
        if t == 2:
            ref.local_step(g_host, gi.LOCAL_LR)
        ref.gossip_round(t)
        reduction_close(gpu.consensus_error(), ref.consensus_error(), "side stream round %d" % t)
    side.synchronize()
    for name in ("x", "m", "v", "u", "zp"):
        got = getattr(gpu, name)[:, :P].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), getattr(ref, name).view(np.uint32)), name
    gpu.close()


@pytest.mark.parametrize("n,topology,dtype,form", [
    (8, "exponential", "f32", "eq"),       # phase kernel
    (24, "one_peer", "bf16", "eq"),        # planned kernel, rows sharing sums
    (40, "complete", "f32", "dadam"),
    (33, "two_peer", "bf16", "alg1"),
])
def test_row_padding_is_never_touched(n, topology, dtype, form):
    # columns p >= P of every buffer (and of the gradients and the mean's
    # output) hold a NaN canary through init, local steps, fused and plain
    # rounds and every reduction: none is written, and none leaks into the
    # stored values
    import torch

    from paper_2606_11081_amd import gasloc as gl

    P = 4_099
    ld = gl.padded_ld(P, dtype) + 96
    gld = ld + 40
    canary32, canary16 = 0x7FC0DEAD, 0x7FCD
    pdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    def filled(shape, dt):
        t = torch.empty(shape, dtype=dt, device="cuda")
        if dt == torch.bfloat16:
            t.view(torch.int16).fill_(canary16)
        else:
            t.view(torch.int32).fill_(canary32)
        return t

    x, y = filled((n, ld), pdt), filled((n, ld), pdt)
    m, v, u, zp = (filled((n, ld), torch.float32) for _ in range(4))
    grads = filled((n, gld), torch.float32)
    mean = filled((P + 64,), pdt)
    gamma = 0.1 if form == "eq" else 0.0
    x[:, :P] = gi.make_x0(P, device="cuda").to(pdt)
    hp = gl.make_hparams(param_dtype=dtype, round_form=form, consensus_momentum=gamma)
    stream = torch.cuda.current_stream()
    ctx = gl.gasloc_init(n, P, gl.make_topology_struct(topology, gi.SEED_TOPOLOGY, 3), hp, x, y, m, v, u, zp, ld,
                         stream.cuda_stream)
    try:
        mu = gi.worker_means(n)
        for t in range(3):
            gi.fill_grads(grads[:, :P], mu, t)
            gl.gasloc_local_step(ctx, grads, gld, None, gi.LOCAL_LR)
            if form in ("eq", "alg1") and t != 1:
                gl.gasloc_local_step_gossip_round(ctx, grads, gld, None, gi.LOCAL_LR, None, t)
            else:
                gl.gasloc_gossip_round(ctx, None, t)
            assert np.isfinite(gl.gasloc_consensus_error(ctx))
            assert np.isfinite(gl.gasloc_pseudo_gradient_sq(ctx))
            gl.gasloc_consensus_error_cols(ctx, 1, P)
            gl.gasloc_replica_mean(ctx, mean)
        torch.cuda.synchronize()
    finally:
        gl.gasloc_destroy(ctx)
    for name, buf in (("x", x), ("y", y), ("m", m), ("v", v), ("u", u), ("zp", zp), ("grads", grads)):
        pad = buf[:, P:]
        bits = pad.view(torch.int16) if buf.dtype == torch.bfloat16 else pad.view(torch.int32)
        want = canary16 if buf.dtype == torch.bfloat16 else canary32
        assert bool((bits == want).all()), "%s: row padding written" % name
    tail = mean[P:].view(torch.int16) if dtype == "bf16" else mean[P:].view(torch.int32)
    assert bool((tail == (canary16 if dtype == "bf16" else canary32)).all()), "mean: padding written"
    assert bool(torch.isfinite(x[:, :P].float()).all()) and bool(torch.isfinite(mean[:P].float()).all())


@pytest.mark.parametrize("n,topology,dtype", [(16, "one_peer_exp", "f32"), (40, "two_peer", "bf16")])
def test_long_run_stays_bit_identical(n, topology, dtype):
    # 60 rounds (the phase kernel at n=16, the planned one at n=40), varying
    # local-step counts and the fused last step every other round: the state
    # never drifts from the fp32 oracle by a single bit
    pair = Pair(n, 2_051, topology, dtype, gamma=0.2, precisions=("f32",))
    rng = np.random.default_rng(77)
    for t in range(60):
        H = rng.integers(1, 4, n)
        for h in range(int(H.max()) - 1):
            pair.local_step(active=(H > h).astype(np.uint8))
        if t % 2:
            pair.local_step_gossip_round(t, active=(H == H.max()).astype(np.uint8))
        else:
            pair.local_step(active=(H == H.max()).astype(np.uint8))
            pair.gossip_round(t)
    reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(), "CE after 60 rounds")
    pair.check_state(tag="60 rounds")

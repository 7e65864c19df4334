"""Oracle pins: the numerical round against library optimizers, closed forms
and the paper's special cases (host, no GPU).

* n = 1 reduces to torch.optim.AdamW (+ torch.optim.SGD for the outer step);
* the first AdamW step has a closed form;
* the complete graph with uniform W reduces to DiLoCo (section 3.1), all
  replicas stay bit-identical and the consensus error is exactly 0;
* a doubly stochastic W preserves the replica mean; with mu = gamma = 0 the
  mean moves as xbar_{t+1} = xbar_t + eta gbar_t (App. A);
* gamma = 0 is plain gossip, and every round matches a dense fp64 brute force
  of Eq. 2 built from torch optimizers (tests/bruteforce.py);
* pure gossip (lr = 0) follows the companion-matrix recurrence of the gossip
  lemma, part (iii) (App. A), and random 1-/2-Peer schedules contract the
  consensus error by the factor that Proposition 1 implies.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from tests.bruteforce import run_rounds

HP = dict(lr=4e-3, beta1=0.9, beta2=0.95, eps=1e-8, wd=0.1)


def make_oracle(n, P, topology="ring", precision="f64", eta=0.7, mu=0.9, nesterov=True, gamma=0.1,
                param_dtype="f32", seed=3):
    hp = oracle.OracleHParams(beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"],
                              weight_decay=HP["wd"], outer_lr=eta, outer_momentum=mu,
                              nesterov=nesterov, consensus_momentum=gamma)
    return oracle.Oracle(n, P, hp, topology=topology, seed=seed, precision=precision,
                         param_dtype=param_dtype)


def grads_fn(n, P, seed=100):
    cache = {}

    def g(step):
        if step not in cache:
            rng = np.random.default_rng(seed + step)
            mu_i = np.random.default_rng(seed - 1).standard_normal(n) * 0.1
            cache[step] = (rng.standard_normal((n, P)) + mu_i[:, None]).astype(np.float32)
        return cache[step]

    return g


def close(a, b, rel):
    b = np.asarray(b, dtype=np.float64)
    a = np.asarray(a, dtype=np.float64)
    rms = math.sqrt(float(np.mean(b * b))) if b.size else 0.0
    bad = np.abs(a - b) > rel * np.abs(b) + rel * rms
    assert not bad.any(), "max |a-b| = %g (rms %g), %d bad" % (np.max(np.abs(a - b)), rms, bad.sum())


# --------------------------------------------------------------------------
# AdamW
# --------------------------------------------------------------------------

@pytest.mark.parametrize("precision", ["f32", "f64"])
def test_first_adamw_step_closed_form(precision):
    # k = 1: m = (1-b1) g, v = (1-b2) g^2, so m_hat = g, sqrt(v_hat) = |g|:
    # y1 = y0 (1 - lr wd) - lr g / (|g| + eps)
    n, P = 2, 257
    o = make_oracle(n, P, precision=precision)
    rng = np.random.default_rng(0)
    y0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(y0)
    g = rng.standard_normal((n, P)).astype(np.float32)
    o.local_step(g, HP["lr"])
    lr, wd, eps = HP["lr"], HP["wd"], HP["eps"]
    if precision == "f32":
        lr, wd, eps = (float(np.float32(v)) for v in (lr, wd, eps))
    g64 = g.astype(np.float64)
    expect = y0.astype(np.float64) * (1 - lr * wd) - lr * g64 / (np.abs(g64) + eps)
    close(o.params_f64("y"), expect, 1e-6 if precision == "f32" else 1e-12)


@pytest.mark.parametrize("precision,rel", [("f32", 2e-6), ("f64", 1e-12)])
def test_n1_local_steps_match_torch_adamw(precision, rel):
    P, steps = 300, 25
    o = make_oracle(1, P, precision=precision)
    rng = np.random.default_rng(1)
    y0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(y0)
    tdt = torch.float32 if precision == "f32" else torch.float64
    p = torch.nn.Parameter(torch.tensor(y0, dtype=tdt))
    opt = torch.optim.AdamW([p], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                            weight_decay=HP["wd"])
    for s in range(steps):
        g = (rng.standard_normal((1, P)) + 0.05).astype(np.float32)
        o.local_step(g, HP["lr"])
        p.grad = torch.tensor(g[0], dtype=tdt)
        opt.step()
    close(o.params_f64("y")[0], p.detach().double().numpy(), rel)
    st = opt.state[p]
    close(o.m[0], st["exp_avg"].double().numpy(), rel * 10)
    close(o.v[0], st["exp_avg_sq"].double().numpy(), rel * 10)


def test_inactive_workers_are_untouched_and_keep_their_step_count():
    n, P = 4, 64
    o = make_oracle(n, P, precision="f64")
    o.set_params(np.linspace(-1, 1, P).astype(np.float32))
    g = np.ones((n, P), dtype=np.float32)
    o.local_step(g, HP["lr"], active=[1, 0, 1, 0])
    assert list(o.k) == [1, 0, 1, 0]
    assert np.array_equal(o.y[1], o.x[1]) and np.all(o.m[1] == 0) and np.all(o.v[1] == 0)
    assert not np.array_equal(o.y[0], o.x[0])


# --------------------------------------------------------------------------
# outer optimizer, n = 1
# --------------------------------------------------------------------------

@pytest.mark.parametrize("nesterov,mu", [(True, 0.9), (False, 0.9), (False, 0.0)])
@pytest.mark.parametrize("precision,rel", [("f32", 5e-6), ("f64", 1e-11)])
def test_n1_round_is_adamw_plus_torch_sgd(nesterov, mu, precision, rel):
    # W = [1], gamma = 0: x_{t+1} = OuterOpt(x_t, x_t - y_t) with torch.optim.SGD
    P, rounds, H = 200, 6, 3
    eta = 0.7
    o = make_oracle(1, P, precision=precision, eta=eta, mu=mu, nesterov=nesterov, gamma=0.0)
    rng = np.random.default_rng(2)
    x0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    tdt = torch.float32 if precision == "f32" else torch.float64
    inner = torch.nn.Parameter(torch.tensor(x0, dtype=tdt))
    outer = torch.nn.Parameter(torch.tensor(x0, dtype=tdt))
    adam = torch.optim.AdamW([inner], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                             weight_decay=HP["wd"])
    sgd = torch.optim.SGD([outer], lr=eta, momentum=mu, nesterov=nesterov)
    W1 = (np.array([0, 1], np.int32), np.array([0], np.int32), np.array([1.0], np.float32))
    for t in range(rounds):
        with torch.no_grad():
            inner.copy_(outer)
        for h in range(H):
            g = rng.standard_normal((1, P)).astype(np.float32)
            o.local_step(g, HP["lr"])
            inner.grad = torch.tensor(g[0], dtype=tdt)
            adam.step()
        outer.grad = (outer - inner).detach().clone()
        sgd.step()
        o.gossip_round(t, csr=W1)
        close(o.params_f64("x")[0], outer.detach().double().numpy(), rel)
    if mu > 0:
        close(o.u[0], sgd.state[outer]["momentum_buffer"].double().numpy(), rel * 10)


# --------------------------------------------------------------------------
# special cases of the graph
# --------------------------------------------------------------------------

@pytest.mark.parametrize("precision", ["f32", "f64"])
def test_complete_graph_is_diloco(precision):
    # Lambda = pi recovers DiLoCo (section 3.1): every row of W is the same,
    # so the replicas stay bit-identical and the consensus error is exactly 0.
    n, P, rounds, H = 5, 128, 4, 2
    eta, mu = 0.7, 0.9
    o = make_oracle(n, P, topology="complete", precision=precision, eta=eta, mu=mu, gamma=0.0)
    rng = np.random.default_rng(4)
    x0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    g = grads_fn(n, P)
    # DiLoCo: H AdamW steps per worker, outer Nesterov on the averaged pseudo-gradient
    tdt = torch.float64
    inner = [torch.nn.Parameter(torch.tensor(x0, dtype=tdt)) for _ in range(n)]
    adam = [torch.optim.AdamW([p], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                              weight_decay=HP["wd"]) for p in inner]
    outer = torch.nn.Parameter(torch.tensor(x0, dtype=tdt))
    sgd = torch.optim.SGD([outer], lr=eta, momentum=mu, nesterov=True)
    step = 0
    for t in range(rounds):
        for i in range(n):
            with torch.no_grad():
                inner[i].copy_(outer)
        for h in range(H):
            gs = g(step)
            step += 1
            o.local_step(gs, HP["lr"])
            for i in range(n):
                inner[i].grad = torch.tensor(gs[i], dtype=tdt)
                adam[i].step()
        outer.grad = torch.stack([(outer - inner[i]).detach() for i in range(n)]).mean(0)
        sgd.step()
        o.gossip_round(t)
        x = o.params_f64("x")
        assert np.all(x == x[0]), "replicas must be bit-identical"
        if precision == "f32":
            # fp32 values: the fp64 mean of identical entries is exact
            assert o.consensus_error() == 0.0
        else:
            assert o.consensus_error() <= 1e-28
        close(x[0], outer.detach().numpy(), 1e-5 if precision == "f32" else 1e-11)


def test_parameter_averaging_when_eta1_no_momentum():
    # complete graph, eta = 1, mu = gamma = 0: x_{t+1} = mean_i y_i (Local SGD)
    n, P = 4, 96
    o = make_oracle(n, P, topology="complete", precision="f64", eta=1.0, mu=0.0, gamma=0.0)
    o.set_params(np.zeros(P, np.float32))
    g = grads_fn(n, P)(0)
    o.local_step(g, HP["lr"])
    y = o.params_f64("y").copy()
    o.gossip_round(0)
    close(o.params_f64("x"), np.tile(y.mean(axis=0), (n, 1)), 1e-12)


DOUBLY_STOCHASTIC = ["ring", "exponential", "one_peer_exp", "one_peer", "two_peer", "random_regular",
                     "complete"]


@pytest.mark.parametrize("kind", DOUBLY_STOCHASTIC)
def test_doubly_stochastic_mix_preserves_the_mean(kind):
    n, P, rounds = 8, 64, 3
    a = make_oracle(n, P, topology=kind, precision="f64", gamma=0.3)
    ident = (np.arange(n + 1, dtype=np.int32), np.arange(n, dtype=np.int32), np.ones(n, np.float32))
    b = make_oracle(n, P, topology=kind, precision="f64", gamma=0.3)
    rng = np.random.default_rng(6)
    x0 = (rng.standard_normal((n, P)) * 0.02)
    a.x[...] = x0
    a.y[...] = x0
    b.x[...] = x0
    b.y[...] = x0
    g = grads_fn(n, P)
    for t in range(rounds):
        a.local_step(g(t), HP["lr"])
        b.local_step(g(t), HP["lr"])
        a.gossip_round(t)
        b.gossip_round(t, csr=ident)
        # fp32 weights: rows/columns sum to 1 within ~1e-7
        close(a.x.mean(axis=0), b.x.mean(axis=0), 1e-6)


def test_mean_dynamics_sgd_outer_step():
    # mu = gamma = 0 and doubly stochastic W: xbar_{t+1} = xbar_t + eta gbar_t (App. A)
    n, P, eta = 6, 80, 0.7
    o = make_oracle(n, P, topology="two_peer", precision="f64", eta=eta, mu=0.0, gamma=0.0)
    o.set_params((np.random.default_rng(7).standard_normal(P) * 0.02).astype(np.float32))
    g = grads_fn(n, P)
    for t in range(4):
        xbar = o.x.mean(axis=0).copy()
        o.local_step(g(2 * t), HP["lr"])
        o.local_step(g(2 * t + 1), HP["lr"])
        gbar = (o.y - o.x).mean(axis=0)  # g_t = x_{t,H} - x_{t,0} (Eq. 1)
        o.gossip_round(t)
        close(o.x.mean(axis=0), xbar + eta * gbar, 1e-6)


# --------------------------------------------------------------------------
# whole rounds against the dense brute force
# --------------------------------------------------------------------------

CASES = [
    ("ring", 4, 1, 0.1, 0.9, True),
    ("exponential", 8, 1, 0.1, 0.9, True),
    ("one_peer_exp", 8, 3, 0.1, 0.9, True),
    ("random_regular", 8, 2, 0.1, 0.5, False),
    ("one_peer", 5, 2, 0.0, 0.9, True),
    ("two_peer", 7, 2, 0.2, 0.0, False),
    ("complete", 3, 2, 0.3, 0.9, True),
]


@pytest.mark.parametrize("kind,n,H,gamma,mu,nesterov", CASES)
@pytest.mark.parametrize("precision,rel", [("f64", 1e-10), ("f32", 1e-5)])
def test_rounds_match_dense_bruteforce(kind, n, H, gamma, mu, nesterov, precision, rel):
    P, rounds, eta = 48, 4, 0.7
    o = make_oracle(n, P, topology=kind, precision=precision, eta=eta, mu=mu, nesterov=nesterov,
                    gamma=gamma)
    rng = np.random.default_rng(8)
    x0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    H_i = np.full(n, H)
    if kind == "one_peer":
        H_i = np.array([H, 0, 1, H, 2])[:n]  # heterogeneous local steps, one idle worker
    g = grads_fn(n, P)
    step = 0
    ces = []
    for t in range(rounds):
        for h in range(int(H_i.max())):
            o.local_step(g(step), HP["lr"], active=(H_i > h).astype(np.uint8))
            step += 1
        o.gossip_round(t)
        ces.append(o.consensus_error())
    W_of_round = lambda t: oracle.csr_to_dense(*o.csr(t), n)  # noqa: E731
    x_b, _, u_b, zp_b, ce_b = run_rounds(np.tile(x0.astype(np.float64), (n, 1)), g, W_of_round, H_i,
                                         rounds, HP["lr"], HP["beta1"], HP["beta2"], HP["eps"],
                                         HP["wd"], eta, mu, nesterov, gamma)
    close(o.params_f64("x"), x_b, rel)
    if mu > 0:
        close(o.u, u_b, rel)
    if gamma != 0:
        close(o.zp, zp_b, rel)
    close(ces, ce_b, rel * 10)


def test_bf16_storage_rounds_like_torch():
    # round-to-nearest-even binary32 -> bfloat16, including ties and specials
    rng = np.random.default_rng(9)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(0.02),
        rng.standard_normal(2000).astype(np.float32) * np.float32(1e30),
        np.array([0.0, -0.0, 1.0, np.inf, -np.inf, 3.3895314e38, 1.00390625, 1.01171875, 1e-40],
                 dtype=np.float32),
    ])
    ours = oracle.f32_to_bf16_bits(vals)
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    nan_bits = oracle.f32_to_bf16_bits(np.array([np.nan], dtype=np.float32))
    assert np.isnan(oracle.bf16_bits_to_f32(nan_bits))[0]


def test_bf16_storage_is_rne_of_the_fp32_result():
    # bf16 parameters (fp32 state and arithmetic): each store is the RNE
    # rounding of the value the fp32-storage oracle computes from the same inputs
    n, P = 4, 256
    ob = make_oracle(n, P, topology="ring", precision="f32", param_dtype="bf16")
    of = make_oracle(n, P, topology="ring", precision="f32", param_dtype="f32")
    x0_bits = oracle.f32_to_bf16_bits(
        (np.random.default_rng(10).standard_normal(P) * 0.02).astype(np.float32))
    ob.set_params(x0_bits)
    of.set_params(oracle.bf16_bits_to_f32(x0_bits))
    g = grads_fn(n, P)
    for t in range(3):
        ob.local_step(g(t), HP["lr"])
        of.local_step(g(t), HP["lr"])
        assert np.array_equal(ob.y, oracle.f32_to_bf16_bits(of.y))
        assert np.array_equal(ob.m, of.m) and np.array_equal(ob.v, of.v)
        of.y[...] = oracle.bf16_bits_to_f32(ob.y)
        ob.gossip_round(t)
        of.gossip_round(t)
        assert np.array_equal(ob.x, oracle.f32_to_bf16_bits(of.x))
        assert np.array_equal(ob.u, of.u) and np.array_equal(ob.zp, of.zp)
        of.x[...] = oracle.bf16_bits_to_f32(ob.x)
        of.y[...] = of.x


# --------------------------------------------------------------------------
# consensus error and pure gossip
# --------------------------------------------------------------------------

def test_consensus_error_definition():
    n, P = 6, 100
    o = make_oracle(n, P, precision="f64")
    x = np.random.default_rng(11).standard_normal((n, P))
    o.x[...] = x
    assert o.consensus_error() == pytest.approx(float((x.var(axis=0) * n).sum()), rel=1e-13)
    c = np.array([1.0, 2.0, 3.0, 4.0, 5.0, 9.0])
    o.x[...] = c[:, None]
    assert o.consensus_error() == P * float(((c - c.mean()) ** 2).sum())
    o.x[...] = 0.25
    assert o.consensus_error() == 0.0
    np.testing.assert_allclose(o.replica_mean(), 0.25)


@pytest.mark.parametrize("precision,param_dtype", [("f64", "f32"), ("f32", "f32"), ("f32", "bf16")])
def test_replica_mean_is_the_network_average(precision, param_dtype):
    # Algorithm 1's output: the average of the n replicas, rounded once to the
    # parameter storage (numpy's fp64 mean, then the storage rounding)
    n, P = 7, 3000
    rng = np.random.default_rng(12)
    o = make_oracle(n, P, precision=precision, param_dtype=param_dtype)
    x = rng.standard_normal((n, P)) * 0.3 + rng.standard_normal(P) * 2.0
    if param_dtype == "bf16":
        o.x[...] = oracle.f32_to_bf16_bits(x.astype(np.float32))
        xs = oracle.bf16_bits_to_f32(o.x).astype(np.float64)
        expect = oracle.f32_to_bf16_bits(np.mean(xs, axis=0).astype(np.float32))
        assert np.array_equal(o.replica_mean(), expect)
    else:
        o.x[...] = x.astype(o.real)
        expect = np.mean(o.x.astype(np.float64), axis=0).astype(o.real)
        got = o.replica_mean()
        if precision == "f64":
            np.testing.assert_allclose(got, expect, rtol=1e-15, atol=1e-15)
        else:
            assert np.array_equal(got.view(np.uint32), expect.view(np.uint32))


def _pure_gossip_oracle(n, P, csr, gamma, x):
    o = make_oracle(n, P, precision="f64", gamma=gamma)
    o.x[...] = x
    o.y[...] = x
    return o


def test_pure_gossip_static_w_matches_companion_matrix():
    # lr = 0 leaves y = x, so z = x and X_{t+1} = (W + gamma I) X_t - gamma X_{t-1}
    # (gossip lemma (iii), App. A) with X_{-1} = X_0 (no gamma term in round 0).
    n, P, gamma, rounds = 4, 32, 0.25, 50
    csr = oracle.topology_csr("ring", n, 0, 0)
    W = oracle.csr_to_dense(*csr, n)
    x = np.random.default_rng(12).standard_normal((n, P))
    o = _pure_gossip_oracle(n, P, csr, gamma, x)
    M = np.block([[W + gamma * np.eye(n), -gamma * np.eye(n)], [np.eye(n), np.zeros((n, n))]])
    pi = np.eye(n) - np.ones((n, n)) / n
    state = np.vstack([W @ x, x])  # after round 0 (no momentum term yet)
    zeros = np.zeros((n, P), np.float32)
    ce0 = o.consensus_error()
    for t in range(rounds):
        o.local_step(zeros, 0.0)
        o.gossip_round(t, csr=csr)
        if t > 0:
            state = M @ state
        expect = float(((pi @ state[:n]) ** 2).sum())
        # fp64 rounding of the O(1) initial state bounds the absolute error
        assert o.consensus_error() == pytest.approx(expect, rel=1e-5, abs=1e-20 * ce0)


def test_accelerated_gossip_rate_bound():
    # gossip lemma (iii): gamma = (1 - sqrt(alpha/chi))^2 gives a contraction
    # rate of at most q = 1 - sqrt(alpha/chi) per round on the disagreement.
    n, P = 12, 8
    alpha = 1.0
    edges = [(i, (i + 1) % n) for i in range(n)]
    from tests.bruteforce import laplacian

    Lam = laplacian(n, edges, [0.5] * n)  # eigenvalues in (0, 1]
    W = np.eye(n) - alpha * Lam
    lam = np.sort(np.linalg.eigvalsh(Lam))
    chi = 1.0 / lam[1]
    q = 1 - math.sqrt(alpha / chi)
    gamma = q * q
    row_ptr = [0]
    col, val = [], []
    for i in range(n):
        for j in range(n):
            if W[i, j] != 0:
                col.append(j)
                val.append(W[i, j])
        row_ptr.append(len(col))
    csr = (np.array(row_ptr, np.int32), np.array(col, np.int32), np.array(val, np.float32))
    x = np.random.default_rng(13).standard_normal((n, P))
    o = _pure_gossip_oracle(n, P, csr, gamma, x)
    zeros = np.zeros((n, P), np.float32)
    ce0 = o.consensus_error()
    T = 120
    for t in range(T):
        o.local_step(zeros, 0.0)
        o.gossip_round(t, csr=csr)
    ce = o.consensus_error()
    # ||pi x_T|| <= C q^T: allow a polynomial prefactor for the defective
    # double root at lambda_min (the bound holds in an equivalent norm)
    assert math.sqrt(ce / ce0) <= 4 * (T + 1) * q ** T
    # without the momentum term the contraction is only 1 - alpha/chi per round
    assert q < 1 - alpha / chi


@pytest.mark.parametrize("kind,f", [
    ("one_peer", lambda n: (n - 2) / (2 * (n - 1))),
    ("two_peer", lambda n: 1 - 2 * n / (3 * (n - 1))),
])
def test_random_schedule_expected_contraction(kind, f):
    # E[CE_{t+1} | x_t] = (1 - 2 alpha c1 + alpha^2 c2) CE_t with c1, c2 from
    # Proposition 1 (section 3.2); alpha = 1 for 1-Peer weights 1/2, 4/3 for
    # uniform 1/3 2-Peer weights.
    n, P, trials = 8, 4, 4000
    x = np.random.default_rng(14).standard_normal((n, P))
    ratios = []
    zeros = np.zeros((n, P), np.float32)
    for t in range(trials):
        o = make_oracle(n, P, topology=kind, precision="f64", mu=0.0, gamma=0.0, seed=21)
        o.x[...] = x
        o.y[...] = x
        ce0 = o.consensus_error()
        o.local_step(zeros, 0.0)
        o.gossip_round(t)
        ratios.append(o.consensus_error() / ce0)
    ratios = np.array(ratios)
    se = ratios.std() / math.sqrt(trials)
    assert abs(ratios.mean() - f(n)) < 4 * se + 1e-12

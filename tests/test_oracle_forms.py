"""Oracle pins for the other round forms (host, no GPU).

* Algorithm 1: the outer optimizer receives the neighbourhood average of
  (x_i - y_j).  On the complete graph it is DiLoCo (section 3.1); with
  eta = 1, mu = 0 it mixes the local iterates, x <- W y; with a doubly
  stochastic W the mean moves by -eta (xbar - ybar); multi-round agreement
  with torch AdamW/SGD and the dense matrix form.
* DAdam (App. C): x <- W x + (y - x) as a dense matmul; the mean becomes
  the mean of y for doubly stochastic W.
* Local-DAdam (App. C): OuterOpt(y_i, sum_j w_ij (x_i - x_j)) against torch
  SGD; with unit outer lr and no momentum it reduces to DAdam (App. C).
"""
import numpy as np
import pytest
import torch

import oracle
from tests.test_oracle_round import HP, close, grads_fn


def make(n, P, topology, form, precision="f64", eta=0.7, mu=0.9, nesterov=True):
    hp = oracle.OracleHParams(beta1=HP["beta1"], beta2=HP["beta2"], eps=HP["eps"], weight_decay=HP["wd"],
                              outer_lr=eta, outer_momentum=mu, nesterov=nesterov, consensus_momentum=0.0,
                              form=form)
    return oracle.Oracle(n, P, hp, topology=topology, seed=3, precision=precision)


def adam_opts(params):
    return [torch.optim.AdamW([p], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                              weight_decay=HP["wd"]) for p in params]


def brute(form, n, P, x0, g, W_of_round, H, rounds, eta, mu, nesterov):
    """Dense fp64 reference built from torch optimizers and matrix algebra."""
    x = np.tile(x0.astype(np.float64), (n, 1))
    inner = [torch.nn.Parameter(torch.zeros(P, dtype=torch.float64)) for _ in range(n)]
    outer = [torch.nn.Parameter(torch.zeros(P, dtype=torch.float64)) for _ in range(n)]
    adam = adam_opts(inner)
    sgd = [torch.optim.SGD([outer[i]], lr=eta, momentum=mu, nesterov=nesterov and mu > 0) for i in range(n)]
    step = 0
    for t in range(rounds):
        for i in range(n):
            with torch.no_grad():
                inner[i].copy_(torch.from_numpy(x[i]))
        for h in range(H):
            gs = g(step)
            step += 1
            for i in range(n):
                inner[i].grad = torch.from_numpy(gs[i].astype(np.float64))
                adam[i].step()
        y = np.stack([p.detach().numpy().copy() for p in inner])
        W = W_of_round(t)
        new = np.empty_like(x)
        if form == "alg1":
            delta = x - W @ y
            base = x
        elif form == "local_dadam":
            delta = x - W @ x
            base = y
        else:  # dadam
            new = W @ x + (y - x)
        if form != "dadam":
            for i in range(n):
                with torch.no_grad():
                    outer[i].copy_(torch.from_numpy(base[i]))
                outer[i].grad = torch.from_numpy(delta[i].copy())
                sgd[i].step()
                new[i] = outer[i].detach().numpy()
        x = new
    return x


def run_oracle(o, g, H, rounds, ces=None):
    step = 0
    for t in range(rounds):
        for h in range(H):
            o.local_step(g(step), HP["lr"])
            step += 1
        o.gossip_round(t)
        if ces is not None:
            ces.append(o.consensus_error())


CASES = [("ring", 4, 1), ("exponential", 8, 2), ("two_peer", 7, 1), ("one_peer", 6, 3),
         ("random_regular", 8, 2)]


@pytest.mark.parametrize("form", ["alg1", "dadam", "local_dadam"])
@pytest.mark.parametrize("kind,n,H", CASES)
@pytest.mark.parametrize("precision,rel", [("f64", 1e-10), ("f32", 1e-5)])
def test_forms_match_dense_bruteforce(form, kind, n, H, precision, rel):
    P, rounds, eta, mu = 40, 3, 0.7, 0.9
    o = make(n, P, kind, form, precision, eta, mu)
    x0 = (np.random.default_rng(20).standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    g = grads_fn(n, P, seed=300)
    run_oracle(o, g, H, rounds)
    ref = brute(form, n, P, x0, g, lambda t: oracle.csr_to_dense(*o.csr(t), n), H, rounds, eta, mu, True)
    close(o.params_f64("x"), ref, rel)


@pytest.mark.parametrize("precision", ["f32", "f64"])
def test_alg1_complete_graph_is_diloco(precision):
    n, P, rounds, H, eta, mu = 5, 64, 3, 2, 0.7, 0.9
    o = make(n, P, "complete", "alg1", precision, eta, mu)
    x0 = (np.random.default_rng(21).standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    g = grads_fn(n, P, seed=310)
    inner = [torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64)) for _ in range(n)]
    adam = adam_opts(inner)
    outer = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    sgd = torch.optim.SGD([outer], lr=eta, momentum=mu, nesterov=True)
    step = 0
    for t in range(rounds):
        for p in inner:
            with torch.no_grad():
                p.copy_(outer)
        for h in range(H):
            gs = g(step)
            step += 1
            o.local_step(gs, HP["lr"])
            for i in range(n):
                inner[i].grad = torch.tensor(gs[i], dtype=torch.float64)
                adam[i].step()
        outer.grad = torch.stack([(outer - p).detach() for p in inner]).mean(0)
        sgd.step()
        o.gossip_round(t)
        x = o.params_f64("x")
        assert np.all(x == x[0]), "the same row of W keeps the replicas identical"
        if precision == "f32":
            assert o.consensus_error() == 0.0
        close(x[0], outer.detach().numpy(), 1e-5 if precision == "f32" else 1e-11)


def test_alg1_unit_outer_step_mixes_the_local_iterates():
    # eta = 1, mu = 0: x_i - sum_j W_ij (x_i - y_j) = sum_j W_ij y_j
    n, P = 6, 50
    o = make(n, P, "two_peer", "alg1", "f64", eta=1.0, mu=0.0)
    o.set_params((np.random.default_rng(22).standard_normal(P) * 0.02).astype(np.float32))
    o.local_step(grads_fn(n, P, seed=320)(0), HP["lr"])
    y = o.params_f64("y").copy()
    o.gossip_round(0)
    W = oracle.csr_to_dense(*o.csr(0), n)
    close(o.params_f64("x"), W @ y, 1e-12)


@pytest.mark.parametrize("form", ["alg1", "dadam"])
def test_mean_dynamics_of_the_forms(form):
    # doubly stochastic W, mu = 0:
    #   Algorithm 1: xbar <- xbar - eta (xbar - ybar);  DAdam: xbar <- ybar
    n, P, eta = 8, 60, 0.7
    o = make(n, P, "random_regular", form, "f64", eta=eta, mu=0.0)
    rng = np.random.default_rng(23)
    x0 = rng.standard_normal((n, P)) * 0.02
    o.x[...] = x0
    o.y[...] = x0
    g = grads_fn(n, P, seed=330)
    for t in range(3):
        xbar = o.x.mean(axis=0).copy()
        o.local_step(g(t), HP["lr"])
        ybar = o.y.mean(axis=0).copy()
        o.gossip_round(t)
        expect = xbar - eta * (xbar - ybar) if form == "alg1" else ybar
        close(o.x.mean(axis=0), expect, 1e-12)


def test_local_dadam_unit_sgd_is_dadam():
    # App. C: with H = 1 and a unit-lr SGD outer step Local-DAdam is DAdam
    n, P = 7, 45
    a = make(n, P, "two_peer", "local_dadam", "f64", eta=1.0, mu=0.0)
    b = make(n, P, "two_peer", "dadam", "f64")
    rng = np.random.default_rng(24)
    x0 = rng.standard_normal((n, P)) * 0.02
    for o in (a, b):
        o.x[...] = x0
        o.y[...] = x0
    g = grads_fn(n, P, seed=340)
    for t in range(4):
        a.local_step(g(t), HP["lr"])
        b.local_step(g(t), HP["lr"])
        a.gossip_round(t)
        b.gossip_round(t)
        close(a.x, b.x, 1e-12)


def test_local_dadam_without_neighbours_keeps_the_local_iterate():
    # W = I: the disagreement is 0, so with mu = 0 the new anchor is y exactly
    n, P = 3, 30
    o = make(n, P, "ring", "local_dadam", "f32", eta=0.7, mu=0.0)
    o.set_params((np.random.default_rng(25).standard_normal(P) * 0.02).astype(np.float32))
    ident = (np.arange(n + 1, dtype=np.int32), np.arange(n, dtype=np.int32), np.ones(n, np.float32))
    o.local_step(grads_fn(n, P, seed=350)(0), HP["lr"])
    y = o.y.copy()
    o.gossip_round(0, csr=ident)
    assert np.array_equal(o.x, y)

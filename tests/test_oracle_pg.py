"""Oracle pins for the pseudo-gradient statistic sum_i ||x_i - y_i||^2 (the
squared norms of Eq. 1's pseudo-gradients g = x_{t,H} - x_{t,0}) (host, no GPU).

* after one AdamW step from x (k = 1) the step has the closed form
  y = x (1 - lr wd) - lr g / (|g| + eps), so the statistic is the fp64 sum of
  (x lr wd + lr g / (|g| + eps))^2;
* a worker without local steps contributes nothing; after a round the live
  iterate is the new anchor, so the statistic is 0 again;
* identical workers with identical gradients contribute identical terms;
* the value a round consumed is the one measured just before it.
"""
import numpy as np
import pytest

import oracle
from tests.test_oracle_round import HP, make_oracle


def closed_form_first_step(x0, g):
    x = x0.astype(np.float64)
    gd = g.astype(np.float64)
    d = x * HP["lr"] * HP["wd"] + HP["lr"] * gd / (np.abs(gd) + HP["eps"])
    return float(np.sum(d * d))


@pytest.mark.parametrize("precision,rel", [("f64", 1e-12), ("f32", 2e-6)])
def test_first_step_closed_form(precision, rel):
    n, P = 3, 5000
    rng = np.random.default_rng(4)
    o = make_oracle(n, P, precision=precision)
    x0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    g = rng.standard_normal((n, P)).astype(np.float32) + np.array([[0.3], [-0.1], [0.0]], np.float32)
    assert o.pseudo_gradient_sq() == 0.0
    o.local_step(g, HP["lr"])
    expect = sum(closed_form_first_step(x0, g[i]) for i in range(n))
    got = o.pseudo_gradient_sq()
    assert abs(got - expect) <= rel * expect, (got, expect)
    # per worker and on a column subset
    cols = np.arange(7, P, 3)
    sub = sum(closed_form_first_step(x0[cols], g[i][cols]) for i in range(n))
    assert abs(o.pseudo_gradient_sq(cols) - sub) <= rel * sub


def test_inactive_workers_contribute_nothing_and_rounds_reset_it():
    n, P = 6, 400
    rng = np.random.default_rng(5)
    o = make_oracle(n, P, topology="two_peer", precision="f64")
    x0 = rng.standard_normal(P) * 0.02
    o.set_params(x0)
    g = rng.standard_normal((n, P)).astype(np.float32)
    active = np.array([1, 0, 1, 0, 0, 1], np.uint8)
    o.local_step(g, HP["lr"], active)
    expect = sum(closed_form_first_step(x0, g[i]) for i in range(n) if active[i])
    got = o.pseudo_gradient_sq()
    assert abs(got - expect) <= 1e-12 * expect
    before = o.pseudo_gradient_sq()
    o.gossip_round(0)
    assert o.pg_last == before
    assert o.pseudo_gradient_sq() == 0.0


def test_identical_workers_give_identical_terms():
    n, P = 5, 2000
    rng = np.random.default_rng(6)
    single = make_oracle(1, P, precision="f32")
    many = make_oracle(n, P, precision="f32")
    x0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    single.set_params(x0)
    many.set_params(x0)
    g1 = rng.standard_normal((1, P)).astype(np.float32)
    for _ in range(3):
        single.local_step(g1, HP["lr"])
        many.local_step(np.repeat(g1, n, axis=0), HP["lr"])
    s = single.pseudo_gradient_sq()
    assert s > 0
    assert abs(many.pseudo_gradient_sq() - n * s) <= 1e-12 * n * s  # fp64 summation order only


def test_bf16_storage_uses_the_stored_values():
    n, P = 2, 3000
    rng = np.random.default_rng(7)
    o = make_oracle(n, P, precision="f32", param_dtype="bf16")
    x0 = (rng.standard_normal(P) * 0.02).astype(np.float32)
    o.set_params(x0)
    o.local_step(rng.standard_normal((n, P)).astype(np.float32), HP["lr"])
    x = oracle.bf16_bits_to_f32(o.x).astype(np.float32)
    y = oracle.bf16_bits_to_f32(o.y).astype(np.float32)
    d = (x - y).astype(np.float64)  # exact: both are bf16 values, their fp32 difference is exact here
    assert o.pseudo_gradient_sq() == pytest.approx(float(np.sum(d * d)), rel=1e-12)

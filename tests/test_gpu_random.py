"""GPU parity on seeded random configurations: worker count, row length
(ragged tails), graph, round form, parameter dtype, outer and consensus
momentum, per-worker local-step counts that change every round, and the
fused or the split last step, all drawn from one seeded generator.  Every
case must stay bit-identical to the fp32 oracle."""
import numpy as np
import pytest

from tests.gpu_harness import Pair, log, reduction_close

pytestmark = pytest.mark.gpu

KINDS = ["ring", "complete", "exponential", "one_peer_exp", "one_peer", "two_peer", "random_regular"]
FORMS = ["eq", "eq", "eq", "alg1", "dadam", "local_dadam"]
CASES = 96


def draw(case):
    rng = np.random.default_rng(9000 + case)
    n = int(rng.choice([1, 2, 3, 5, 8, 12, 16, 17, 24, 33, 40, 64]))
    kind = str(rng.choice(KINDS))
    if kind == "random_regular" and (n < 4 or (3 * n) % 2):
        kind = "two_peer"
    form = str(rng.choice(FORMS))
    return dict(n=n, P=int(rng.integers(1, 20_000)), topology=kind, form=form,
                dtype=str(rng.choice(["f32", "bf16"])),
                gamma=float(rng.choice([0.0, 0.1, 0.3])) if form == "eq" else 0.0,
                mu=float(rng.choice([0.0, 0.5, 0.9])), nesterov=bool(rng.integers(2)),
                seed=int(rng.integers(1 << 30)))


@pytest.mark.parametrize("case", range(CASES))
def test_random_configuration(case):
    cfg = draw(case)
    log("case %d: %s" % (case, cfg))
    rng = np.random.default_rng(cfg.pop("seed"))
    n = cfg["n"]
    pair = Pair(cfg["n"], cfg["P"], cfg["topology"], cfg["dtype"], gamma=cfg["gamma"], mu=cfg["mu"],
                nesterov=cfg["nesterov"], form=cfg["form"], precisions=("f32",))
    for t in range(3):
        H = rng.integers(0, 4, n)
        hmax = int(H.max())
        fused = cfg["form"] in ("eq", "alg1") and hmax > 0 and bool(rng.integers(2))
        last = hmax - 1 if fused else hmax
        for h in range(last):
            pair.local_step(active=(H > h).astype(np.uint8))
        if fused:
            pair.local_step_gossip_round(t, active=(H > last).astype(np.uint8))
        else:
            pair.gossip_round(t)
        reduction_close(pair.gpu.consensus_error(), pair.oracles["f32"].consensus_error(),
                        "case %d round %d consensus error" % (case, t))
    stats = pair.check_state(tag="random case %d" % case)
    log("bit-exact fraction vs fp32 oracle: %s" % stats)

"""Oracle pins: SplitMix64, bounded draws, Fisher-Yates (host, no GPU)."""
import itertools
import math

import numpy as np
import pytest

import oracle


def _kat(golden_dir):
    rows = []
    with open(golden_dir + "/splitmix64_kat.txt") as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                vals = [int(v) for v in line.split()]
                rows.append((vals[0], vals[1:]))
    return rows


@pytest.mark.parametrize("precision", ["f32", "f64"])
def test_splitmix64_known_answers(golden_dir, precision):
    for seed, expected in _kat(golden_dir):
        assert oracle.splitmix64_stream(seed, len(expected), precision) == expected


def test_bounded_range_and_uniformity():
    state = oracle.round_state(7, 0)
    for k in (1, 2, 3, 5, 7, 64, 96):
        draws = np.array(oracle.bounded_draws(state, k, 6000))
        assert draws.min() >= 0 and draws.max() < k
        if k > 1:
            counts = np.bincount(draws, minlength=k)
            expected = len(draws) / k
            chi2 = ((counts - expected) ** 2 / expected).sum()
            # chi-square with k-1 dof: mean k-1, sd sqrt(2(k-1)); 6 sd is a generous bound
            assert chi2 < (k - 1) + 6 * math.sqrt(2 * (k - 1))


def test_bounded_rejects_only_the_biased_tail():
    # k = 2^63 + 1: the rejection threshold 2^64 mod k = 2^63 - 1 is huge, so
    # accepted raw draws r satisfy r >= 2^63 - 1 and the result is r - k or r mod k.
    k = (1 << 63) + 1
    state = oracle.round_state(11, 3)
    draws = oracle.bounded_draws(state, k, 200)
    assert all(0 <= d < k for d in draws)


def test_shuffle_is_a_uniform_permutation():
    perms = {}
    trials = 24000
    for t in range(trials):
        p = tuple(oracle.shuffled_identity(oracle.round_state(5, t), 4))
        assert sorted(p) == [0, 1, 2, 3]
        perms[p] = perms.get(p, 0) + 1
    assert set(perms) == set(itertools.permutations(range(4)))
    expected = trials / 24
    chi2 = sum((c - expected) ** 2 / expected for c in perms.values())
    assert chi2 < 23 + 6 * math.sqrt(46)


def test_round_state_depends_on_seed_and_round():
    states = {oracle.round_state(s, t) for s in range(8) for t in range(64)}
    assert len(states) == 8 * 64

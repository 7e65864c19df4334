"""Oracle pins for the learning-rate schedule of App. B "Optimization":
10% warmup starting at 1% of the peak, then cosine decay."""
import math

import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("total", [10, 100, 1000, 2569])
def test_schedule_shape(total):
    peak = 4e-3
    lrs = np.array([oracle.lr_schedule(peak, s, total) for s in range(total + 1)], dtype=np.float64)
    W = int(math.floor(0.1 * total))
    f32 = lambda v: float(np.float32(v))  # noqa: E731
    assert lrs[0] == f32(0.01 * peak), "warmup starts at 1% of the peak"
    assert lrs[W] == f32(peak), "the peak is reached when warmup ends"
    assert lrs[total] == 0.0, "cosine decay ends at final_frac * peak = 0"
    assert np.all(np.diff(lrs[: W + 1]) > 0), "warmup increases"
    assert np.all(np.diff(lrs[W:]) <= 0), "decay does not increase"
    assert abs(lrs[:W].size - 0.1 * total) < 1, "warmup covers 10% of the steps"
    if (total - W) % 2 == 0:  # the cosine midpoint is half the peak
        assert lrs[W + (total - W) // 2] == pytest.approx(peak / 2, rel=1e-6)


def test_schedule_warmup_is_linear_and_final_fraction():
    total, peak = 200, 1.0
    W = 20
    for s in range(W):
        assert oracle.lr_schedule(peak, s, total) == pytest.approx(0.01 + 0.99 * s / W, rel=1e-6)
    assert oracle.lr_schedule(peak, total, total, final_frac=0.1) == pytest.approx(0.1, rel=1e-6)
    # clamps outside [0, total]
    assert oracle.lr_schedule(peak, -5, total) == oracle.lr_schedule(peak, 0, total)
    assert oracle.lr_schedule(peak, total + 9, total) == oracle.lr_schedule(peak, total, total)

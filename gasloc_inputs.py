"""Seeded synthetic inputs and workload shapes for the GASLoC gossip round.

This module is shared by the GPU-side callers (tests, bench) and the oracle
side; it holds none of the method's arithmetic, only what the inputs are:

  * workload shapes: worker count n, parameter count P (synthetic replicas
    sized like the paper's 134M / 551M Llama models, App. B Table 4), the
    communication graph, local steps H, consensus momentum gamma;
  * hyperparameters of App. B "Optimization" (AdamW weight decay 0.1,
    betas (0.9, 0.95), local lr inside the swept 1e-3..8e-3 range) and the
    outer Nesterov step (outer lr / momentum inside the swept grids);
  * seeded generators: initial parameters x0 ~ N(0, 0.02^2) shared by every
    worker (identical initialisation), per-worker gradient means
    mu_i ~ N(0, 0.1^2), per-step gradients g = mu_i + N(0, 1) standing in
    for backpropagated gradients, and per-worker local-step counts H_i.

The paper trains on FineWeb; no dataset is used here.  Gradients are drawn
with torch's generator on the device the caller asks for (CPU for host-only
tests, the GPU for device runs); when both sides need the same bits, the
device tensor is copied (or its sampled columns gathered) to the host.
"""
from dataclasses import dataclass, field

import numpy as np

LOCAL_LR = 4e-3
BETA1, BETA2 = 0.9, 0.95
EPS = 1e-8
WEIGHT_DECAY = 0.1
OUTER_LR = 0.7
OUTER_MOMENTUM = 0.9

SEED_X0 = 0
SEED_MU = 1
SEED_GRAD_BASE = 2  # gradients of global local-step s use seed SEED_GRAD_BASE + s
SEED_TOPOLOGY = 3
SEED_H = 4


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    P: int
    topology: str
    param_dtype: str  # "f32" or "bf16"; optimizer state is always fp32
    H: int  # local steps per round (upper end when heterogeneous)
    gamma: float
    rounds: int  # rounds used by the parity tests
    degree: int = 3  # random_regular only
    hetero_H: tuple = field(default=None)  # (lo, hi) inclusive: H_i ~ U{lo..hi}
    description: str = ""


WORKLOADS = {
    "ring-n4-p1m": Workload(
        "ring-n4-p1m", 4, 1_048_576, "ring", "f32", 1, 0.1, 10,
        description="n=4 static ring (weights 1/3), P=1,048,576 fp32, H=1, 10 rounds"),
    "exp-n8-p124m": Workload(
        "exp-n8-p124m", 8, 124_000_000, "exponential", "f32", 1, 0.1, 10,
        description="n=8 static exponential graph (hops 1,2,4; weights 1/4), P=124M fp32, H=1"),
    "onepeer-exp-n16-p350m": Workload(
        "onepeer-exp-n16-p350m", 16, 350_000_000, "one_peer_exp", "f32", 10, 0.1, 5,
        description="n=16 one-peer exponential graph (i <- i+2^(t mod 4)), P=350M fp32, H=10"),
    "regular3-n32-p150m-bf16": Workload(
        "regular3-n32-p150m-bf16", 32, 150_000_000, "random_regular", "bf16", 30, 0.1, 3, degree=3,
        description="n=32 random 3-regular graph resampled per round (Metropolis 1/4), "
                    "P=150M bf16 params, fp32 state, H=30"),
    "matching-n64-p50m-hetH": Workload(
        "matching-n64-p50m-hetH", 64, 50_000_000, "one_peer", "f32", 50, 0.0, 3, hetero_H=(5, 50),
        description="n=64 random perfect matching per round (0.5/0.5), P=50M fp32, "
                    "H_i ~ U{5..50}, gamma=0, consensus error every round"),
}

WORKLOAD_ORDER = ["ring-n4-p1m", "exp-n8-p124m", "onepeer-exp-n16-p350m",
                  "regular3-n32-p150m-bf16", "matching-n64-p50m-hetH"]


def padded_ld(P, param_dtype):
    """Row stride (elements) so that every row starts 16-byte aligned."""
    per16 = 8 if param_dtype == "bf16" else 4
    return (P + per16 - 1) // per16 * per16


def local_steps(w: Workload):
    """Per-worker local-step counts H_i (fixed for the whole run)."""
    if w.hetero_H is None:
        return np.full(w.n, w.H, dtype=np.int64)
    lo, hi = w.hetero_H
    return np.random.default_rng(SEED_H).integers(lo, hi + 1, size=w.n).astype(np.int64)


def active_masks(H_i):
    """active[h][i] = 1 iff worker i still takes local step h of this round."""
    H_i = np.asarray(H_i)
    return [(H_i > h).astype(np.uint8) for h in range(int(H_i.max()) if H_i.size else 0)]


def worker_means(n):
    return (np.random.default_rng(SEED_MU).standard_normal(n) * 0.1).astype(np.float32)


def make_x0(P, device="cpu", dtype=None):
    """x0 ~ N(0, 0.02^2), fp32, drawn with torch's generator on `device`."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(SEED_X0)
    x0 = torch.empty(P, dtype=torch.float32, device=device)
    x0.normal_(0.0, 0.02, generator=gen)
    if dtype is not None:
        x0 = x0.to(dtype)
    return x0


def fill_grads(out, mu, step):
    """out[i, :] = mu_i + N(0, 1) for the global local-step index `step`.

    `out` is an [n, ld] fp32 torch tensor; columns beyond P are left as drawn.
    """
    import torch

    gen = torch.Generator(device=out.device)
    gen.manual_seed(SEED_GRAD_BASE + int(step))
    out.normal_(0.0, 1.0, generator=gen)
    out.add_(torch.as_tensor(np.asarray(mu, dtype=np.float32), device=out.device).view(-1, 1))
    return out


def sample_columns(P, count, seed=12345, edge=64):
    """Sorted distinct column indices: both ends of the row plus uniform picks."""
    rng = np.random.default_rng(seed)
    picks = set(range(min(edge, P)))
    picks.update(range(max(0, P - edge), P))
    if count > len(picks):
        picks.update(rng.choice(P, size=min(P, count - len(picks)), replace=False).tolist())
    return np.array(sorted(picks), dtype=np.int64)

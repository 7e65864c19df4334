"""Lock-step driver for GPU-vs-oracle parity (tests only).

Runs the same seeded workload through the HIP library (via the ctypes
binding) and through the oracle, on all columns or on a sample of columns
(every stored value at column p depends only on column p of the inputs, so
the oracle can simulate any subset of columns exactly).

Tolerances (fp32 state): |a - b| <= 1e-5 |b| + 1e-5 rms(b); reductions:
1e-4 relative; schedules and indices: bit-exact.
"""
import math
import sys

import numpy as np

import gasloc_inputs as gi
import oracle

REL = 1e-5
RED_REL = 1e-4


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def within(a, b, rel=REL, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    # non-finite reference values must be reproduced exactly (the same
    # infinity, or a NaN); the tolerance applies to the finite ones
    nonfinite = ~np.isfinite(b)
    if nonfinite.any():
        an, bn = a[nonfinite], b[nonfinite]
        ok = (an == bn) | (np.isnan(an) & np.isnan(bn))
        assert ok.all(), "%s: %d non-finite reference values not reproduced" % (what, int((~ok).sum()))
        a, b = a[~nonfinite], b[~nonfinite]
    rms = math.sqrt(float(np.mean(b * b))) if b.size else 0.0
    err = np.abs(a - b)
    bad = err > rel * np.abs(b) + rel * rms
    if bad.any():
        idx = np.unravel_index(np.argmax(err), err.shape)
        raise AssertionError("%s: %d of %d elements outside tolerance; worst at %s: %r vs %r (rms %g)"
                             % (what, int(bad.sum()), bad.size, idx, a[idx], b[idx], rms))


def bf16_ulp_check(gpu_bits, ref_bits, what="", max_frac=1e-6):
    """Every bf16 value within one ulp and at most max_frac of them differing."""
    g = np.asarray(gpu_bits).astype(np.int64)
    r = np.asarray(ref_bits).astype(np.int64)
    gs = np.where(g & 0x8000, -(g & 0x7FFF), g)  # sign-magnitude to a monotone integer line
    rs = np.where(r & 0x8000, -(r & 0x7FFF), r)
    diff = np.abs(gs - rs)
    assert diff.max(initial=0) <= 1, "%s: bf16 values %d ulp apart" % (what, diff.max())
    frac = float((diff != 0).mean()) if diff.size else 0.0
    assert frac <= max_frac, "%s: %.3g of bf16 values differ" % (what, frac)


def reduction_close(a, b, what=""):
    if b == 0.0:
        assert a == 0.0, "%s: expected exactly 0, got %r" % (what, a)
        return
    assert abs(a - b) <= RED_REL * abs(b), "%s: %r vs %r (rel %.3g)" % (what, a, b, abs(a - b) / abs(b))


class Pair:
    """A GPU context and its oracles driven with identical inputs."""

    def __init__(self, n, P, topology="ring", param_dtype="f32", gamma=0.1, mu=0.9, nesterov=True,
                 eta=0.7, seed=gi.SEED_TOPOLOGY, degree=3, cols=None, precisions=("f32", "f64"),
                 lr=gi.LOCAL_LR, form="eq"):
        import torch

        import paper_2606_11081_amd as g

        self.torch = torch
        self.n, self.P, self.param_dtype, self.lr = n, P, param_dtype, lr
        self.gpu = g.GASLoC(n, P, topology=topology, seed=seed, degree=degree, param_dtype=param_dtype,
                            beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY,
                            outer_lr=eta, outer_momentum=mu, outer_nesterov=nesterov,
                            consensus_momentum=gamma, round_form=form)
        self.cols = np.arange(P) if cols is None else np.asarray(cols)
        self.full = cols is None
        self.cols_dev = torch.as_tensor(self.cols, device="cuda")
        hp = oracle.OracleHParams(beta1=gi.BETA1, beta2=gi.BETA2, eps=gi.EPS, weight_decay=gi.WEIGHT_DECAY,
                                  outer_lr=eta, outer_momentum=mu, nesterov=nesterov,
                                  consensus_momentum=gamma, form=form)
        if param_dtype == "bf16":
            precisions = ("f32",)
        self.oracles = {p: oracle.Oracle(n, len(self.cols), hp, topology=topology, seed=seed, degree=degree,
                                         precision=p, param_dtype=param_dtype) for p in precisions}
        x0 = gi.make_x0(P, device="cuda")
        self.gpu.set_params(x0)
        if param_dtype == "bf16":
            x0_host = x0.to(torch.bfloat16)[self.cols_dev].view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            x0_host = x0[self.cols_dev].cpu().numpy()
        for o in self.oracles.values():
            o.set_params(x0_host)
        self.grads = torch.empty((n, self.gpu.ld), dtype=torch.float32, device="cuda")
        self.mu_i = gi.worker_means(n)
        self.step = 0

    def local_step(self, active=None):
        gi.fill_grads(self.grads, self.mu_i, self.step)
        g_host = self.grads[:, self.cols_dev].cpu().numpy()
        self.gpu.local_step(self.grads, self.lr, active)
        for o in self.oracles.values():
            o.local_step(g_host, self.lr, active)
        self.step += 1

    def local_step_gossip_round(self, t, active=None, W=None):
        """The fused entry on the GPU; the oracle takes the two steps in turn."""
        gi.fill_grads(self.grads, self.mu_i, self.step)
        g_host = self.grads[:, self.cols_dev].cpu().numpy()
        self.gpu.local_step_gossip_round(self.grads, self.lr, t, active, W)
        for o in self.oracles.values():
            o.local_step(g_host, self.lr, active)
            if W is None:
                o.gossip_round(t)
            else:
                rp, col, val = W
                o.gossip_round(t, csr=(rp, col, val.astype(o.real)))
        self.step += 1
        self.check_pg("fused round %d" % t)

    def gossip_round(self, t, W=None):
        self.gpu.gossip_round(t, W)
        for o in self.oracles.values():
            if W is None:
                o.gossip_round(t)
            else:
                rp, col, val = W
                o.gossip_round(t, csr=(rp, col, val.astype(o.real)))
        self.check_pg("round %d" % t)

    def check_pg(self, what):
        """The round's fused pseudo-gradient statistic against the fp32 oracle's
        (only when the oracle holds every column)."""
        if not self.full or "f32" not in self.oracles:
            return
        reduction_close(self.gpu.pseudo_gradient_sq(), self.oracles["f32"].pg_last, "pseudo-gradient sq, " + what)

    def gather(self, name, rows=None):
        t = getattr(self.gpu, name)
        self.torch.cuda.synchronize()
        sel = t[:, self.cols_dev] if rows is None else t[rows][:, self.cols_dev]
        if t.dtype == self.torch.bfloat16:
            return sel.view(self.torch.int16).cpu().numpy().view(np.uint16)
        return sel.cpu().numpy()

    def params_f64(self, bits_or_f32):
        if self.param_dtype == "bf16":
            return oracle.bf16_bits_to_f32(bits_or_f32).astype(np.float64)
        return bits_or_f32.astype(np.float64)

    def check_state(self, names=("x", "u", "zp", "m", "v"), y_rows=None, tag=""):
        """Compare GPU buffers with every oracle; y only for `y_rows` (stepped workers)."""
        stats = {}
        for name in names:
            if name in ("u", "zp") and getattr(self.gpu, name) is None:
                continue
            gpu = self.gather(name)
            for prec, o in self.oracles.items():
                ref = getattr(o, name)
                what = "%s %s vs %s oracle" % (tag, name, prec)
                if name in ("x",) and self.param_dtype == "bf16":
                    bf16_ulp_check(gpu, ref, what)
                else:
                    within(gpu if name not in ("x",) else self.params_f64(gpu),
                           ref if name not in ("x",) else o.params_f64("x"), REL, what)
                if prec == "f32":
                    gb = gpu.view(np.uint32) if gpu.dtype == np.float32 else gpu
                    rb = np.asarray(ref)
                    rb = rb.view(np.uint32) if rb.dtype == np.float32 else rb
                    stats[name] = float(np.mean(gb == rb))
        # the kernels take every rounding step in the fp32 oracle's order, so
        # the fp32 state must be bit-identical, not merely within tolerance
        if stats:
            assert min(stats.values()) == 1.0, "%s: not bit-identical to the fp32 oracle: %s" % (tag, stats)
        if y_rows is not None and len(y_rows):
            rows = np.asarray(y_rows)
            gy = self.gather("y", rows=self.torch.as_tensor(rows, device="cuda"))
            for prec, o in self.oracles.items():
                what = "%s y vs %s oracle" % (tag, prec)
                if self.param_dtype == "bf16":
                    bf16_ulp_check(gy, o.y[rows], what)
                else:
                    within(gy, o.y[rows], REL, what)
        return stats

"""Python front end of the plain-C GASLoC oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module.  It loads liboracle_f32.so / liboracle_f64.so (oracle/build.py)
and keeps the per-worker state of the method as numpy arrays:

  x, y      [n, P] parameters: round anchor x_t^i and live local iterate
            x_{t,h}^i (Eq. 1; Algorithm 1), fp32 / bf16 (uint16) / fp64
  m, v      [n, P] AdamW moments (App. B "Optimization")
  u         [n, P] outer (Nesterov) momentum (section 4, App. B)
  zp        [n, P] previous post-outer iterate x_{t-1} + eta g_{t-1} (Eq. 2)
  k         [n]    AdamW step count per worker
  rounds_done      completed gossip rounds

Every method is a direct call of the C routine that follows the paper's
definition; nothing here does arithmetic of the method.
"""
import ctypes
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))

TOPOLOGY_CODES = {
    "ring": 1,
    "complete": 2,
    "exponential": 3,
    "one_peer_exp": 4,
    "one_peer": 5,
    "two_peer": 6,
    "random_regular": 7,
}

PARAM_NATIVE = 0
PARAM_BF16 = 1

_u64p = ctypes.POINTER(ctypes.c_uint64)
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_d = ctypes.c_double


def _load(tag):
    path = os.path.join(HERE, "liboracle_%s.so" % tag)
    if not os.path.exists(path):
        from . import build as _build  # test infrastructure: compile on demand

        _build.build()
    lib = ctypes.CDLL(path)
    lib.orc_real_size.restype = ctypes.c_int
    lib.orc_mix64.restype = ctypes.c_uint64
    lib.orc_mix64.argtypes = [ctypes.c_uint64]
    lib.orc_next.restype = ctypes.c_uint64
    lib.orc_next.argtypes = [_u64p]
    lib.orc_round_state.restype = ctypes.c_uint64
    lib.orc_round_state.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.orc_bounded.restype = ctypes.c_uint64
    lib.orc_bounded.argtypes = [_u64p, ctypes.c_uint64]
    lib.orc_shuffle.restype = None
    lib.orc_shuffle.argtypes = [_u64p, _vp, ctypes.c_int32]
    lib.orc_topology.restype = ctypes.c_int
    lib.orc_topology.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_uint64,
                                 ctypes.c_uint64, _vp, _vp, _vp, ctypes.c_int]
    lib.orc_topology_restricted.restype = ctypes.c_int
    lib.orc_topology_restricted.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_uint64,
                                            ctypes.c_uint64, _vp, _vp, _vp, _vp, ctypes.c_int]
    lib.orc_skip_exchanges.restype = ctypes.c_int
    lib.orc_skip_exchanges.argtypes = [ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_int]
    lib.orc_adamw_scalars.restype = None
    lib.orc_adamw_scalars.argtypes = [_d, _d, _d, _d, _i64, _vp, _vp, _vp]
    lib.orc_local_step.restype = ctypes.c_int
    lib.orc_local_step.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp, _i64, _vp, _vp,
                                   _vp, _vp, _d, _d, _d, _d, _d]
    lib.orc_gossip_round.restype = ctypes.c_int
    lib.orc_gossip_round.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp, _vp,
                                     _vp, _vp, _vp, _d, _d, ctypes.c_int, _d, _i64]
    lib.orc_alg1_round.restype = ctypes.c_int
    lib.orc_alg1_round.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp,
                                   _d, _d, ctypes.c_int]
    lib.orc_dadam_round.restype = ctypes.c_int
    lib.orc_dadam_round.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.orc_local_dadam_round.restype = ctypes.c_int
    lib.orc_local_dadam_round.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp, _vp,
                                          _vp, _vp, _d, _d, ctypes.c_int]
    lib.orc_lr_schedule.restype = ctypes.c_float
    lib.orc_lr_schedule.argtypes = [_d, _i64, _i64, _d, _d, _d]
    lib.orc_consensus_error.restype = _d
    lib.orc_consensus_error.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp]
    lib.orc_pseudo_gradient_sq.restype = _d
    lib.orc_pseudo_gradient_sq.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp]
    lib.orc_replica_mean.restype = None
    lib.orc_replica_mean.argtypes = [ctypes.c_int, _i64, _i64, ctypes.c_int, _vp, _vp]
    lib.orc_f32_to_bf16.restype = ctypes.c_uint16
    lib.orc_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.orc_bf16_to_f32.restype = ctypes.c_float
    lib.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    return lib


_LIBS = {}


def lib(precision="f32"):
    if precision not in _LIBS:
        _LIBS[precision] = _load(precision)
    return _LIBS[precision]


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


# --------------------------------------------------------------------------
# generator and schedule helpers
# --------------------------------------------------------------------------

def splitmix64_stream(seed, count, precision="f32"):
    L = lib(precision)
    s = ctypes.c_uint64(seed)
    return [L.orc_next(ctypes.byref(s)) for _ in range(count)]


def round_state(seed, t):
    return lib().orc_round_state(seed, t)


def bounded_draws(state, k, count):
    L = lib()
    s = ctypes.c_uint64(state)
    return [L.orc_bounded(ctypes.byref(s), k) for _ in range(count)]


def shuffled_identity(state, N):
    L = lib()
    a = np.arange(N, dtype=np.int32)
    s = ctypes.c_uint64(state)
    L.orc_shuffle(ctypes.byref(s), _ptr(a), N)
    return a


def topology_csr(kind, n, seed, t, degree=3, precision="f32", admissible=None):
    """CSR (row_ptr int32[n+1], col int32[nnz], val[nnz]) of round t.

    Weights are float32 from the fp32 oracle (the library's CSR format) and
    float64 from the fp64 oracle.  admissible: optional [n, n] 0/1 matrix
    restricting the randomized 1-/2-Peer selections.
    """
    cap = n * n
    row_ptr = np.zeros(n + 1, dtype=np.int32)
    col = np.zeros(max(cap, 1), dtype=np.int32)
    val = np.zeros(max(cap, 1), dtype=np.float32 if precision == "f32" else np.float64)
    adm = None if admissible is None else np.ascontiguousarray(admissible, dtype=np.uint8)
    nnz = lib(precision).orc_topology_restricted(TOPOLOGY_CODES[kind], n, degree, seed, t,
                                                 None if adm is None else _ptr(adm), _ptr(row_ptr),
                                                 _ptr(col), _ptr(val), cap)
    if nnz < 0:
        raise ValueError("oracle: bad topology arguments (%s, n=%d, degree=%d)" % (kind, n, degree))
    return row_ptr, col[:nnz].copy(), val[:nnz].copy()


def skip_exchanges(W, n, alive=None, link_ok=None, precision="f32"):
    """The CSR W with every exchange of a dead worker or a failed link skipped."""
    rp, col, val = W
    real = np.float32 if precision == "f32" else np.float64
    rp = np.ascontiguousarray(rp, dtype=np.int32)
    col = np.ascontiguousarray(col, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=real)
    al = None if alive is None else np.ascontiguousarray(alive, dtype=np.uint8)
    lk = None if link_ok is None else np.ascontiguousarray(link_ok, dtype=np.uint8)
    cap = n * n
    orp = np.zeros(n + 1, np.int32)
    ocol = np.zeros(cap, np.int32)
    oval = np.zeros(cap, real)
    nnz = lib(precision).orc_skip_exchanges(n, _ptr(rp), _ptr(col), _ptr(val), None if al is None else _ptr(al),
                                            None if lk is None else _ptr(lk), _ptr(orp), _ptr(ocol), _ptr(oval),
                                            cap)
    if nnz < 0:
        raise ValueError("oracle: bad skip_exchanges arguments")
    return orp, ocol[:nnz].copy(), oval[:nnz].copy()


def csr_to_dense(row_ptr, col, val, n):
    W = np.zeros((n, n), dtype=np.float64)
    for i in range(n):
        for k in range(row_ptr[i], row_ptr[i + 1]):
            W[i, col[k]] = val[k]
    return W


def lr_schedule(peak, step, total, warmup_frac=0.1, start_frac=0.01, final_frac=0.0):
    return lib().orc_lr_schedule(peak, step, total, warmup_frac, start_frac, final_frac)


def adamw_scalars(lr, beta1, beta2, wd, k, precision="f32"):
    dt = np.float32 if precision == "f32" else np.float64
    out = [np.zeros(1, dtype=dt) for _ in range(3)]
    lib(precision).orc_adamw_scalars(lr, beta1, beta2, wd, k, *[_ptr(o) for o in out])
    return tuple(o[0] for o in out)


def f32_to_bf16_bits(a):
    L = lib()
    flat = np.asarray(a, dtype=np.float32).ravel()
    return np.array([L.orc_f32_to_bf16(float(f)) for f in flat], dtype=np.uint16).reshape(np.shape(a))


def bf16_bits_to_f32(h):
    h = np.asarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# the stateful oracle
# --------------------------------------------------------------------------

@dataclass
class OracleHParams:
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1
    outer_lr: float = 0.7
    outer_momentum: float = 0.9
    nesterov: bool = True
    consensus_momentum: float = 0.1
    # "eq": Eq. 1 / Eq. 2; "alg1": Algorithm 1; "dadam", "local_dadam": App. C
    form: str = "eq"


class Oracle:
    """All n workers' state on the host; P columns (or a sample of columns)."""

    def __init__(self, n, P, hp, topology="ring", seed=0, degree=3, precision="f32",
                 param_dtype="f32", admissible=None):
        self.n, self.P, self.hp = int(n), int(P), hp
        self.admissible = admissible
        self.topology, self.seed, self.degree = topology, int(seed), int(degree)
        self.precision = precision
        self.L = lib(precision)
        self.real = np.float32 if precision == "f32" else np.float64
        if param_dtype == "bf16":
            if precision != "f32":
                raise ValueError("bf16 parameter storage needs the fp32-arithmetic oracle")
            self.pcode, self.pdt = PARAM_BF16, np.uint16
        else:
            self.pcode, self.pdt = PARAM_NATIVE, self.real
        shape = (self.n, self.P)
        self.x = np.zeros(shape, dtype=self.pdt)
        self.y = np.zeros(shape, dtype=self.pdt)
        self.m = np.zeros(shape, dtype=self.real)
        self.v = np.zeros(shape, dtype=self.real)
        self.u = np.zeros(shape, dtype=self.real)
        self.zp = np.zeros(shape, dtype=self.real)
        self.z = np.zeros(shape, dtype=self.real)
        self.k = np.zeros(self.n, dtype=np.int64)
        self.rounds_done = 0
        self.pg_last = 0.0  # pseudo_gradient_sq() of the state the last round consumed

    # hyperparameters as the library receives them: fp32 values for the fp32
    # oracle, the exact values for the fp64 one
    def _h(self, v):
        return float(np.float32(v)) if self.precision == "f32" else float(v)

    def set_params(self, x0):
        """Identical initial replicas x_0^i = x_0 (section 3.3, Proposition 2's assumption)."""
        x0 = np.asarray(x0)
        if self.pcode == PARAM_BF16:
            src = x0 if x0.dtype == np.uint16 else f32_to_bf16_bits(x0.astype(np.float32))
        else:
            src = x0.astype(self.real)
        self.x[...] = src
        self.y[...] = src

    def params_f64(self, which="x"):
        a = getattr(self, which)
        if self.pcode == PARAM_BF16:
            return bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)

    def local_step(self, g, lr, active=None):
        g = np.ascontiguousarray(g, dtype=np.float32)
        assert g.shape == (self.n, self.P)
        act = np.ones(self.n, dtype=np.uint8) if active is None else np.asarray(active, dtype=np.uint8)
        self.k += act.astype(np.int64)
        hp = self.hp
        rc = self.L.orc_local_step(self.n, self.P, self.P, self.pcode, _ptr(self.y), _ptr(g), self.P,
                                   _ptr(self.m), _ptr(self.v), _ptr(act), _ptr(self.k),
                                   self._h(lr), self._h(hp.beta1), self._h(hp.beta2), self._h(hp.eps),
                                   self._h(hp.weight_decay))
        if rc != 0:
            raise ValueError("oracle local_step rejected its arguments")

    def csr(self, t):
        return topology_csr(self.topology, self.n, self.seed, t, self.degree, self.precision, self.admissible)

    def gossip_round(self, t=0, csr=None):
        row_ptr, col, val = self.csr(t) if csr is None else csr
        row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
        col = np.ascontiguousarray(col, dtype=np.int32)
        val = np.ascontiguousarray(val, dtype=self.real)
        hp = self.hp
        self.pg_last = self.pseudo_gradient_sq()
        common = (self.n, self.P, self.P, self.pcode, _ptr(self.x), _ptr(self.y))
        outer = (self._h(hp.outer_momentum), self._h(hp.outer_lr), int(bool(hp.nesterov)))
        csr = (_ptr(row_ptr), _ptr(col), _ptr(val))
        if hp.form == "eq":
            rc = self.L.orc_gossip_round(*common, _ptr(self.u), _ptr(self.zp), _ptr(self.z), *csr, *outer[:2],
                                         outer[2], self._h(hp.consensus_momentum), self.rounds_done)
        elif hp.form == "alg1":
            rc = self.L.orc_alg1_round(*common, _ptr(self.u), *csr, *outer)
        elif hp.form == "dadam":
            rc = self.L.orc_dadam_round(*common, _ptr(self.z), *csr)
        elif hp.form == "local_dadam":
            rc = self.L.orc_local_dadam_round(*common, _ptr(self.u), _ptr(self.z), *csr, *outer)
        else:
            raise ValueError("unknown round form %r" % hp.form)
        if rc != 0:
            raise ValueError("oracle gossip_round rejected its arguments")
        self.rounds_done += 1

    def consensus_error(self, cols=None):
        """||pi x||^2 over all columns, or over the column slice/index array `cols`."""
        if cols is None:
            return self.L.orc_consensus_error(self.n, self.P, self.P, self.pcode, _ptr(self.x))
        sub = np.ascontiguousarray(self.x[:, cols])
        return self.L.orc_consensus_error(self.n, sub.shape[1], sub.shape[1], self.pcode, _ptr(sub))

    def pseudo_gradient_sq(self, cols=None):
        """sum_i ||x_i - y_i||^2 of the current anchors and live iterates (Eq. 1's
        pseudo-gradients), over all columns or the slice/index array `cols`."""
        if cols is None:
            return self.L.orc_pseudo_gradient_sq(self.n, self.P, self.P, self.pcode, _ptr(self.x), _ptr(self.y))
        sx, sy = np.ascontiguousarray(self.x[:, cols]), np.ascontiguousarray(self.y[:, cols])
        return self.L.orc_pseudo_gradient_sq(self.n, sx.shape[1], sx.shape[1], self.pcode, _ptr(sx), _ptr(sy))

    def replica_mean(self):
        out = np.zeros(self.P, dtype=self.pdt)
        self.L.orc_replica_mean(self.n, self.P, self.P, self.pcode, _ptr(self.x), _ptr(out))
        return out

"""Thin ctypes binding of libgasloc.so: same names as include/gasloc.h.

Argument marshalling only: torch tensors become device pointers, numpy
arrays become host pointers, status codes become GaslocError.  Every step of
the round runs in the library's HIP kernels; there is no fallback path.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgasloc.so")

GASLOC_OK, GASLOC_EINVAL, GASLOC_ENOMEM, GASLOC_EDEVICE, GASLOC_ESTATE = range(5)
STATUS_NAMES = {0: "OK", 1: "EINVAL", 2: "ENOMEM", 3: "EDEVICE", 4: "ESTATE"}
GASLOC_F32, GASLOC_BF16 = 0, 1
ROUND_FORM = {"eq": 0, "alg1": 1, "dadam": 2, "local_dadam": 3}
TOPOLOGY = {
    "explicit": 0,
    "ring": 1,
    "complete": 2,
    "exponential": 3,
    "one_peer_exp": 4,
    "one_peer": 5,
    "two_peer": 6,
    "random_regular": 7,
}


class GaslocError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


class gasloc_topology(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("degree", ctypes.c_int32), ("seed", ctypes.c_uint64),
                ("admissible", ctypes.c_void_p)]


class gasloc_hparams(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("outer_lr", ctypes.c_float),
                ("outer_momentum", ctypes.c_float), ("outer_nesterov", ctypes.c_int32),
                ("consensus_momentum", ctypes.c_float), ("param_dtype", ctypes.c_int32),
                ("round_form", ctypes.c_int32)]


class gasloc_buffers(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("y", ctypes.c_void_p), ("m", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("u", ctypes.c_void_p), ("zp", ctypes.c_void_p),
                ("ld", ctypes.c_int64)]


class gasloc_csr(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("nnz", ctypes.c_int32), ("row_ptr", ctypes.c_void_p),
                ("col", ctypes.c_void_p), ("val", ctypes.c_void_p)]


_vp = ctypes.c_void_p
_i32, _i64, _u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
_SIGNATURES = {
    "gasloc_init": (ctypes.c_int, [_i32, _i64, ctypes.POINTER(gasloc_topology),
                                   ctypes.POINTER(gasloc_hparams), ctypes.POINTER(gasloc_buffers), _vp,
                                   ctypes.POINTER(_vp)]),
    "gasloc_local_step": (ctypes.c_int, [_vp, _vp, _i64, _vp, ctypes.c_float]),
    "gasloc_gossip_round": (ctypes.c_int, [_vp, ctypes.POINTER(gasloc_csr), _u64]),
    "gasloc_local_step_gossip_round": (ctypes.c_int, [_vp, _vp, _i64, _vp, ctypes.c_float,
                                                      ctypes.POINTER(gasloc_csr), _u64]),
    "gasloc_consensus_error": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_double)]),
    "gasloc_pseudo_gradient_sq": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_double)]),
    "gasloc_consensus_error_cols": (ctypes.c_int, [_vp, _i64, _i64, ctypes.POINTER(ctypes.c_double)]),
    "gasloc_consensus_error_cols_noalloc": (ctypes.c_int, [_vp, _i32, _i32, _i64, _i64, _i64, _vp, _vp]),
    "gasloc_replica_mean": (ctypes.c_int, [_vp, _vp]),
    "gasloc_topology_csr": (ctypes.c_int, [_vp, _u64, _vp, _vp, _vp, _i32, ctypes.POINTER(_i32)]),
    "gasloc_make_topology": (ctypes.c_int, [ctypes.POINTER(gasloc_topology), _i32, _u64, _vp, _vp, _vp,
                                            _i32, ctypes.POINTER(_i32)]),
    "gasloc_validate_csr": (ctypes.c_int, [ctypes.POINTER(gasloc_csr), _i32]),
    "gasloc_skip_exchanges": (ctypes.c_int, [ctypes.POINTER(gasloc_csr), _vp, _vp, _vp, _vp, _vp, _i32,
                                             ctypes.POINTER(_i32)]),
    "gasloc_set_alive": (ctypes.c_int, [_vp, _vp]),
    "gasloc_get_counters": (ctypes.c_int, [_vp, _vp, _vp, ctypes.POINTER(_i64)]),
    "gasloc_set_counters": (ctypes.c_int, [_vp, _vp, _vp, _i64]),
    "gasloc_lr_schedule": (ctypes.c_float, [ctypes.c_float, _i64, _i64, ctypes.c_float, ctypes.c_float,
                                            ctypes.c_float]),
    "gasloc_stream_probe": (ctypes.c_int, [_i32, _i32, _i32, _i32, _vp, _vp, _i64, _i32, _vp, _vp]),
    "gasloc_last_error": (ctypes.c_char_p, [_vp]),
    "gasloc_build_info": (ctypes.c_char_p, []),
    "gasloc_destroy": (None, [_vp]),
}

_lib = None


def library():
    """Load libgasloc.so (built by paper_2606_11081_amd/build.py); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libgasloc.so is not built (%s); run __graft_entry__.build() or "
                              "python paper_2606_11081_amd/build.py" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status, ctx=None):
    if status != GASLOC_OK:
        msg = library().gasloc_last_error(ctx)
        raise GaslocError(status, msg.decode() if msg else "")


def _dev(t):
    """Device pointer of a torch tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def make_topology_struct(kind="ring", seed=0, degree=3, admissible=None):
    """Topology struct; with `admissible` (an [n, n] 0/1 array) the array is
    kept alive on the struct as `_keep`."""
    code = TOPOLOGY[kind] if isinstance(kind, str) else int(kind)
    if admissible is None:
        return gasloc_topology(code, int(degree), int(seed), None)
    adm, ptr = _host(admissible, np.uint8)
    t = gasloc_topology(code, int(degree), int(seed), ptr)
    t._keep = adm
    return t


def make_hparams(beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, outer_lr=0.7, outer_momentum=0.9,
                 outer_nesterov=True, consensus_momentum=0.1, param_dtype="f32", round_form="eq"):
    dt = GASLOC_BF16 if param_dtype in ("bf16", GASLOC_BF16) else GASLOC_F32
    form = ROUND_FORM[round_form] if isinstance(round_form, str) else int(round_form)
    return gasloc_hparams(beta1, beta2, eps, weight_decay, outer_lr, outer_momentum, int(bool(outer_nesterov)),
                          consensus_momentum, dt, form)


def make_csr(row_ptr, col, val):
    """Host CSR struct; the returned tuple keeps the arrays alive."""
    rp, rpp = _host(row_ptr, np.int32)
    c, cp = _host(col, np.int32)
    v, vp = _host(val, np.float32)
    return gasloc_csr(len(rp) - 1, len(c), rpp, cp, vp), (rp, c, v)


# --------------------------------------------------------------------------
# the ABI calls
# --------------------------------------------------------------------------

def gasloc_init(n, P, topology, hparams, x, y, m, v, u, zp, ld, stream=None):
    """Returns the context handle (an int).  Buffers are torch device tensors."""
    bufs = gasloc_buffers(_dev(x), _dev(y), _dev(m), _dev(v), _dev(u), _dev(zp), int(ld))
    out = ctypes.c_void_p()
    st = library().gasloc_init(int(n), int(P), ctypes.byref(topology), ctypes.byref(hparams),
                               ctypes.byref(bufs), stream, ctypes.byref(out))
    _check(st)
    return out.value


def gasloc_local_step(ctx, grads, grad_ld, active=None, lr=0.0):
    keep = None
    ap = None
    if active is not None:
        keep, ap = _host(active, np.uint8)
    _check(library().gasloc_local_step(ctx, _dev(grads), int(grad_ld), ap, float(lr)), ctx)
    del keep


def gasloc_gossip_round(ctx, W=None, t=0):
    """W: None, or a (row_ptr, col, val) tuple of host arrays."""
    if W is None:
        _check(library().gasloc_gossip_round(ctx, None, int(t)), ctx)
        return
    csr, keep = make_csr(*W)
    _check(library().gasloc_gossip_round(ctx, ctypes.byref(csr), int(t)), ctx)
    del keep


def gasloc_local_step_gossip_round(ctx, grads, grad_ld, active=None, lr=0.0, W=None, t=0):
    """The last local step and the gossip round in one pass (same results as the two calls)."""
    keep_a = ap = None
    if active is not None:
        keep_a, ap = _host(active, np.uint8)
    if W is None:
        st = library().gasloc_local_step_gossip_round(ctx, _dev(grads), int(grad_ld), ap, float(lr), None, int(t))
    else:
        csr, keep = make_csr(*W)
        st = library().gasloc_local_step_gossip_round(ctx, _dev(grads), int(grad_ld), ap, float(lr),
                                                      ctypes.byref(csr), int(t))
    _check(st, ctx)
    del keep_a


def gasloc_consensus_error(ctx):
    out = ctypes.c_double()
    _check(library().gasloc_consensus_error(ctx, ctypes.byref(out)), ctx)
    return out.value


def gasloc_pseudo_gradient_sq(ctx):
    """sum_i ||x_i - y_i||^2 of the pseudo-gradients the last round consumed (fp64); blocks."""
    out = ctypes.c_double()
    _check(library().gasloc_pseudo_gradient_sq(ctx, ctypes.byref(out)), ctx)
    return out.value


def gasloc_consensus_error_cols(ctx, p_begin, p_end):
    out = ctypes.c_double()
    _check(library().gasloc_consensus_error_cols(ctx, int(p_begin), int(p_end), ctypes.byref(out)), ctx)
    return out.value


def gasloc_consensus_error_cols_noalloc(x, param_dtype, n, ld, p_begin, p_end, out, stream=None):
    """Context-free, allocation-free consensus error of columns [p_begin, p_end)
    of the device buffer x ([n, ld]) into the device fp64 `out` (enqueued on
    `stream`, a torch stream or None for the null stream; does not wait)."""
    dt = GASLOC_BF16 if param_dtype in ("bf16", GASLOC_BF16) else GASLOC_F32
    _check(library().gasloc_consensus_error_cols_noalloc(_dev(x), dt, int(n), int(ld), int(p_begin), int(p_end),
                                                          _dev(out), None if stream is None else stream.cuda_stream))


def gasloc_replica_mean(ctx, out):
    _check(library().gasloc_replica_mean(ctx, _dev(out)), ctx)


def _csr_out(n, cap):
    return (np.zeros(n + 1, np.int32), np.zeros(max(cap, 1), np.int32), np.zeros(max(cap, 1), np.float32))


def gasloc_topology_csr(ctx, t, n):
    rp, col, val = _csr_out(n, n * n)
    nnz = _i32()
    _check(library().gasloc_topology_csr(ctx, int(t), rp.ctypes.data, col.ctypes.data, val.ctypes.data,
                                         n * n, ctypes.byref(nnz)), ctx)
    return rp, col[:nnz.value].copy(), val[:nnz.value].copy()


def gasloc_make_topology(topology, n, t):
    rp, col, val = _csr_out(n, n * n)
    nnz = _i32()
    _check(library().gasloc_make_topology(ctypes.byref(topology), int(n), int(t), rp.ctypes.data,
                                          col.ctypes.data, val.ctypes.data, n * n, ctypes.byref(nnz)))
    return rp, col[:nnz.value].copy(), val[:nnz.value].copy()


def gasloc_validate_csr(W, n):
    csr, keep = make_csr(*W)
    _check(library().gasloc_validate_csr(ctypes.byref(csr), int(n)))
    del keep


def gasloc_skip_exchanges(W, n, alive=None, link_ok=None):
    csr, keep = make_csr(*W)
    al = lk = None
    if alive is not None:
        al, alp = _host(alive, np.uint8)
    if link_ok is not None:
        lk, lkp = _host(link_ok, np.uint8)
    rp, col, val = _csr_out(n, n * n)
    nnz = _i32()
    _check(library().gasloc_skip_exchanges(ctypes.byref(csr), None if al is None else alp,
                                           None if lk is None else lkp, rp.ctypes.data, col.ctypes.data,
                                           val.ctypes.data, n * n, ctypes.byref(nnz)))
    del keep
    return rp, col[:nnz.value].copy(), val[:nnz.value].copy()


def gasloc_set_alive(ctx, alive=None):
    keep = ptr = None
    if alive is not None:
        keep, ptr = _host(alive, np.uint8)
    _check(library().gasloc_set_alive(ctx, ptr), ctx)
    del keep


def gasloc_get_counters(ctx, n):
    k = np.zeros(n, np.int64)
    stepped = np.zeros(n, np.uint8)
    rounds = _i64()
    _check(library().gasloc_get_counters(ctx, k.ctypes.data, stepped.ctypes.data, ctypes.byref(rounds)), ctx)
    return k, stepped, rounds.value


def gasloc_set_counters(ctx, k, stepped, rounds_done):
    kk, kp = _host(k, np.int64)
    ss, sp = _host(stepped, np.uint8)
    _check(library().gasloc_set_counters(ctx, kp, sp, int(rounds_done)), ctx)
    del kk, ss


def gasloc_lr_schedule(peak, step, total_steps, warmup_frac=0.1, start_frac=0.01, final_frac=0.0):
    return library().gasloc_lr_schedule(peak, int(step), int(total_steps), warmup_frac, start_frac, final_frac)


def gasloc_stream_probe(reads_f32, reads_bf16, writes_f32, writes_bf16, src, dst, count, sink=None,
                        stream=None, threads=256):
    """Measurement support (include/gasloc_probe.h): one launch of the streaming
    kernel with the given byte mix.  src, dst: lists of torch device tensors
    (fp32 streams first, then bf16); sink: a device tensor of at least 4 bytes
    for read-only mixes; stream: a torch stream (None = the null stream);
    threads: the workgroup size (64, 128 or 256)."""
    srcs = (ctypes.c_void_p * max(1, len(src)))(*[_dev(t) for t in src])
    dsts = (ctypes.c_void_p * max(1, len(dst)))(*[_dev(t) for t in dst])
    st = library().gasloc_stream_probe(int(reads_f32), int(reads_bf16), int(writes_f32), int(writes_bf16), srcs,
                                       dsts, int(count), int(threads), _dev(sink),
                                       None if stream is None else stream.cuda_stream)
    _check(st)


def gasloc_last_error(ctx=None):
    msg = library().gasloc_last_error(ctx)
    return msg.decode() if msg else ""


def gasloc_build_info():
    """The library's build record: the hash of the sources it was compiled from, arch, flags."""
    return library().gasloc_build_info().decode()


def gasloc_destroy(ctx):
    library().gasloc_destroy(ctx)


# --------------------------------------------------------------------------
# device memory plumbing (torch allocates, the library computes)
# --------------------------------------------------------------------------

def padded_ld(P, param_dtype):
    per16 = 8 if param_dtype in ("bf16", GASLOC_BF16) else 4
    return (P + per16 - 1) // per16 * per16


def alloc_buffers(n, P, param_dtype="f32", device="cuda", with_u=True, with_zp=True):
    """torch tensors x, y, m, v, u, zp of shape [n, ld] (u / zp None when not wanted)."""
    import torch

    ld = padded_ld(P, param_dtype)
    pdt = torch.bfloat16 if param_dtype in ("bf16", GASLOC_BF16) else torch.float32
    x = torch.empty((n, ld), dtype=pdt, device=device)
    y = torch.empty((n, ld), dtype=pdt, device=device)
    m = torch.empty((n, ld), dtype=torch.float32, device=device)
    v = torch.empty((n, ld), dtype=torch.float32, device=device)
    u = torch.empty((n, ld), dtype=torch.float32, device=device) if with_u else None
    zp = torch.empty((n, ld), dtype=torch.float32, device=device) if with_zp else None
    return dict(x=x, y=y, m=m, v=v, u=u, zp=zp, ld=ld)


class GASLoC:
    """Owns one context plus its torch buffers; methods are the ABI calls."""

    def __init__(self, n, P, topology="ring", seed=0, degree=3, param_dtype="f32", device="cuda",
                 stream=None, admissible=None, **hp):
        import torch

        self.n, self.P, self.param_dtype = int(n), int(P), param_dtype
        hpar = make_hparams(param_dtype=param_dtype, **hp)
        self.bufs = alloc_buffers(n, P, param_dtype, device,
                                  with_u=hpar.outer_momentum != 0.0 and hpar.round_form != ROUND_FORM["dadam"],
                                  with_zp=hpar.consensus_momentum != 0.0)
        self.ld = self.bufs["ld"]
        self.stream = torch.cuda.current_stream(device) if stream is None else stream
        b = self.bufs
        self.ctx = gasloc_init(n, P, make_topology_struct(topology, seed, degree, admissible), hpar, b["x"], b["y"],
                               b["m"], b["v"], b["u"], b["zp"], self.ld, self.stream.cuda_stream)

    def __getattr__(self, name):
        bufs = self.__dict__.get("bufs")
        if bufs is not None and name in bufs:
            return bufs[name]
        raise AttributeError(name)

    def set_params(self, x0):
        """Identical start: every worker's x is x0 (torch tensor of length P),
        written on the context's stream so that later calls see it."""
        import torch

        self.stream.wait_stream(torch.cuda.current_stream(self.stream.device))  # x0 may come from there
        with torch.cuda.stream(self.stream):
            self.bufs["x"][:, : self.P].copy_(x0.to(self.bufs["x"].dtype).view(1, -1).expand(self.n, -1))

    def local_step(self, grads, lr, active=None):
        gasloc_local_step(self.ctx, grads, grads.shape[1], active, lr)

    def gossip_round(self, t, W=None):
        gasloc_gossip_round(self.ctx, W, t)

    def local_step_gossip_round(self, grads, lr, t, active=None, W=None):
        gasloc_local_step_gossip_round(self.ctx, grads, grads.shape[1], active, lr, W, t)

    def consensus_error(self):
        return gasloc_consensus_error(self.ctx)

    def pseudo_gradient_sq(self):
        return gasloc_pseudo_gradient_sq(self.ctx)

    def consensus_error_cols(self, p_begin, p_end):
        return gasloc_consensus_error_cols(self.ctx, p_begin, p_end)

    def replica_mean(self, out):
        gasloc_replica_mean(self.ctx, out)

    def counters(self):
        """(k, stepped, rounds_done): per-worker AdamW step counts, which workers
        stepped since the last round, and the rounds done (for checkpoints)."""
        return gasloc_get_counters(self.ctx, self.n)

    def set_counters(self, k, stepped, rounds_done):
        """Restore the counters of a checkpoint (with the [n, ld] buffers)."""
        gasloc_set_counters(self.ctx, k, stepped, rounds_done)

    def set_alive(self, alive=None):
        """Mark dead workers (uint8 [n], 0 = dead; None = all alive): they skip
        their exchanges and local steps."""
        gasloc_set_alive(self.ctx, alive)

    def topology_csr(self, t):
        """The generated mixing matrix of round t as (row_ptr, col, val)."""
        return gasloc_topology_csr(self.ctx, t, self.n)

    def close(self):
        if self.__dict__.get("ctx"):
            gasloc_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

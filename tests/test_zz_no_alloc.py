"""The allocation-free consensus error (gasloc_consensus_error_cols_noalloc)
through the C ABI, against the context's gasloc_consensus_error_cols on the
same stored x: two calls in a row, the second on a smaller input (another,
smaller context), and the first on a range long enough that both entry points
group the fp64 sums the same way (bit-identical).  Runs alone in a fresh
process and after the rest of the suite."""
import numpy as np
import pytest

import gasloc_inputs as gi
import oracle
import paper_2606_11081_amd as g

pytestmark = pytest.mark.gpu

REL = 1e-4  # the reductions' tolerance against the reference


def _state(n, P, topology, dtype, rounds=2):
    """A context whose stored x has disagreement between workers."""
    import torch

    lib = g.GASLoC(n, P, topology=topology, seed=gi.SEED_TOPOLOGY, param_dtype=dtype, outer_lr=gi.OUTER_LR,
                   outer_momentum=gi.OUTER_MOMENTUM, consensus_momentum=0.1)
    lib.set_params(gi.make_x0(P, device="cuda"))
    grads = torch.empty((n, lib.ld), dtype=torch.float32, device="cuda")
    for t in range(rounds):
        gi.fill_grads(grads, gi.worker_means(n), t)
        lib.local_step(grads, gi.LOCAL_LR)
        lib.gossip_round(t)
    torch.cuda.synchronize()
    return lib


def _noalloc(lib, p0, p1):
    import torch

    out = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
    g.gasloc.gasloc_consensus_error_cols_noalloc(lib.x, lib.param_dtype, lib.n, lib.ld, p0, p1, out, lib.stream)
    torch.cuda.synchronize()
    return float(out.item())


def _host_ce(lib, p0, p1):
    """The oracle's two-pass fp64 consensus error of the downloaded columns."""
    import ctypes

    import torch

    part = lib.x[:, p0:p1].contiguous()
    if lib.param_dtype == "bf16":
        host, code = part.view(torch.int16).cpu().numpy().view(np.uint16), oracle.PARAM_BF16
    else:
        host, code = part.cpu().numpy(), oracle.PARAM_NATIVE
    host = np.ascontiguousarray(host)
    return oracle.lib("f32").orc_consensus_error(lib.n, p1 - p0, p1 - p0, code, host.ctypes.data_as(ctypes.c_void_p))


def test_noalloc_matches_the_context_entry_point_twice():
    import torch

    # first call: n=4, P=40M fp32, 2^13 + ... steps: 8 per workgroup on both sides
    n, P = 4, 40_000_003
    print("case noalloc call 1: n=%d P=%d f32 ring, columns [0, P)" % (n, P), flush=True)
    lib = _state(n, P, "ring", "f32")
    ref = lib.consensus_error_cols(0, P)
    got = _noalloc(lib, 0, P)
    assert got == ref, (got, ref)  # same kernel, same steps per workgroup, same segmented finalize
    assert abs(got - ref) <= REL * abs(ref)
    lib.close()
    del lib
    torch.cuda.empty_cache()
    # second call in a row, a smaller input (the scratch keeps the first
    # call's partials, which must not leak into this one)
    n, P = 6, 9_001
    print("case noalloc call 2: n=%d P=%d bf16 two_peer, columns [3, P-5)" % (n, P), flush=True)
    lib = _state(n, P, "two_peer", "bf16")
    ref = lib.consensus_error_cols(3, P - 5)
    got = _noalloc(lib, 3, P - 5)
    assert abs(got - ref) <= REL * abs(ref), (got, ref)
    assert abs(got - _host_ce(lib, 3, P - 5)) <= REL * abs(ref)
    # an empty range and identical replicas give exactly 0
    assert _noalloc(lib, 7, 7) == 0.0
    lib.close()


def test_noalloc_identical_replicas_give_zero():
    lib = _state(3, 5_000, "complete", "f32", rounds=0)
    assert _noalloc(lib, 0, 5_000) == 0.0
    lib.close()

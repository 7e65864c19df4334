"""The streaming probe kernel (measurement support, include/gasloc_probe.h):
every supported mix stores the fp32 sum of its sources, in order, to every
destination (bf16 destinations rounded to nearest-even), in place or not, over
several tiles and a ragged tail; a read-only mix leaves its sink alone."""
import numpy as np
import pytest

import paper_2606_11081_amd as g

pytestmark = pytest.mark.gpu

MIXES = [(4, 0, 0, 0), (0, 0, 3, 0), (1, 0, 1, 0), (4, 0, 3, 0), (3, 0, 2, 0), (3, 1, 2, 1), (2, 2, 2, 1),
         (7, 0, 5, 0), (6, 0, 4, 0), (5, 2, 4, 1)]


def _bf16_bits(a):
    """Round fp32 values to bf16 bit patterns (nearest, ties to even), as torch does."""
    import torch

    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(
        np.uint16)


@pytest.mark.parametrize("mix", MIXES)
@pytest.mark.parametrize("in_place", [False, True])
@pytest.mark.parametrize("threads", [256, 128, 64])
def test_probe_mix_stores_the_sum(mix, in_place, threads):
    import torch

    r32, r16, w32, w16 = mix
    count = 5 * 1024 + 7  # several tiles (of every workgroup size) and a ragged tail
    print("case probe mix %s in_place=%s count=%d threads=%d" % (mix, in_place, count, threads), flush=True)
    gen = torch.Generator(device="cpu").manual_seed(sum(mix) * 7 + int(in_place) + threads)
    src32 = [torch.randn(count, generator=gen).cuda() for _ in range(r32)]
    src16 = [torch.randn(count, generator=gen).to(torch.bfloat16).cuda() for _ in range(r16)]
    expect = np.zeros(count, np.float32)
    for t in src32 + src16:
        expect = expect + t.float().cpu().numpy()  # fp32 sums in stream order
    if in_place:
        dst32 = [src32[k] if k < r32 else torch.zeros(count).cuda() for k in range(w32)]
        dst16 = [src16[k] if k < r16 else torch.zeros(count, dtype=torch.bfloat16).cuda() for k in range(w16)]
    else:
        dst32 = [torch.zeros(count).cuda() for _ in range(w32)]
        dst16 = [torch.zeros(count, dtype=torch.bfloat16).cuda() for _ in range(w16)]
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    g.gasloc.gasloc_stream_probe(r32, r16, w32, w16, src32 + src16, dst32 + dst16, count, sink, threads=threads)
    torch.cuda.synchronize()
    for t in dst32:
        assert np.array_equal(t.cpu().numpy().view(np.uint32), expect.view(np.uint32))
    for t in dst16:
        assert np.array_equal(t.view(torch.int16).cpu().numpy().view(np.uint16), _bf16_bits(expect))
    assert int(sink.item()) == 0

"""heal_split_f32 on the GPU against the oracle's split, over all 2^32 inputs."""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from gpu_util import announce, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]


def _isnan16(h):
    return np.isnan((h.astype(np.uint32) << 16).view(np.float32))


def _compare(x_bits_start, n, hi_g, lo_g, hi_o, lo_o, x):
    """Bitwise equal, except NaNs compared by NaN-ness (payload and sign of a
    NaN are not part of the definition)."""
    hn, ln, hon, lon = _isnan16(hi_g), _isnan16(lo_g), _isnan16(hi_o), _isnan16(lo_o)
    assert np.array_equal(hn, hon), "NaN-ness of hi differs from the oracle's"
    assert np.array_equal(ln, lon), "NaN-ness of lo differs from the oracle's"
    ok = ~(hon | lon)
    bad = np.nonzero((hi_g[ok] != hi_o[ok]) | (lo_g[ok] != lo_o[ok]))[0]
    if bad.size:
        i = np.nonzero(ok)[0][bad[0]]
        raise AssertionError("split differs at x=0x%08x: gpu (%04x,%04x) oracle (%04x,%04x); "
                             "%d mismatches in chunk" % ((x_bits_start + i) & 0xffffffff, hi_g[i],
                                                         lo_g[i], hi_o[i], lo_o[i], bad.size))


def test_split_exhaustive_vs_oracle(orc):
    chunk = 1 << 28
    for start in range(0, 1 << 32, chunk):
        announce("split exhaustive chunk 0x%08x" % start)
        bits = torch.arange(start, start + chunk, dtype=torch.int64, device="cuda").to(torch.int32)
        x = bits.view(torch.float32)
        hi, lo = heal.heal_split_f32(x)
        torch.cuda.synchronize()
        hi_g = hi.cpu().numpy()
        lo_g = lo.cpu().numpy()
        xs = x.cpu().numpy()
        hi_o, lo_o = orc.split_range(start, chunk)
        _compare(start, chunk, hi_g, lo_g, hi_o, lo_o, xs)


@pytest.mark.parametrize("n,offset", [(1, 0), (7, 0), (8, 0), (9, 1), (1000003, 3), (4096, 2)])
def test_split_sizes_and_misalignment(orc, n, offset):
    announce("split n=%d offset=%d" % (n, offset))
    rng = np.random.default_rng(n)
    x = rng.standard_normal(n + offset).astype(np.float32)
    xt = torch.from_numpy(x).cuda()[offset:]
    hi = torch.empty(n + 1, dtype=torch.uint16, device="cuda")[1:]
    lo = torch.empty(n + 1, dtype=torch.uint16, device="cuda")[1:]
    heal.heal_split_f32(xt, hi, lo)
    torch.cuda.synchronize()
    hi_o, lo_o = orc.split(x[offset:])
    assert np.array_equal(hi.cpu().numpy(), hi_o)
    assert np.array_equal(lo.cpu().numpy(), lo_o)

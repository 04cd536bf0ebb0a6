"""A seeded sweep of random shapes through the packed-weight products.

Each case draws M and N (half of them 130..600, half log-uniform over
1..130), K (1..300), a weight scale, padded leading dimensions of A and C
and an A base pointer that is 4- but not always 16-byte aligned.  For
HEAL-Base and HEAL-Full (the packed FP16 weight) every forced instance must
give the bits of the automatic choice, leave the padding of C untouched and
meet the oracle's bars (the normwise one on outputs of
256 elements or more); the product with the pre-split B must equal
heal_gemm_f32 on the same operands bit for bit, on every instance.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from gpu_util import announce, check_tolerance, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]

INSTANCES = [heal.INSTANCE_LARGE, heal.INSTANCE_MEDIUM, heal.INSTANCE_SKINNY]
CASES = 128


def _draw(i):
    rng = np.random.default_rng(9000 + i)

    def size():
        if rng.random() < 0.5:
            return int(rng.integers(130, 601))
        return max(1, int(np.exp(rng.uniform(0.0, np.log(130.0)))))

    M, N = size(), size()
    K = int(rng.integers(1, 301))
    sigma_w = float(rng.choice([0.02, 1.0, 40.0]))
    pad_a, pad_c = (int(x) for x in rng.integers(0, 6, size=2))
    off = int(rng.integers(0, 2))
    return rng, M, N, K, sigma_w, pad_a, pad_c, off


def _padded(rows, cols, pad, off, fill):
    ld = cols + pad
    buf = torch.full((off + rows * ld,), fill, device="cuda")
    return buf, buf[off:].view(rows, ld)[:, :cols]


@pytest.mark.parametrize("case", range(CASES))
def test_random_packed_products(orc, case):
    rng, M, N, K, sigma_w, pad_a, pad_c, off = _draw(case)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * sigma_w).astype(np.float32)     # N x K weight
    what = "case %d: %dx%dx%d, weight sigma %g, lda +%d, ldc +%d, offset %d" % (
        case, M, N, K, sigma_w, pad_a, pad_c, off)
    announce(what)
    _, Ad = _padded(M, K, pad_a, off, 0.0)
    Ad.copy_(to_dev(A))
    Wd = to_dev(W)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    W16 = heal.heal_pack_f16_weight(Wd, e)
    w16 = np.asarray(orc.f16_weights(W, e), np.uint16).view(np.float16).astype(np.float64)
    absprod = np.ldexp(np.abs(A.astype(np.float64)) @ np.abs(w16).T, -e)

    for products in (1, 2):
        def run(instance):
            Cbuf, Cd = _padded(M, N, pad_c, off, float("nan"))
            heal.heal_gemm_f16w(Ad, W16, N, e, products, out=Cd, instance=instance)
            torch.cuda.synchronize()
            return Cbuf, Cd

        ref_buf, ref = run(heal.INSTANCE_AUTO)
        pad_mask = torch.ones_like(ref_buf, dtype=torch.bool)
        pad_mask[off:].view(M, N + pad_c)[:, :N] = False
        pad_mask[:off] = True
        assert torch.isnan(ref_buf[pad_mask]).all(), "%s p%d: padding of C written" % (what, products)
        bits = ref.contiguous().view(torch.int32)
        for inst in INSTANCES:
            got_buf, got = run(inst)
            assert torch.isnan(got_buf[pad_mask]).all(), \
                "%s p%d: instance %d wrote the padding" % (what, products, inst)
            assert torch.equal(got.contiguous().view(torch.int32), bits), \
                "%s p%d: instance %d differs from the automatic choice" % (what, products, inst)
        _, S = orc.gemm_f16w(A, W, e, products)
        check_tolerance(ref.cpu().numpy(), S, absprod, "%s p%d" % (what, products),
                        normwise_min_elements=256)

    # the pre-split B (B = W^T, K x N) against heal_gemm_f32 on the same operands
    Bd = Wd.t().contiguous()
    Bp = heal.heal_presplit_b(Bd)
    C0 = heal.heal_gemm_f32(Ad, Bd)
    torch.cuda.synchronize()
    for inst in [heal.INSTANCE_AUTO] + INSTANCES:
        Cp = heal.heal_gemm_f32_presplit(Ad, Bp, N, instance=inst)
        torch.cuda.synchronize()
        assert torch.equal(Cp.view(torch.int32), C0.view(torch.int32)), \
            "%s: pre-split product on instance %d differs from heal_gemm_f32" % (what, inst)

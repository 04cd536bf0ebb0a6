"""A seeded sweep of random shapes and layouts through every kernel instance.

Each case draws M and N (half of them 130..600, half log-uniform over
1..130), K (0..300), a batch of 1 to
3, B stored K x N or N x K, alpha, leading dimensions padded beyond the
width, batch strides with gaps, and base pointers that are 4- but not always
16-byte aligned.  The automatic choice and every forced instance must give
the same bits (the reduction order is the same in all of them), leave the
padding of C untouched, and meet the oracle's bars (the normwise one on outputs of
256 elements or more) on every batch entry
(K = 0 must write alpha * (+0), the empty sum scaled in the epilogue).
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from gpu_util import abs_product, announce, check_tolerance, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]

INSTANCES = [heal.INSTANCE_LARGE, heal.INSTANCE_MEDIUM, heal.INSTANCE_SKINNY]
ALPHAS = [1.0, 0.125, -2.5, float(np.float32(1.0 / np.sqrt(128.0)))]
CASES = 160


def _draw(i):
    rng = np.random.default_rng(7000 + i)
    def size():
        # half of the sizes up to two tiles and a ragged tail (130..600),
        # half log-uniform over 1..130 (the skinny and single-tile range)
        if rng.random() < 0.5:
            return int(rng.integers(130, 601))
        return max(1, int(np.exp(rng.uniform(0.0, np.log(130.0)))))

    M, N = size(), size()
    K = int(rng.integers(0, 301)) if rng.random() < 0.92 else 0
    batch = int(rng.integers(1, 4))
    trans_b = bool(rng.integers(0, 2))
    alpha = ALPHAS[int(rng.integers(0, len(ALPHAS)))]
    pads = [int(x) for x in rng.integers(0, 6, size=3)]
    gaps = [int(x) for x in rng.integers(0, 7, size=3)]
    off = int(rng.integers(0, 2))
    return rng, M, N, K, batch, trans_b, alpha, pads, gaps, off


def _layout(rows, cols, pad, gap, batch, off):
    ld = max(cols, 1) + pad
    stride = rows * ld + gap
    return ld, stride, off + batch * stride


@pytest.mark.parametrize("case", range(CASES))
def test_random_shape_all_instances(orc, case):
    rng, M, N, K, batch, trans_b, alpha, pads, gaps, off = _draw(case)
    rb, cb = (N, K) if trans_b else (K, N)
    lda, sA, nA = _layout(M, K, pads[0], gaps[0], batch, off)
    ldb, sB, nB = _layout(rb, cb, pads[1], gaps[1], batch, off)
    ldc, sC, nC = _layout(M, N, pads[2], gaps[2], batch, off)
    Abuf = rng.standard_normal(nA).astype(np.float32)
    Bbuf = rng.standard_normal(nB).astype(np.float32)
    Ad = torch.from_numpy(Abuf).cuda().as_strided((batch, M, K), (sA, lda, 1), off)
    Bd = torch.from_numpy(Bbuf).cuda().as_strided((batch, rb, cb), (sB, ldb, 1), off)
    what = "case %d: batch %d, %dx%dx%d, trans_b %d, alpha %g, ld %d/%d/%d, offset %d" % (
        case, batch, M, N, K, trans_b, alpha, lda, ldb, ldc, off)
    announce(what)

    def run(instance):
        Cbuf = torch.full((nC,), float("nan"), device="cuda")
        Cd = Cbuf.as_strided((batch, M, N), (sC, ldc, 1), off)
        if instance is None:
            heal.heal_gemm_f32_strided_batched(Ad, Bd, alpha=alpha, trans_b=trans_b, out=Cd)
        else:
            heal.heal_gemm_f32_instance(instance, Ad, Bd, alpha=alpha, trans_b=trans_b, out=Cd)
        torch.cuda.synchronize()
        return Cbuf

    ref = run(None)
    mask = torch.zeros(nC, dtype=torch.bool, device="cuda")
    mask.as_strided((batch, M, N), (sC, ldc, 1), off).fill_(True)
    assert torch.isnan(ref[~mask]).all(), "%s: padding of C written" % what
    ref_bits = ref[mask].view(torch.int32)
    for inst in INSTANCES:
        got = run(inst)
        assert torch.isnan(got[~mask]).all(), "%s: instance %d wrote the padding" % (what, inst)
        assert torch.equal(got[mask].view(torch.int32), ref_bits), \
            "%s: instance %d differs from the automatic choice" % (what, inst)

    C = ref.cpu().numpy()
    a32 = float(np.float32(alpha))
    for b in range(batch):
        Cb = np.lib.stride_tricks.as_strided(C[off + b * sC:], (M, N), (4 * ldc, 4))
        if K == 0:
            # an empty sum is +0, scaled once by alpha in the epilogue:
            # -0 for a negative alpha, as for any exactly-zero sum
            assert (Cb == 0).all() and (np.signbit(Cb) == (a32 < 0)).all(), \
                "%s: K = 0 must write alpha * (+0)" % what
            continue
        A = np.lib.stride_tricks.as_strided(Abuf[off + b * sA:], (M, K), (4 * lda, 4))
        Bs = np.lib.stride_tricks.as_strided(Bbuf[off + b * sB:], (rb, cb), (4 * ldb, 4))
        B = np.ascontiguousarray(Bs.T) if trans_b else np.ascontiguousarray(Bs)
        _, S = orc.gemm3(np.ascontiguousarray(A), B, alpha=alpha)
        check_tolerance(Cb, a32 * S, abs(a32) * abs_product(A, B), "%s, entry %d" % (what, b),
                        normwise_min_elements=256)

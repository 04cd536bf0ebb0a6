"""The short-K panel kernel: products with B stored N x K and K <= 128 (the
attention scores), bf16x3 and INT16 scores.

Shapes span ragged row panels (M not a multiple of the panel height: 256
rows for bf16x3, 128 for the scores), ragged column steps (N not a multiple
of 128), every K depth from one to four 32-deep chunks with a K tail,
batches, the smallest shapes the kernel takes (one panel of rows, N = 4,
K = 4 or 8) and one bf16x3 shape below a panel (130 rows, tiled kernels).
Each output is compared element by element with the oracle's FP64 sum
under the usual bars and bit for bit with the tiled kernels, which run the
same products in the same order: the skinny instance for bf16x3 (over 64
rows it runs generic tiles) and, for the scores, the same codes behind a
row pitch that is not a multiple of eight codes (the panel kernel needs
16-byte rows, so those go to the tiled kernel).
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from gpu_util import abs_product, announce, check_tolerance, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]

BF16X3_SHAPES = [(2, 258, 132, 36), (3, 384, 260, 64), (1, 257, 2052, 124), (2, 256, 512, 128),
                 (1, 256, 4, 4), (2, 520, 136, 96), (1, 1000, 1000, 100), (2, 130, 132, 36)]
SCORE_SHAPES = [(2, 130, 136, 40), (3, 384, 264, 128), (1, 129, 2052, 64), (1, 128, 8, 8),
                (2, 256, 1028, 96)]


@pytest.mark.parametrize("shape", BF16X3_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_panel_bf16x3(orc, shape):
    bat, M, N, K = shape
    rng = np.random.default_rng(M + 3 * N + 7 * K)
    A = rng.standard_normal((bat, M, K)).astype(np.float32)
    Bt = rng.standard_normal((bat, N, K)).astype(np.float32)
    alpha = float(np.float32(1.0 / np.sqrt(K)))
    Ad, Bd = to_dev(A), to_dev(Bt)
    assert heal.select_instance(M, N) != heal.INSTANCE_SKINNY
    announce("panel bf16x3 %s" % (shape,))
    C = heal.heal_gemm_f32_strided_batched(Ad, Bd, alpha=alpha, trans_b=True)
    announce("panel bf16x3 tiled reference %s" % (shape,))
    Ct = heal.heal_gemm_f32_instance(heal.INSTANCE_SKINNY, Ad, Bd, alpha=alpha, trans_b=True)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int32), Ct.view(torch.int32)), "panel differs from tiles"
    Cn = C.cpu().numpy()
    for b in range(bat):
        Bb = np.ascontiguousarray(Bt[b].T)
        _, S = orc.gemm3(A[b], Bb, alpha=alpha)
        check_tolerance(Cn[b], alpha * S, alpha * abs_product(A[b], Bb), "panel %s b%d" % (shape, b))


@pytest.mark.parametrize("shape", SCORE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_panel_scores(orc, shape):
    bat, M, N, K = shape
    rng = np.random.default_rng(M + 5 * N + 11 * K)
    Q = rng.integers(-32767, 32768, size=(bat, M, K)).astype(np.int16)
    Kt = rng.integers(-32767, 32768, size=(bat, N, K)).astype(np.int16)
    mq, mk, alpha = np.float32(3.5), np.float32(0.625), 0.125
    mqd, mkd = torch.tensor([mq], device="cuda"), torch.tensor([mk], device="cuda")
    Qd, Kd = to_dev(Q), to_dev(Kt)
    announce("panel scores %s" % (shape,))
    S = heal.heal_scores_i16(Qd, Kd, mqd, mkd, alpha)
    # the same codes with a row pitch of K + 1: not 16-byte rows, tiled kernel
    Qp = torch.zeros((bat, M, K + 1), dtype=torch.int16, device="cuda")[:, :, :K]
    Qp.copy_(Qd)
    announce("panel scores tiled reference %s" % (shape,))
    St = heal.heal_scores_i16(Qp, Kd, mqd, mkd, alpha)
    torch.cuda.synchronize()
    assert torch.equal(S.view(torch.int32), St.view(torch.int32)), "panel differs from tiles"
    f = orc.scores_factor(mq, mk, alpha)
    Sn = S.cpu().numpy()
    for b in range(bat):
        _, So = orc.scores_i16(Q[b], Kt[b], mq, mk, alpha)
        absprod = abs(f) * (np.abs(Q[b].astype(np.float64)) @ np.abs(Kt[b].astype(np.float64)).T)
        check_tolerance(Sn[b], f * So, absprod, "panel scores %s b%d" % (shape, b))

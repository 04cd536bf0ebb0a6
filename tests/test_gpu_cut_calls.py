"""Calls larger than one launch.

A dispatch counts its work-items in 32 bits, so the library runs a call whose
output exceeds 2^21 blocks of 16 x 16 (over its batch entries) as several
launches over ranges of batch entries, rows (multiples of 256) and columns
(2^20 at a time).  Every kernel sums each output element in the same K order,
so the cut must not change a bit.  Each case checks, on the GPU, the parts on
both sides of a cut against a separate smaller call that covers them with
other part boundaries (bit for bit), and sampled elements against the oracle
under the usual bars.  Two cases are the largest shapes of their kind that a
single launch could not hold (a 2^28-column decode row, 2^23 + 1 batch entries
of the short-K panel kernel); they need several GiB of device memory.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from gpu_util import abs_product, announce, check_tolerance, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]

CUT_COLS = 1 << 20


def _bits(t):
    return t.contiguous().view(torch.int32)


def _gen(seed):
    return torch.Generator(device="cuda").manual_seed(seed)


def _free_gib():
    free, _ = torch.cuda.mem_get_info()
    return free / float(1 << 30)


@pytest.fixture(autouse=True)
def _release():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_cut_batch_attention(orc):
    """130 heads of 2048 x 2048 x 64: 2^21 blocks hold 128 heads, so the call
    is cut after head 127 (bf16x3 with B stored N x K and alpha)."""
    bat, M, N, K = 130, 2048, 2048, 64
    g = _gen(31)
    Q = torch.randn((bat, M, K), device="cuda", generator=g)
    Kh = torch.randn((bat, N, K), device="cuda", generator=g)
    alpha = float(np.float32(0.125))
    announce("cut batch: bf16x3 %d x %dx%dx%d" % (bat, M, N, K))
    S = heal.heal_gemm_f32_strided_batched(Q, Kh, alpha=alpha, trans_b=True)
    for b in (0, 127, 128, 129):
        Sb = heal.heal_gemm_f32_strided_batched(Q[b:b + 1], Kh[b:b + 1], alpha=alpha, trans_b=True)
        assert torch.equal(_bits(S[b]), _bits(Sb[0])), "head %d differs from a one-head call" % b
    rows = [0, 777, 2047]
    for b in (127, 129):
        A = Q[b].cpu().numpy()
        Bb = np.ascontiguousarray(Kh[b].cpu().numpy().T)
        _, So = orc.gemm3(A, Bb, alpha=alpha, rows=rows)
        check_tolerance(S[b, rows].cpu().numpy(), alpha * So, alpha * abs_product(A[rows], Bb),
                        "cut batch head %d" % b)


def test_cut_batch_scores(orc):
    """The INT16 scores of the same 130 heads."""
    bat, M, N, K = 130, 2048, 2048, 64
    g = _gen(32)
    Q = torch.randint(-32767, 32768, (bat, M, K), device="cuda", generator=g, dtype=torch.int16)
    Kt = torch.randint(-32767, 32768, (bat, N, K), device="cuda", generator=g, dtype=torch.int16)
    mq, mk, alpha = np.float32(2.5), np.float32(0.75), 0.125
    mqd, mkd = torch.tensor([mq], device="cuda"), torch.tensor([mk], device="cuda")
    announce("cut batch: INT16 scores %d x %dx%dx%d" % (bat, M, N, K))
    S = heal.heal_scores_i16(Q, Kt, mqd, mkd, alpha)
    for b in (0, 127, 128, 129):
        Sb = heal.heal_scores_i16(Q[b:b + 1], Kt[b:b + 1], mqd, mkd, alpha)
        assert torch.equal(_bits(S[b]), _bits(Sb[0])), "head %d differs from a one-head call" % b
    f = orc.scores_factor(mq, mk, alpha)
    rows = [0, 1031, 2047]
    for b in (127, 128):
        Qb, Kb = Q[b].cpu().numpy(), Kt[b].cpu().numpy()
        _, So = orc.scores_i16(Qb, Kb, mq, mk, alpha, rows=rows)
        absprod = abs(f) * (np.abs(Qb[rows].astype(np.float64)) @ np.abs(Kb.astype(np.float64)).T)
        check_tolerance(S[b, rows].cpu().numpy(), f * So, absprod, "cut scores head %d" % b)


def test_cut_columns(orc):
    """3 x (2^20 + 1028) x 36 (a K tail): cut after column 2^20, for bf16x3,
    the pre-split B (bitwise equal to bf16x3) and HEAL-Full."""
    M, N, K = 3, CUT_COLS + 1028, 36
    rng = np.random.default_rng(33)
    A = rng.standard_normal((M, K)).astype(np.float32)
    Ad = to_dev(A)
    B = torch.randn((K, N), device="cuda", generator=_gen(34)) * 0.02
    announce("cut columns: bf16x3 %dx%dx%d" % (M, N, K))
    C = heal.heal_gemm_f32(Ad, B)
    n0 = CUT_COLS - 512
    Cr = heal.heal_gemm_f32(Ad, B[:, n0:])
    assert torch.equal(_bits(C[:, n0:]), _bits(Cr)), "columns across the cut differ"
    cols = np.r_[0:8, n0 - 8:n0 + 8, CUT_COLS - 8:CUT_COLS + 8, N - 8:N]
    Bs = B[:, torch.from_numpy(cols).cuda()].cpu().numpy()
    _, So = orc.gemm3(A, Bs)
    check_tolerance(C[:, torch.from_numpy(cols).cuda()].cpu().numpy(), So, abs_product(A, Bs),
                    "cut columns bf16x3")

    announce("cut columns: pre-split B")
    Bp = heal.heal_presplit_b(B)
    Cp = heal.heal_gemm_f32_presplit(Ad, Bp, N)
    assert torch.equal(_bits(Cp), _bits(C)), "pre-split product differs from bf16x3"
    del Bp, Cp

    announce("cut columns: HEAL-Full")
    W = B.t().contiguous()
    e = heal.heal_f16_weight_exponent(float(W.abs().max().item()))
    W16 = heal.heal_pack_f16_weight(W, e)
    Cf = heal.heal_gemm_f16w(Ad, W16, N, e, 2)
    block_vals = ((K + 31) // 32) * 512            # one column block of the packed weight
    Cfr = heal.heal_gemm_f16w(Ad, W16[(n0 // 16) * block_vals:], N - n0, e, 2)
    assert torch.equal(_bits(Cf[:, n0:]), _bits(Cfr)), "HEAL-Full columns across the cut differ"


def test_cut_rows(orc):
    """(2^17 + 300) x 4096 x 8: 2^21 blocks hold 2^17 rows of 4096 columns."""
    M, N, K = (1 << 17) + 300, 4096, 8
    g = _gen(35)
    A = torch.randn((M, K), device="cuda", generator=g)
    B = torch.randn((K, N), device="cuda", generator=g)
    announce("cut rows: bf16x3 %dx%dx%d" % (M, N, K))
    C = heal.heal_gemm_f32(A, B)
    m0 = (1 << 17) - 256
    Cr = heal.heal_gemm_f32(A[m0:], B)
    assert torch.equal(_bits(C[m0:]), _bits(Cr)), "rows across the cut differ"
    rows = np.array([0, m0, (1 << 17) - 1, 1 << 17, M - 1])
    Ah = A[torch.from_numpy(rows).cuda()].cpu().numpy()
    Bh = B.cpu().numpy()
    _, So = orc.gemm3(Ah, Bh)
    check_tolerance(C[torch.from_numpy(rows).cuda()].cpu().numpy(), So, abs_product(Ah, Bh),
                    "cut rows")


def test_max_columns_decode_row(orc):
    """1 x (2^28 + 4) x 4: one 16-column workgroup per block would be 2^24 + 1
    workgroups, more work-items than one dispatch counts (B 4 GiB, C 1 GiB)."""
    if _free_gib() < 8:
        pytest.skip("needs 8 GiB of free device memory")
    M, N, K = 1, (1 << 28) + 4, 4
    A = torch.tensor([[1.5, -0.25, 3.0, 0.5]], device="cuda")
    B = torch.randn((K, N), device="cuda", generator=_gen(36))
    announce("max columns: bf16x3 %dx%dx%d" % (M, N, K))
    C = heal.heal_gemm_f32(A, B)
    n0 = N - 4100
    Cr = heal.heal_gemm_f32(A, B[:, n0:])
    assert torch.equal(_bits(C[:, n0:]), _bits(Cr)), "last columns differ"
    cols = np.r_[0:4, CUT_COLS - 4:CUT_COLS + 4, 7 * CUT_COLS + 100:7 * CUT_COLS + 104, N - 8:N]
    idx = torch.from_numpy(cols).cuda()
    Ah, Bs = A.cpu().numpy(), B[:, idx].cpu().numpy()
    _, So = orc.gemm3(Ah, Bs)
    check_tolerance(C[:, idx].cpu().numpy(), So, abs_product(Ah, Bs), "max columns")


def test_max_batch_panel(orc):
    """(2^23 + 1) entries of 256 x 4 x 4 with B stored N x K (the short-K
    panel kernel, two workgroups per entry: 2^24 + 2 workgroups of 256
    threads in one launch would exceed the count).  A and B are one matrix
    each with batch stride 0; C takes 32 GiB."""
    bat, M, N, K = (1 << 23) + 1, 256, 4, 4
    if _free_gib() < 36:
        pytest.skip("needs 36 GiB of free device memory")
    rng = np.random.default_rng(37)
    A = rng.standard_normal((M, K)).astype(np.float32)
    Bt = rng.standard_normal((N, K)).astype(np.float32)
    Ad = to_dev(A).unsqueeze(0).expand(bat, M, K)
    Bd = to_dev(Bt).unsqueeze(0).expand(bat, N, K)
    assert Ad.stride(0) == 0 and Bd.stride(0) == 0
    announce("max batch panel: %d x %dx%dx%d" % (bat, M, N, K))
    C = heal.heal_gemm_f32_strided_batched(Ad, Bd, trans_b=True)
    first = _bits(C[0])
    step = 1 << 18
    for b0 in range(0, bat, step):
        part = C[b0:b0 + step].view(-1, M * N).view(torch.int32)
        assert bool((part == first.view(1, -1)).all()), "an entry in [%d, %d) differs" % (b0, b0 + step)
    Bb = np.ascontiguousarray(Bt.T)
    _, So = orc.gemm3(A, Bb)
    check_tolerance(C[bat - 1].cpu().numpy(), So, abs_product(A, Bb), "max batch panel")

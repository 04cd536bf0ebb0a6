"""Accuracy against the exact product, beside the native FP32 and bf16 GEMMs.

The method's claim (Section 4, GEMM paragraph) is FP32-level accuracy from
16-bit matrix units.  On sampled rows of each workload the exact product of
the FP32 inputs is formed in FP64 on the host (a plain numpy matmul of the
widened inputs), and three GPU results are compared with it:
  * the compensated product (heal_gemm_f32);
  * the native FP32 GEMM (torch.matmul, TF32 off, highest precision);
  * a single bf16 product (both operands cast, FP32 accumulation).
The oracle's FP64 sum of the three bf16 products separates the compensated
product's error into the method's own truncation (the dropped lo*lo product
and the rounding of lo) and the kernel's FP32 accumulation.  The bars: the
compensated product stays within 1e-5 normwise of the exact product and at
least 30 times closer to it than the single bf16 product; the figures are
printed for the record.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from paper_2606_21023_amd import workloads as wl
from gpu_util import announce, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]


def _normwise(X, E):
    return float(np.linalg.norm(np.asarray(X, np.float64) - E) / np.linalg.norm(E))


def _rows(M, n, seed):
    rng = np.random.default_rng(1000 + seed)
    return np.array(sorted({0, M - 1} | set(rng.choice(M, min(n, M), replace=False).tolist())))


@pytest.fixture
def fp32_matmul():
    tf32 = torch.backends.cuda.matmul.allow_tf32
    prec = torch.get_float32_matmul_precision()
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.set_float32_matmul_precision("highest")
    yield
    torch.backends.cuda.matmul.allow_tf32 = tf32
    torch.set_float32_matmul_precision(prec)


def _report(name, rows, heal_c, fp32_c, bf16_c, S, E):
    e_heal, e_fp32, e_bf16 = _normwise(heal_c, E), _normwise(fp32_c, E), _normwise(bf16_c, E)
    e_method, e_acc = _normwise(S, E), _normwise(heal_c, S)
    print("%s rows %d: normwise error vs exact  bf16x3 %.3g (method %.3g, FP32 accumulation "
          "%.3g)  native FP32 %.3g  bf16 %.3g" % (name, len(rows), e_heal, e_method, e_acc,
                                                  e_fp32, e_bf16))
    assert e_heal <= 1e-5, "%s: compensated product too far from the exact product" % name
    assert 30 * e_heal <= e_bf16, "%s: compensated product not clearly better than bf16" % name
    return e_heal, e_fp32, e_bf16


@pytest.mark.parametrize("name,nrows", [("square256", 256), ("decode", 16), ("prefill_up", 6),
                                        ("square8192", 4), ("lm_head", 3)])
def test_accuracy_vs_exact(orc, fp32_matmul, name, nrows):
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    rows = _rows(w.M, nrows, w.seed)
    announce("accuracy %s %dx%dx%d" % (name, w.M, w.N, w.K))
    Ad, Bd = to_dev(A), to_dev(B)
    idx = torch.from_numpy(rows).cuda()
    heal_c = heal.heal_gemm_f32(Ad, Bd)[idx].cpu().numpy()
    fp32_c = torch.matmul(Ad, Bd)[idx].cpu().numpy()
    bf16_c = torch.matmul(Ad.bfloat16(), Bd.bfloat16()).float()[idx].cpu().numpy()
    del Ad, Bd
    torch.cuda.empty_cache()
    E = A[rows].astype(np.float64) @ B.astype(np.float64)
    _, S = orc.gemm3(A, B, rows=rows)
    _report(name, rows, heal_c, fp32_c, bf16_c, S, E)


def test_accuracy_vs_exact_attention(orc, fp32_matmul):
    """Scores of heads 0 and 31 (alpha applied after the sum on every side)."""
    w = wl.WORKLOADS["attn_scores"]
    Q, Kh = wl.make_inputs(w)
    alpha = float(np.float32(w.alpha))
    announce("accuracy attn_scores")
    Qd, Kd = to_dev(Q), to_dev(Kh)
    C = heal.heal_gemm_f32_strided_batched(Qd, Kd, alpha=w.alpha, trans_b=True)
    for h in (0, 31):
        rows = _rows(w.M, 8, h)
        idx = torch.from_numpy(rows).cuda()
        Kt = Kd[h].t().contiguous()
        heal_c = C[h][idx].cpu().numpy()
        fp32_c = (torch.matmul(Qd[h], Kt) * alpha)[idx].cpu().numpy()
        bf16_c = (torch.matmul(Qd[h].bfloat16(), Kt.bfloat16()).float() * alpha)[idx].cpu().numpy()
        B = np.ascontiguousarray(Kh[h].T)
        E = alpha * (Q[h][rows].astype(np.float64) @ B.astype(np.float64))
        _, S = orc.gemm3(Q[h], B, alpha=w.alpha, rows=rows)
        _report("attn_scores head %d" % h, rows, heal_c, fp32_c, bf16_c, alpha * S, E)

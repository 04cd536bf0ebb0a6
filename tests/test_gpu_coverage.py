"""Whole-output parity of every dedicated kernel on aligned multi-tile shapes.

The sampled full-size checks elsewhere compare a few rows of the benchmark
workloads with the oracle; here every element of an output that spans several
tiles, edge tiles and a K tail is compared with the oracle's FP64 sum, for
each product and each kernel instance.  The shapes are chosen so that the
dispatcher takes the dedicated kernels (16-byte aligned rows, K and N
multiples of 4):

  * 520 x 528 x 296: 3 x 3 large tiles with ragged last row and column of
    tiles and a K tail of 8 (296 = 9 * 32 + 8);
  * 1024 x 1024 x 1024: 4 x 4 whole large tiles, every wave position;
  * 64 x 1024 x 4096: the skinny kernel (one 64-row strip per column block)
    and the narrow skinny op tiles over a long K;
  * 64 x 98304 x 96 and 16 x 98304 x 64: the wide skinny strips (384 and
    more 256-column tiles);
  * 2048 x 14336 x 64: the 224-column tiles of the packed-weight products
    (fewer rounds of workgroups than 256 columns on 256 CUs).

On the large instance the bf16x3 product runs gemm_large8_kernel and the
HEAL-Base, HEAL-Full and pre-split products run gemm_op8_kernel; on the
skinny instance with M <= 64 the bf16x3 product runs gemm_skinny_kernel.
A batch of 3 goes through every instance (both B layouts, with and without
alpha), each entry bitwise equal to the same product run alone and within
the bars of the oracle.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from paper_2606_21023_amd import workloads as wl
from gpu_util import abs_product, announce, check_tolerance, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]

INSTANCES = [heal.INSTANCE_LARGE, heal.INSTANCE_MEDIUM, heal.INSTANCE_SKINNY]
INAME = {heal.INSTANCE_LARGE: "large", heal.INSTANCE_MEDIUM: "medium",
         heal.INSTANCE_SKINNY: "skinny"}

COVER_SHAPES = [(520, 528, 296), (1024, 1024, 1024), (64, 1024, 4096), (64, 98304, 96),
                (16, 98304, 64), (2048, 14336, 64)]

_cache = {}


def _inputs(shape):
    M, N, K = shape
    A = wl.random_matrix((M, K), seed=M + 2 * N + 3 * K)
    A[:, (M + N) % K] *= np.float32(50.0)           # one outlier channel
    B = wl.random_matrix((K, N), seed=M + 5 * N + 7 * K, sigma=0.02)
    return A, B


def _oracle(orc, shape, what):
    key = (shape, what)
    if key not in _cache:
        A, B = _inputs(shape)
        if what == "bf16x3":
            _, S = orc.gemm3(A, B)
            _cache[key] = (S, abs_product(A, B))
        else:
            products = 1 if what == "base" else 2
            W = np.ascontiguousarray(B.T)
            e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
            _, S = orc.gemm_f16w(A, W, e, products)
            w16 = orc.f16_weights(W, e).view(np.float16).astype(np.float64)
            absprod = np.ldexp(np.abs(A.astype(np.float64)) @ np.abs(w16).T, -e)
            _cache[key] = (S, absprod)
    return _cache[key]


def _instances(shape):
    # the skinny instance over 64 rows runs generic 64-row tiles; keep it for
    # the shapes it is meant for
    return [i for i in INSTANCES if i != heal.INSTANCE_SKINNY or shape[0] <= 64 or
            shape == (520, 528, 296)]


@pytest.mark.parametrize("shape", COVER_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_bf16x3_and_presplit_whole_output(orc, shape):
    A, B = _inputs(shape)
    Ad, Bd = to_dev(A), to_dev(B)
    Bp = heal.heal_presplit_b(Bd)
    S, absprod = _oracle(orc, shape, "bf16x3")
    for inst in _instances(shape):
        announce("whole output bf16x3 %s %s" % (INAME[inst], shape))
        C = heal.heal_gemm_f32_instance(inst, Ad, Bd)
        announce("whole output presplit %s %s" % (INAME[inst], shape))
        Cp = heal.heal_gemm_f32_presplit(Ad, Bp, shape[1], instance=inst)
        torch.cuda.synchronize()
        nw, ew = check_tolerance(C.cpu().numpy(), S, absprod, "bf16x3 %s %s" % (INAME[inst], shape))
        print("bf16x3 %s %s normwise %.3g elementwise %.3g" % (INAME[inst], shape, nw, ew))
        assert torch.equal(Cp.view(torch.int32), C.view(torch.int32)), "pre-split differs"


@pytest.mark.parametrize("products", [1, 2], ids=["base", "full"])
@pytest.mark.parametrize("shape", COVER_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_f16w_whole_output(orc, shape, products):
    A, B = _inputs(shape)
    W = np.ascontiguousarray(B.T)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    Ad = to_dev(A)
    S, absprod = _oracle(orc, shape, "base" if products == 1 else "full")
    outs = []
    for inst in _instances(shape):
        announce("whole output f16w p%d %s %s" % (products, INAME[inst], shape))
        C = heal.heal_gemm_f16w(Ad, W16, shape[1], e, products, instance=inst)
        torch.cuda.synchronize()
        nw, ew = check_tolerance(C.cpu().numpy(), S, absprod,
                                 "f16w p%d %s %s" % (products, INAME[inst], shape))
        print("f16w p%d %s %s normwise %.3g elementwise %.3g" % (products, INAME[inst], shape,
                                                                  nw, ew))
        outs.append(C)
    for C in outs[1:]:
        assert torch.equal(C.view(torch.int32), outs[0].view(torch.int32)), "instances differ"


def test_scores_large_tiles_whole_output(orc):
    """INT16 scores on a shape above 2048^2 outputs (the 128 x 256 tiles of
    the large instance), every element against the oracle."""
    M, N, K = 2304, 2048, 128
    rng = np.random.default_rng(123)
    Q = rng.integers(-32767, 32768, size=(M, K)).astype(np.int16)
    Kt = rng.integers(-32767, 32768, size=(N, K)).astype(np.int16)
    mq, mk, alpha = np.float32(4.75), np.float32(5.5), float(wl.ATTN_SCALE)
    assert heal.select_instance(M, N) == heal.INSTANCE_LARGE
    announce("whole output scores large %dx%dx%d" % (M, N, K))
    S = heal.heal_scores_i16(to_dev(Q), to_dev(Kt), torch.tensor([mq], device="cuda"),
                             torch.tensor([mk], device="cuda"), alpha)
    torch.cuda.synchronize()
    _, So = orc.scores_i16(Q, Kt, mq, mk, alpha)
    f = orc.scores_factor(mq, mk, alpha)
    absprod = abs(f) * (np.abs(Q.astype(np.float64)) @ np.abs(Kt.astype(np.float64)).T)
    check_tolerance(S.cpu().numpy(), f * So, absprod, "scores large")


@pytest.mark.parametrize("trans_b,alpha", [(False, 1.0), (True, float(wl.ATTN_SCALE)),
                                           (False, 0.375)], ids=["b", "bt-alpha", "b-alpha"])
def test_batch3_every_instance(orc, trans_b, alpha):
    """A batch of 3 through every instance (the large kernel's batch loop on
    grid y, strided operands): each entry bitwise equal to the entry run
    alone, all instances bitwise equal, and each entry within the bars."""
    bat, M, N, K = 3, 520, 264, 136
    rng = np.random.default_rng(7 + trans_b)
    A = rng.standard_normal((bat, M, K)).astype(np.float32)
    B = rng.standard_normal((bat, N, K) if trans_b else (bat, K, N)).astype(np.float32)
    Ad, Bd = to_dev(A), to_dev(B)
    a32 = float(np.float32(alpha))
    ref = None
    for inst in INSTANCES:
        announce("batch 3 %s trans_b=%d alpha=%g" % (INAME[inst], trans_b, alpha))
        C = heal.heal_gemm_f32_instance(inst, Ad, Bd, alpha=alpha, trans_b=trans_b)
        torch.cuda.synchronize()
        for b in range(bat):
            Cb = heal.heal_gemm_f32_instance(inst, Ad[b:b + 1], Bd[b:b + 1], alpha=alpha,
                                             trans_b=trans_b)
            torch.cuda.synchronize()
            assert torch.equal(Cb[0].view(torch.int32), C[b].view(torch.int32)), \
                "%s entry %d differs from its own run" % (INAME[inst], b)
        if ref is None:
            ref = C
            for b in range(bat):
                Bb = np.ascontiguousarray(B[b].T) if trans_b else B[b]
                _, S = orc.gemm3(A[b], Bb, alpha=alpha)
                check_tolerance(C[b].cpu().numpy(), a32 * S, a32 * abs_product(A[b], Bb),
                                "batch entry %d" % b)
        else:
            assert torch.equal(C.view(torch.int32), ref.view(torch.int32)), \
                "%s differs from large" % INAME[inst]


SUBNORMAL_CLASSES = [
    # name, scale of A, scale of B: what falls below 2^-126
    ("lo_subnormal", 2.0 ** -119, 1.0),     # lo of A (about 2^-9 |a|) is bf16-subnormal
    ("hi_subnormal", 2.0 ** -130, 1.0),     # hi and lo of A are subnormal
    ("products_subnormal", 2.0 ** -64, 2.0 ** -66),   # every product and sum is subnormal
]


@pytest.mark.parametrize("name,sa,sb", SUBNORMAL_CLASSES, ids=[c[0] for c in SUBNORMAL_CLASSES])
def test_subnormal_operands(orc, name, sa, sb):
    """bf16-subnormal operand parts and FP32-subnormal products and sums (the
    workloads never reach them) through every instance: the bf16 MFMA keeps
    subnormal inputs and subnormal FP32 results (measured on MI355X: no
    flush, errors 1.6e-7 to 2.8e-7 of |A||B|), so the oracle, which keeps
    every subnormal, holds the GPU to the usual bars; all instances give the
    same bits.  The error figures are printed for the record."""
    M, N, K = 96, 80, 64
    A = (wl.random_matrix((M, K), seed=301) * np.float32(sa)).astype(np.float32)
    B = (wl.random_matrix((K, N), seed=302) * np.float32(sb)).astype(np.float32)
    _, S = orc.gemm3(A, B)
    absAB = abs_product(A, B)
    outs = []
    for inst in INSTANCES:
        announce("subnormal record %s %s" % (name, INAME[inst]))
        C = heal.heal_gemm_f32_instance(inst, to_dev(A), to_dev(B))
        torch.cuda.synchronize()
        Cn = C.cpu().numpy().astype(np.float64)
        err = np.abs(Cn - S)
        ratio = float(np.max(err / np.where(absAB > 0, absAB, 1.0)))
        rel = float(np.linalg.norm(Cn - S) / max(np.linalg.norm(S), 1e-300))
        print("[subnormal-record] %s %s: normwise %.3g, max |C-S|/(|A||B|) %.3g, "
              "zero outputs %d of %d, oracle zeros %d"
              % (name, INAME[inst], rel, ratio, int(np.sum(Cn == 0)), Cn.size, int(np.sum(S == 0))))
        check_tolerance(Cn, S, absAB, "subnormal %s %s" % (name, INAME[inst]))
        outs.append(C)
    for C in outs[1:]:
        assert torch.equal(C.view(torch.int32), outs[0].view(torch.int32)), "instances differ"

"""Every product captured into a HIP graph and replayed.

A serving loop captures its launch-bound steps into HIP graphs.  The
library's calls only launch kernels on the caller's stream (no allocation,
no memset, no wait for the host), so they can be captured: here each call is
recorded into a `torch.cuda.CUDAGraph` with preallocated outputs, the graph
is replayed several times with eager work and synchronizations in between
and the outputs cleared before each replay, and every replay's output must
equal the eager call's output bit for bit.  The INT16 codes take their
maximum through a reduction word that a kernel of the call clears, so a
replay starts from a cleared word like an eager call.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from paper_2606_21023_amd import workloads as wl
from gpu_util import announce, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]

REPLAYS = 3


def _bits(t):
    """The tensor's bits as a flat integer view (comparable and clearable)."""
    t = t.view(-1)
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    if t.dtype == torch.uint16:
        return t.view(torch.int16)
    return t


def _replay_matches(run, outs, what):
    """run() writes every tensor of `outs`; eager result vs graph replays."""
    outs = [_bits(o) for o in outs]
    announce("graph %s: eager" % what)
    run()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    for o in outs:
        o.zero_()
    torch.cuda.synchronize()
    announce("graph %s: capture" % what)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        # eager work and a synchronization between replays
        x = torch.randn(1024, 1024, device="cuda")
        heal.heal_gemm_f32(x, x)
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        announce("graph %s: replay %d" % (what, r))
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, ref):
            assert torch.equal(o, e), "%s: replay %d differs from the eager call" % (what, r)


@pytest.mark.parametrize("M,N,K", [(16, 4096, 4096), (300, 257, 100), (1024, 1024, 256)],
                         ids=["decode", "misaligned", "square1024"])
def test_graph_gemm_f32(M, N, K):
    A = to_dev(wl.random_matrix((M, K), seed=M + K))
    B = to_dev(wl.random_matrix((K, N), seed=N + K, sigma=0.02))
    C = torch.empty((M, N), device="cuda")
    _replay_matches(lambda: heal.heal_gemm_f32(A, B, out=C), [C], "gemm_f32 %dx%dx%d" % (M, N, K))


def test_graph_attention_scores_panel():
    """The short-K panel kernel (bf16x3, B stored N x K, alpha) and the INT16
    codes and scores of the same heads."""
    bat, M, N, K = 2, 512, 1024, 128
    rng = np.random.default_rng(5)
    Q = to_dev(rng.standard_normal((bat, M, K)).astype(np.float32))
    Kh = to_dev(rng.standard_normal((bat, N, K)).astype(np.float32))
    S = torch.empty((bat, M, N), device="cuda")
    _replay_matches(lambda: heal.heal_gemm_f32_strided_batched(Q, Kh, alpha=float(wl.ATTN_SCALE),
                                                               trans_b=True, out=S),
                    [S], "attention bf16x3")
    q = torch.empty((bat, M, K), dtype=torch.int16, device="cuda")
    k = torch.empty((bat, N, K), dtype=torch.int16, device="cuda")
    mq = torch.empty(1, device="cuda")
    mk = torch.empty(1, device="cuda")
    S16 = torch.empty((bat, M, N), device="cuda")

    def scores():
        heal.heal_quantize_i16(Q.view(-1), q=q.view(-1), maxabs=mq)
        heal.heal_quantize_i16(Kh.view(-1), q=k.view(-1), maxabs=mk)
        heal.heal_scores_i16(q, k, mq, mk, float(wl.ATTN_SCALE), out=S16)
    _replay_matches(scores, [q, k, mq, mk, S16], "INT16 codes and scores")


def test_graph_split_presplit_and_f16w():
    M, N, K = 64, 2048, 1024
    A = to_dev(wl.random_matrix((M, K), seed=11))
    B = to_dev(wl.random_matrix((K, N), seed=12, sigma=0.02))
    hi = torch.empty(K * N, dtype=torch.uint16, device="cuda")
    lo = torch.empty(K * N, dtype=torch.uint16, device="cuda")
    _replay_matches(lambda: heal.heal_split_f32(B.view(-1), hi=hi, lo=lo), [hi, lo], "split_f32")
    Bp = heal.heal_presplit_b(B)
    Cp = torch.empty((M, N), device="cuda")
    _replay_matches(lambda: heal.heal_gemm_f32_presplit(A, Bp, N, out=Cp), [Cp], "presplit")
    W = B.t().contiguous()
    e = heal.heal_f16_weight_exponent(float(W.abs().max().item()))
    W16 = heal.heal_pack_f16_weight(W, e)
    for products in (1, 2):
        Cf = torch.empty((M, N), device="cuda")
        _replay_matches(lambda: heal.heal_gemm_f16w(A, W16, N, e, products, out=Cf), [Cf],
                        "f16w products=%d" % products)

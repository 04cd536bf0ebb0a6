"""One GPU's share of a sharded layer, and the bits of its shards.

Split over GPUs by columns of B (tensor parallel, A replicated) or by rows
of A (data parallel), the product needs no exchange of partial sums, and
every output element keeps its K order; so each shard's output must equal
the matching block of the unsharded product bit for bit.  Each shard's
operand here is a separate contiguous copy, as a GPU holding only its shard
would store it, and the shards run as separate calls (the smaller shapes
can take other kernels than the whole product).  The shard workloads at
their real shapes (one of eight column shards of lm_head and of the prefill
up-projection) are also checked against the oracle on sampled rows.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from paper_2606_21023_amd import workloads as wl
from gpu_util import abs_product, announce, check_tolerance, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]


def _bits(t):
    return t.contiguous().view(torch.int32)


@pytest.mark.parametrize("name", ["lm_head", "prefill_up"])
def test_column_shards_bitwise(name):
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    Ad, Bd = to_dev(A), to_dev(B)
    announce("column shards %s: whole product" % name)
    C = heal.heal_gemm_f32(Ad, Bd)
    shards = 8
    ns = w.N // shards
    assert ns * shards == w.N
    for s in range(shards):
        Bs = Bd[:, s * ns:(s + 1) * ns].contiguous()
        announce("column shards %s: shard %d of %d (%dx%dx%d)" % (name, s, shards, w.M, ns, w.K))
        Cs = heal.heal_gemm_f32(Ad, Bs)
        assert torch.equal(_bits(Cs), _bits(C[:, s * ns:(s + 1) * ns])), "shard %d differs" % s


@pytest.mark.parametrize("name,shards", [("prefill_up", 4), ("decode", 16)])
def test_row_shards_bitwise(name, shards):
    """Data parallel over token rows: 4 shards of 512 prefill rows, and the
    16 decode rows one per shard."""
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    Ad, Bd = to_dev(A), to_dev(B)
    announce("row shards %s: whole product" % name)
    C = heal.heal_gemm_f32(Ad, Bd)
    ms = w.M // shards
    for s in range(shards):
        As = Ad[s * ms:(s + 1) * ms].contiguous()
        announce("row shards %s: shard %d of %d (%dx%dx%d)" % (name, s, shards, ms, w.N, w.K))
        Cs = heal.heal_gemm_f32(As, Bd)
        assert torch.equal(_bits(Cs), _bits(C[s * ms:(s + 1) * ms])), "shard %d differs" % s


@pytest.mark.parametrize("name,nrows", [("lm_head_tp8", 4), ("prefill_up_tp8", 6)])
def test_shard_workload_sampled(orc, name, nrows):
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    announce("shard workload %s %dx%dx%d" % (name, w.M, w.N, w.K))
    C = heal.heal_gemm_f32(to_dev(A), to_dev(B))
    torch.cuda.synchronize()
    rng = np.random.default_rng(w.seed)
    rows = np.array(sorted({0, w.M - 1} | set(rng.choice(w.M, nrows, replace=False).tolist())))
    Cr = C[torch.from_numpy(rows).cuda()].cpu().numpy()
    _, S = orc.gemm3(A, B, rows=rows)
    nw, ew = check_tolerance(Cr, S, abs_product(A[rows], B), name)
    print("%s rows %s normwise %.3g elementwise %.3g" % (name, rows.tolist(), nw, ew))


@pytest.mark.parametrize("name", ["lm_head", "prefill_up"])
def test_packed_weight_column_shards_bitwise(name):
    """The packed-weight products (HEAL-Full, HEAL-Base, pre-split B) split
    8 ways by columns: a shard of the packed operand is the contiguous range
    of its 16-column blocks; each shard, packed on its own from its slice of
    the weight as a GPU holding only that slice would (with the whole
    weight's power-of-two scale, which the shards share), equals its block
    of the whole product bit for bit."""
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    Ad, Bd = to_dev(A), to_dev(B)
    W = Bd.t().contiguous()                      # the N x K weight of the layer
    e = heal.heal_f16_weight_exponent(float(W.abs().max().item()))
    shards = 8
    ns = w.N // shards
    W16 = heal.heal_pack_f16_weight(W, e)
    Bp = heal.heal_presplit_b(Bd)
    for products in (1, 2):
        announce("packed shards %s: HEAL f16w products=%d" % (name, products))
        C = heal.heal_gemm_f16w(Ad, W16, w.N, e, products)
        for s in range(shards):
            Ws = heal.heal_pack_f16_weight(W[s * ns:(s + 1) * ns].contiguous(), e)
            Cs = heal.heal_gemm_f16w(Ad, Ws, ns, e, products)
            assert torch.equal(_bits(Cs), _bits(C[:, s * ns:(s + 1) * ns])), \
                "f16w products=%d shard %d differs" % (products, s)
    announce("packed shards %s: pre-split" % name)
    C = heal.heal_gemm_f32_presplit(Ad, Bp, w.N)
    for s in range(shards):
        Bps = heal.heal_presplit_b(Bd[:, s * ns:(s + 1) * ns].contiguous())
        Cs = heal.heal_gemm_f32_presplit(Ad, Bps, ns)
        assert torch.equal(_bits(Cs), _bits(C[:, s * ns:(s + 1) * ns])), "pre-split shard %d differs" % s

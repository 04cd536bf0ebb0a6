"""FP16 forms (HEAL-Base, HEAL-Full), the pre-split operand and the INT16
score product on the GPU, against the CPU oracle.

Parity bars as for the bf16x3 GEMM (gpu_util): the GPU differs from the
oracle's FP64 sums only by FP32 accumulation, so normwise <= 2e-6 and
elementwise |C - S| <= 1e-5 (|A||W16|)_ij 2^-e (|Q||K|^T f for the scores).
Element-wise operations (the HEAL-Full pair, FP16 weights, pre-split planes,
max|x|, INT16 codes) are compared bit for bit.  Invariants: 10 repeated runs,
every M for the same row, every kernel instance, and the pre-split product
against heal_gemm_f32, all bitwise.
"""
import numpy as np
import pytest
import torch

import paper_2606_21023_amd as heal
from paper_2606_21023_amd import workloads as wl
from gpu_util import announce, check_tolerance, needs_gpu, to_dev

pytestmark = [pytest.mark.gpu, needs_gpu]

INSTANCES = [heal.INSTANCE_LARGE, heal.INSTANCE_MEDIUM, heal.INSTANCE_SKINNY]
INAME = {heal.INSTANCE_LARGE: "large", heal.INSTANCE_MEDIUM: "medium",
         heal.INSTANCE_SKINNY: "skinny"}


def unpack(packed, K, N, planes):
    """Inverse of the packed layout (include/heal.h): (planes, N, K) uint16."""
    KC, NB = (K + 31) // 32, (N + 15) // 16
    a = np.asarray(packed).reshape(NB, KC, planes, 4, 16, 8)   # [jb, kc, p, g, r, t]
    a = a.transpose(2, 0, 4, 1, 3, 5).reshape(planes, NB * 16, KC * 32)
    full = a
    assert np.all(full[:, N:, :] == 0) and np.all(full[:, :, K:] == 0), "padding is not +0"
    return full[:, :N, :K]


def f16_values(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


def _isnanh(h):
    return np.isnan(np.asarray(h, np.uint16).view(np.float16))


# ---------------------------------------------------------------------------
# the HEAL-Full pair, exhaustively
# ---------------------------------------------------------------------------
def test_split_f16_exhaustive_vs_oracle(orc):
    chunk = 1 << 28
    for start in range(0, 1 << 32, chunk):
        announce("split_f16 exhaustive chunk 0x%08x" % start)
        bits = torch.arange(start, start + chunk, dtype=torch.int64, device="cuda").to(torch.int32)
        hi, lo = heal.heal_split_f16(bits.view(torch.float32))
        torch.cuda.synchronize()
        hg, lg = hi.cpu().numpy(), lo.cpu().numpy()
        ho, lo_o = orc.split_f16_range(start, chunk)
        assert np.array_equal(_isnanh(hg), _isnanh(ho)), "NaN-ness of hi differs"
        assert np.array_equal(_isnanh(lg), _isnanh(lo_o)), "NaN-ness of lo differs"
        ok = ~(_isnanh(ho) | _isnanh(lo_o))
        bad = np.nonzero((hg[ok] != ho[ok]) | (lg[ok] != lo_o[ok]))[0]
        if bad.size:
            i = np.nonzero(ok)[0][bad[0]]
            raise AssertionError("f16 pair differs at x=0x%08x: gpu (%04x,%04x) oracle (%04x,%04x)"
                                 % ((start + i) & 0xffffffff, hg[i], lg[i], ho[i], lo_o[i]))


@pytest.mark.parametrize("n,offset", [(1, 0), (9, 1), (1000003, 3)])
def test_split_f16_sizes(orc, n, offset):
    announce("split_f16 n=%d offset=%d" % (n, offset))
    x = wl.random_matrix((n + offset,), seed=n, sigma=300.0)
    hi = torch.empty(n + 1, dtype=torch.uint16, device="cuda")[1:]
    lo = torch.empty(n + 1, dtype=torch.uint16, device="cuda")[1:]
    heal.heal_split_f16(to_dev(x)[offset:], hi, lo)
    torch.cuda.synchronize()
    ho, lo_o = orc.split_f16(x[offset:])
    assert np.array_equal(hi.cpu().numpy(), ho) and np.array_equal(lo.cpu().numpy(), lo_o)


# ---------------------------------------------------------------------------
# max|x|, weight exponent and packing
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("rows,cols,pad", [(1, 1, 0), (7, 13, 3), (300, 4096, 0), (1, 1000001, 0),
                                           (0, 5, 0)])
def test_maxabs(orc, rows, cols, pad):
    announce("maxabs %dx%d pad %d" % (rows, cols, pad))
    buf = wl.random_matrix((max(rows, 1), cols + pad), seed=rows + cols, sigma=3.0)
    if rows * cols:
        buf[rows // 2, cols // 3] = -77.5
    x = buf[:rows, :cols]
    xd = to_dev(buf)[:rows, :cols]
    m = heal.heal_maxabs_f32(xd)
    torch.cuda.synchronize()
    assert m.item() == float(orc.maxabs(x)), (m.item(), orc.maxabs(x))


PACK_SHAPES = [(1, 1), (16, 32), (17, 33), (100, 70), (257, 1000), (4096, 64)]


@pytest.mark.parametrize("N,K", PACK_SHAPES, ids=lambda s: str(s))
def test_pack_f16_weight(orc, N, K):
    W = wl.random_matrix((N, K), seed=N * 3 + K, sigma=0.02)
    W[0, 0] = 0.0
    if N * K > 2:
        W.flat[1] = -3e-8          # lands in the FP16 subnormal range after scaling
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    assert e == orc.f16_weight_exponent(float(np.abs(W).max()))
    announce("pack f16 weight %dx%d e=%d" % (N, K, e))
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    torch.cuda.synchronize()
    got = unpack(W16.cpu().numpy(), K, N, 1)[0]
    assert np.array_equal(got, orc.f16_weights(W, e)), "packed FP16 weights differ"


@pytest.mark.parametrize("K,N", [(1, 1), (33, 17), (1000, 257), (64, 4096)], ids=lambda s: str(s))
@pytest.mark.parametrize("trans", [False, True])
def test_presplit_pack(orc, K, N, trans):
    B = wl.random_matrix((K, N), seed=K + 7 * N)
    announce("presplit pack K=%d N=%d trans=%s" % (K, N, trans))
    Bsrc = np.ascontiguousarray(B.T) if trans else B
    Bp = heal.heal_presplit_b(to_dev(Bsrc), trans_b=trans)
    torch.cuda.synchronize()
    planes = unpack(Bp.cpu().numpy(), K, N, 2)
    hi, lo = orc.split(B.T)                     # (N, K) element (n, k) = B[k, n]
    assert np.array_equal(planes[0], hi) and np.array_equal(planes[1], lo)


# ---------------------------------------------------------------------------
# HEAL-Base / HEAL-Full GEMM
# ---------------------------------------------------------------------------
def f16w_case(M, N, K, seed, sigma_w=0.02, outliers=True):
    A = wl.random_matrix((M, K), seed=seed)
    if outliers and K >= 10:
        A[:, seed % K] *= np.float32(50.0)
    W = wl.random_matrix((N, K), seed=seed + 1, sigma=sigma_w)
    return A, W


def run_f16w(A, W, products, instance=heal.INSTANCE_AUTO):
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()) if W.size else 0.0)
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    C = heal.heal_gemm_f16w(to_dev(A), W16, W.shape[0], e, products, instance=instance)
    torch.cuda.synchronize()
    return C.cpu().numpy(), e


def f16w_absprod(orc, A, W, e):
    w16 = f16_values(orc.f16_weights(W, e))
    return np.ldexp(np.abs(A.astype(np.float64)) @ np.abs(w16).T, -e)


F16_SHAPES = [(1, 1, 1), (15, 16, 17), (16, 16, 32), (17, 31, 33), (33, 100, 257), (64, 300, 1000),
              (65, 129, 96), (255, 257, 257), (300, 64, 64), (520, 530, 300)]


@pytest.mark.parametrize("products", [1, 2], ids=["base", "full"])
@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
@pytest.mark.parametrize("shape", F16_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_f16w_parity(orc, products, instance, shape):
    M, N, K = shape
    A, W = f16w_case(M, N, K, seed=M + 3 * N + 7 * K)
    announce("f16w products=%d %s %s" % (products, INAME[instance], shape))
    C, e = run_f16w(A, W, products, instance)
    _, S = orc.gemm_f16w(A, W, e, products)
    check_tolerance(C, S, f16w_absprod(orc, A, W, e), "f16w p%d %s" % (products, shape))


@pytest.mark.parametrize("products", [1, 2], ids=["base", "full"])
def test_f16w_integer_exact(orc, products):
    """|a| <= 2^11 and |w| <= 32 (e = 10): every product and partial sum is an
    integer below 2^24, so any order gives the exact integer GEMM."""
    rng = np.random.default_rng(40)
    for (M, N, K) in ((17, 33, 31), (300, 257, 64), (16, 512, 40)):
        A = rng.integers(-2048, 2049, size=(M, K)).astype(np.float32)
        W = rng.integers(-32, 33, size=(N, K)).astype(np.float32)
        W[0, 0] = 32.0
        announce("f16w integer exact p%d %s" % (products, (M, N, K)))
        C, e = run_f16w(A, W, products)
        assert e == 10
        exact = (A.astype(np.int64) @ W.astype(np.int64).T)
        assert np.abs(exact).max() < 2 ** 24
        assert np.array_equal(C, exact.astype(np.float32))


def test_f16w_k_zero_and_empty():
    announce("f16w K=0 / empty")
    A = torch.empty((5, 0), device="cuda")
    C = heal.heal_gemm_f16w(A, torch.empty(0, dtype=torch.uint16, device="cuda"), 7, 0, 2)
    torch.cuda.synchronize()
    assert torch.equal(C, torch.zeros_like(C))
    C = heal.heal_gemm_f16w(torch.empty((0, 4), device="cuda"),
                            torch.zeros(512, dtype=torch.uint16, device="cuda"), 3, 0, 2)
    assert C.shape == (0, 3)


def _rows(M, n, seed):
    rng = np.random.default_rng(seed)
    r = {0, M - 1} | set(rng.choice(M, min(n, M), replace=False).tolist())
    return np.array(sorted(r), dtype=np.int64)


@pytest.mark.parametrize("name,nrows", [("decode", 16), ("prefill_up", 4), ("lm_head", 3),
                                        ("square8192", 3)])
def test_f16w_workloads_sampled(orc, name, nrows):
    """The linear-layer workloads at full size, W = B^T (a linear layer's N x K
    weight), both forms, sampled rows against the oracle."""
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    W = np.ascontiguousarray(B.T)
    del B
    rows = _rows(w.M, nrows, w.seed)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    Ad = to_dev(A)
    w16 = f16_values(orc.f16_weights(W, e))
    absprod = np.ldexp(np.abs(A[rows].astype(np.float64)) @ np.abs(w16).T, -e)
    del w16
    for products in (1, 2):
        announce("f16w workload %s products=%d" % (name, products))
        C = heal.heal_gemm_f16w(Ad, W16, w.N, e, products)
        torch.cuda.synchronize()
        Cr = C[torch.from_numpy(rows).cuda()].cpu().numpy()
        del C
        _, S = orc.gemm_f16w(A, W, e, products, rows=rows)
        nw, ew = check_tolerance(Cr, S, absprod, "%s p%d" % (name, products))
        print("%s products=%d normwise %.3g elementwise %.3g" % (name, products, nw, ew))


@pytest.mark.parametrize("products", [1, 2], ids=["base", "full"])
def test_f16w_bitwise_invariants(products):
    """10 runs, every instance, and rows independent of M (batch invariance)."""
    M, N, K = 300, 1000, 777
    A, W = f16w_case(M, N, K, seed=55)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    Ad = to_dev(A)
    announce("f16w bitwise invariants p%d" % products)
    ref = heal.heal_gemm_f16w(Ad, W16, N, e, products)
    for r in range(10):
        C = heal.heal_gemm_f16w(Ad, W16, N, e, products)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref.view(torch.int32)), "run %d differs" % r
    for inst in INSTANCES:
        C = heal.heal_gemm_f16w(Ad, W16, N, e, products, instance=inst)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref.view(torch.int32)), INAME[inst]
    for m in (1, 2, 15, 16, 17, 33, 63, 64, 65, 127, 128, 129, 255, 256, 299):
        C = heal.heal_gemm_f16w(Ad[:m], W16, N, e, products)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), "M=%d differs" % m


def _large_widths_shapes():
    """Two ragged shapes: one where the large instance keeps 256-column tiles
    and one where 224-column tiles take fewer rounds of workgroups (one
    workgroup per CU; the choice follows the device's CU count)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count

    def cost(M, N, bn):
        wgs = -(-M // 256) * -(-N // bn)
        return -(-wgs // cus) * bn

    tm = max(1, cus // 16)
    wide = (256 * tm - 56, 256 * 16 - 6)                 # tm x 16 tiles: one round
    narrow = (256 * 8 - 48, 224 * (-(-2 * cus // 8 // 8) * 8) - 36)
    assert cost(*wide, 256) < cost(*wide, 224), wide
    assert cost(*narrow, 224) < cost(*narrow, 256), narrow
    return [wide, narrow]


@pytest.mark.parametrize("K", [72, 37, 96])
def test_large_tile_widths(orc, K):
    """Both tile widths of the large instance: the whole output bitwise equal
    to the medium instance (and, pre-split, to heal_gemm_f32), sampled rows
    against the oracle."""
    for (M, N) in _large_widths_shapes():
        A, W = f16w_case(M, N, K, seed=M + N + K)
        e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
        W16 = heal.heal_pack_f16_weight(to_dev(W), e)
        Ad = to_dev(A)
        rows = _rows(M, 6, K)
        absprod = f16w_absprod(orc, A[rows], W, e)
        for products in (1, 2):
            announce("large widths f16w p%d %dx%dx%d" % (products, M, N, K))
            C = heal.heal_gemm_f16w(Ad, W16, N, e, products, instance=heal.INSTANCE_LARGE)
            Cm = heal.heal_gemm_f16w(Ad, W16, N, e, products, instance=heal.INSTANCE_MEDIUM)
            torch.cuda.synchronize()
            assert torch.equal(C.view(torch.int32), Cm.view(torch.int32)), "large != medium"
            _, S = orc.gemm_f16w(A, W, e, products, rows=rows)
            check_tolerance(C[torch.from_numpy(rows).cuda()].cpu().numpy(), S, absprod,
                            "large widths p%d %dx%dx%d" % (products, M, N, K))
            del C, Cm
        announce("large widths presplit %dx%dx%d" % (M, N, K))
        Bd = to_dev(np.ascontiguousarray(W.T))
        Bp = heal.heal_presplit_b(Bd)
        Cp = heal.heal_gemm_f32_presplit(Ad, Bp, N, instance=heal.INSTANCE_LARGE)
        C0 = heal.heal_gemm_f32(Ad, Bd)
        torch.cuda.synchronize()
        assert torch.equal(Cp.view(torch.int32), C0.view(torch.int32)), "presplit differs"


# ---------------------------------------------------------------------------
# pre-split B: bitwise equal to heal_gemm_f32
# ---------------------------------------------------------------------------
PRESPLIT_SHAPES = [(1, 1, 1), (17, 31, 33), (64, 300, 1000), (255, 257, 257), (520, 530, 300)]


@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
@pytest.mark.parametrize("shape", PRESPLIT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_presplit_bitwise_equal(orc, instance, shape):
    M, N, K = shape
    A = wl.random_matrix((M, K), seed=M + K)
    B = wl.random_matrix((K, N), seed=N + K)
    Ad, Bd = to_dev(A), to_dev(B)
    announce("presplit %s %s" % (INAME[instance], shape))
    Bp = heal.heal_presplit_b(Bd)
    Cp = heal.heal_gemm_f32_presplit(Ad, Bp, N, instance=instance)
    C0 = heal.heal_gemm_f32(Ad, Bd)
    torch.cuda.synchronize()
    assert torch.equal(Cp.view(torch.int32), C0.view(torch.int32)), "differs from heal_gemm_f32"
    Bpt = heal.heal_presplit_b(Bd.t().contiguous(), trans_b=True)
    torch.cuda.synchronize()
    assert torch.equal(Bpt, Bp), "packing of the transposed storage differs"


@pytest.mark.parametrize("name", ["decode", "lm_head", "prefill_up", "square8192"])
def test_presplit_workloads_bitwise(name):
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    Ad, Bd = to_dev(A), to_dev(B)
    del B
    announce("presplit workload %s" % name)
    Bp = heal.heal_presplit_b(Bd)
    C0 = heal.heal_gemm_f32(Ad, Bd)
    del Bd
    Cp = heal.heal_gemm_f32_presplit(Ad, Bp, w.N)
    torch.cuda.synchronize()
    assert torch.equal(Cp.view(torch.int32), C0.view(torch.int32))


# ---------------------------------------------------------------------------
# INT16 codes and dual-FP16 scores
# ---------------------------------------------------------------------------
def test_f16w_and_presplit_a_rows_past_2gib(orc):
    """A leading dimension that puts A's byte offsets past 2^31: every
    instance of both FP16 forms and of the pre-split product bitwise equal to
    the same call on a compact A, and the FP16 forms within the oracle
    bound."""
    M, N, K = 65, 300, 96
    big = (1 << 23) + 32
    A, W = f16w_case(M, N, K, seed=123)
    Ac = to_dev(A)
    full = torch.zeros((M, big), device="cuda")
    full[:, :K] = Ac
    Aw = full[:, :K]
    assert (M - 1) * big * 4 >= 2 ** 31
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    Bd = to_dev(np.ascontiguousarray(W.T))
    Bp = heal.heal_presplit_b(Bd)
    for inst in INSTANCES:
        for products in (1, 2):
            announce("f16w A past 2 GiB p%d %s" % (products, INAME[inst]))
            C = heal.heal_gemm_f16w(Aw, W16, N, e, products, instance=inst)
            C0 = heal.heal_gemm_f16w(Ac, W16, N, e, products, instance=inst)
            torch.cuda.synchronize()
            assert torch.equal(C.view(torch.int32), C0.view(torch.int32)), (products, INAME[inst])
            _, S = orc.gemm_f16w(A, W, e, products)
            check_tolerance(C.cpu().numpy(), S, f16w_absprod(orc, A, W, e),
                            "A past 2 GiB p%d %s" % (products, INAME[inst]))
        announce("presplit A past 2 GiB %s" % INAME[inst])
        Cp = heal.heal_gemm_f32_presplit(Aw, Bp, N, instance=inst)
        Cp0 = heal.heal_gemm_f32_presplit(Ac, Bp, N, instance=inst)
        torch.cuda.synchronize()
        assert torch.equal(Cp.view(torch.int32), Cp0.view(torch.int32)), INAME[inst]
    del full


def test_scores_batch_beyond_grid_limit():
    """INT16 scores with more heads than one grid dimension holds: each head
    bitwise equal to the same head run alone."""
    M, N, d, P, batch = 5, 9, 24, 7, 70001
    rng = np.random.default_rng(77)
    Q7 = torch.from_numpy(rng.integers(-32767, 32768, size=(P, M, d)).astype(np.int16)).cuda()
    K7 = torch.from_numpy(rng.integers(-32767, 32768, size=(P, N, d)).astype(np.int16)).cuda()
    mq = torch.tensor([3.0], device="cuda")
    mk = torch.tensor([0.5], device="cuda")
    idx = (torch.arange(batch) % P).cuda()
    announce("scores batch %d" % batch)
    ref = heal.heal_scores_i16(Q7, K7, mq, mk, alpha=0.125)
    S = heal.heal_scores_i16(Q7[idx].contiguous(), K7[idx].contiguous(), mq, mk, alpha=0.125)
    torch.cuda.synchronize()
    assert torch.equal(S.view(torch.int32), ref[idx].view(torch.int32))


@pytest.mark.parametrize("n,offset", [(1, 0), (7, 1), (4096, 0), (1000003, 2)])
def test_quantize_bitwise(orc, n, offset):
    announce("quantize n=%d offset=%d" % (n, offset))
    x = wl.random_matrix((n + offset,), seed=n + 1, sigma=2.0)
    q = torch.empty(n + 1, dtype=torch.int16, device="cuda")[1:]
    qd, md = heal.heal_quantize_i16(to_dev(x)[offset:], q=q)
    torch.cuda.synchronize()
    qo, mo = orc.quantize_i16(x[offset:])
    assert md.item() == float(mo)
    assert np.array_equal(qd.cpu().numpy(), qo), "INT16 codes differ"


def test_quantize_golden_near_ties(orc):
    """Elements of the attention workload whose exactly rounded code differs
    from an FP32 decision (tests/golden/quantize_i16_cases.txt, exact rational
    codes): the GPU code is the golden one."""
    import pins
    for xb, mb, code in pins.load_quantize_golden():
        x = np.array([xb, mb, xb ^ 0x80000000], np.uint32).view(np.float32)
        announce("quantize golden x=0x%08x m=0x%08x" % (xb, mb))
        q, m = heal.heal_quantize_i16(to_dev(x))
        torch.cuda.synchronize()
        assert m.item() == float(x[1])
        assert q.cpu().numpy().tolist() == [code, 32767, -code], "x=0x%08x" % xb


@pytest.mark.parametrize("m", [40.0, 5.0978498, 1e-3, 4e-35, 1e-36, 2.0 ** -140],
                         ids=lambda v: "%g" % v)
def test_quantize_next_to_ties_and_tiny_maxima(orc, m):
    """Values whose quotient 32767 x / m lies within an ulp of a half-integer,
    for ordinary, tiny (32767 / m overflows FP32) and subnormal maxima: codes
    bitwise equal to the oracle's exact rounding."""
    import pins
    rng = np.random.default_rng(int(abs(np.log2(m))) + 3)
    m32 = np.float32(m)
    x = np.concatenate([np.array([m32, -m32], np.float32),
                        pins.near_half_integer_inputs(rng, m32, 20000),
                        np.clip(rng.standard_normal(5000).astype(np.float32) * (m32 / 4),
                                -m32, m32)])
    announce("quantize next to ties, m=%g n=%d" % (m, x.size))
    qd, md = heal.heal_quantize_i16(to_dev(x))
    torch.cuda.synchronize()
    qo, mo = orc.quantize_i16(x)
    assert md.item() == float(mo) == float(m32)
    assert np.array_equal(qd.cpu().numpy(), qo), "INT16 codes differ"


def test_quantize_all_zero():
    announce("quantize all-zero")
    q, m = heal.heal_quantize_i16(torch.zeros(1000, device="cuda"))
    torch.cuda.synchronize()
    assert m.item() == 0.0 and not q.any()


def scores_case(bat, M, N, K, seed, bound=32767):
    rng = np.random.default_rng(seed)
    Q = rng.integers(-bound, bound + 1, size=(bat, M, K)).astype(np.int16)
    Kt = rng.integers(-bound, bound + 1, size=(bat, N, K)).astype(np.int16)
    return Q, Kt


def scores_absprod(Q, Kt, f):
    return abs(f) * (np.abs(Q.astype(np.float64)) @ np.abs(Kt.astype(np.float64)).T)


def factor(orc, mq, mk, alpha):
    """The oracle's FP64 dequantisation factor alpha (mq/32767)(mk/32767)."""
    return orc.scores_factor(mq, mk, alpha)


# the last two: at most 64 rows and 8196 or 16004 columns, on 32- and
# 64-column tiles
SCORE_SHAPES = [(1, 1, 1, 1), (1, 17, 31, 33), (2, 64, 70, 128), (3, 129, 257, 64),
                (1, 300, 200, 136), (2, 16, 8196, 40), (1, 33, 16004, 64)]


@pytest.mark.parametrize("shape", SCORE_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_scores_parity(orc, shape):
    bat, M, N, K = shape
    Q, Kt = scores_case(bat, M, N, K, seed=M + N + K)
    mq, mk = np.float32(3.5), np.float32(0.625)
    alpha = float(wl.ATTN_SCALE)
    announce("scores %s" % (shape,))
    S = heal.heal_scores_i16(to_dev(Q), to_dev(Kt), torch.tensor([mq], device="cuda"),
                             torch.tensor([mk], device="cuda"), alpha)
    torch.cuda.synchronize()
    S = S.cpu().numpy()
    f = factor(orc, mq, mk, alpha)
    for b in range(bat):
        _, So = orc.scores_i16(Q[b], Kt[b], mq, mk, alpha)
        check_tolerance(S[b], f * So, scores_absprod(Q[b], Kt[b], f), "scores %s b%d" % (shape, b))


def test_scores_integer_exact(orc):
    """Codes |q| <= 2^11 are FP16-exact; with K = 4 every partial sum is below
    2^24, so the scores are exactly f * (integer dot product)."""
    Q, Kt = scores_case(2, 40, 50, 4, seed=7, bound=2048)
    one = torch.tensor([np.float32(32767.0)], device="cuda")      # f = 1 * 1 * alpha
    announce("scores integer exact")
    S = heal.heal_scores_i16(to_dev(Q), to_dev(Kt), one, one, 1.0)
    torch.cuda.synchronize()
    exact = np.einsum("bmk,bnk->bmn", Q.astype(np.int64), Kt.astype(np.int64))
    assert np.array_equal(S.cpu().numpy(), exact.astype(np.float32))


def test_scores_attention_workload(orc):
    """The attention-score shape end to end: FP32 Q, K of 32 heads quantized on
    the GPU (codes bitwise against the oracle), then the dual-FP16 scores with
    the 1/sqrt(128) scale, sampled rows against the oracle; 10 runs and every
    M bitwise equal."""
    w = wl.WORKLOADS["attn_scores"]
    Qf, Kf = wl.make_inputs(w)
    announce("scores workload: quantize")
    Qd, Kd = to_dev(Qf), to_dev(Kf)
    q, mq = heal.heal_quantize_i16(Qd)
    k, mk = heal.heal_quantize_i16(Kd)
    torch.cuda.synchronize()
    qo, mqo = orc.quantize_i16(Qf)
    ko, mko = orc.quantize_i16(Kf)
    assert mq.item() == float(mqo) and mk.item() == float(mko)
    assert np.array_equal(q.cpu().numpy(), qo) and np.array_equal(k.cpu().numpy(), ko)
    announce("scores workload: scores")
    S = heal.heal_scores_i16(q, k, mq, mk, w.alpha)
    torch.cuda.synchronize()
    f = factor(orc, mqo, mko, w.alpha)
    for h in (0, 17, 31):
        rows = _rows(w.M, 4, h)
        Sr = S[h][torch.from_numpy(rows).cuda()].cpu().numpy()
        _, So = orc.scores_i16(qo[h], ko[h], mqo, mko, w.alpha, rows=rows)
        check_tolerance(Sr, f * So, scores_absprod(qo[h][rows], ko[h], f), "head %d" % h)
    announce("scores workload: bitwise invariants")
    for r in range(10):
        S2 = heal.heal_scores_i16(q, k, mq, mk, w.alpha)
        torch.cuda.synchronize()
        assert torch.equal(S2.view(torch.int32), S.view(torch.int32)), "run %d" % r
    for m in (1, 15, 16, 17, 127, 128, 129, 1000, 2047):
        S3 = heal.heal_scores_i16(q[:, :m].contiguous(), k, mq, mk, w.alpha)
        torch.cuda.synchronize()
        assert torch.equal(S3.view(torch.int32), S[:, :m].view(torch.int32)), "M=%d" % m


@pytest.mark.parametrize("products", [1, 2], ids=["base", "full"])
@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
def test_f16w_padded_and_misaligned(orc, products, instance):
    """Leading dimensions above the width, A's base off 16 bytes (scalar load
    path), C padded: the padding of C is untouched."""
    M, N, K = 70, 90, 77
    lda, ldc = K + 5, N + 7
    rng = np.random.default_rng(6)
    Abuf = (rng.standard_normal(M * lda + 1) * 2.0).astype(np.float32)
    A = Abuf[1:].reshape(M, lda)[:, :K]
    W = wl.random_matrix((N, K), seed=8, sigma=0.02)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    W16 = heal.heal_pack_f16_weight(to_dev(W), e)
    Ad = torch.from_numpy(Abuf).cuda()[1:].view(M, lda)[:, :K]
    Cbuf = torch.full((M * ldc + 1,), float("nan"), device="cuda")
    Cd = Cbuf[1:].view(M, ldc)[:, :N]
    announce("f16w padded/misaligned p%d %s" % (products, INAME[instance]))
    heal.heal_gemm_f16w(Ad, W16, N, e, products, out=Cd, instance=instance)
    torch.cuda.synchronize()
    _, S = orc.gemm_f16w(np.ascontiguousarray(A), W, e, products)
    check_tolerance(Cd.cpu().numpy(), S, f16w_absprod(orc, np.ascontiguousarray(A), W, e), "padded")
    assert torch.isnan(Cbuf[1:].view(M, ldc)[:, N:]).all()


def test_scores_padded_rows(orc):
    """Q and K rows with leading dimensions above the head dimension (views
    of wider buffers), batch strides of the views."""
    bat, M, N, K = 2, 40, 50, 64
    Qw, Kw = scores_case(bat, M, N, K + 8, seed=12)
    Qv, Kv = to_dev(Qw)[:, :, :K], to_dev(Kw)[:, :, :K]
    mq, mk = np.float32(1.25), np.float32(2.5)
    announce("scores padded rows")
    S = heal.heal_scores_i16(Qv, Kv, torch.tensor([mq], device="cuda"),
                             torch.tensor([mk], device="cuda"), 0.5)
    torch.cuda.synchronize()
    f = factor(orc, mq, mk, 0.5)
    for b in range(bat):
        Q, Kt = np.ascontiguousarray(Qw[b, :, :K]), np.ascontiguousarray(Kw[b, :, :K])
        _, So = orc.scores_i16(Q, Kt, mq, mk, 0.5)
        check_tolerance(S[b].cpu().numpy(), f * So, scores_absprod(Q, Kt, f), "padded b%d" % b)


def test_f16w_full_wide_weight_range(orc):
    """HEAL-Full with weight columns spread over 2^-20 of the largest weight:
    the residual product's weight fragment is scaled by 2^-10 in FP16, which
    stays exact down to |w16| = 2^-4 and rounds below it, by at most 2^-25
    per weight; the bars still hold over this range."""
    M, N, K = 64, 96, 200
    A = wl.random_matrix((M, K), seed=70, sigma=3.0)
    W = wl.random_matrix((N, K), seed=71, sigma=0.05)
    W *= np.exp2(-np.linspace(0.0, 20.0, N, dtype=np.float32))[:, None].astype(np.float32)
    announce("f16w full, wide weight range")
    C, e = run_f16w(A, W, 2)
    _, S = orc.gemm_f16w(A, W, e, 2)
    check_tolerance(C, S, f16w_absprod(orc, A, W, e), "wide weight range")


@pytest.mark.parametrize("N,K", [(1040, 1028), (300, 40), (272, 4096)],
                         ids=["ragged-n-ktail", "one-stage", "long-k"])
def test_stream_tiles_every_m_bitwise(orc, N, K):
    """Every row count 1..64 through the skinny instance of the packed-weight
    products (the streamed narrow tiles of 16, 32 and 64 rows: a loader /
    compute hand-over through a ring of LDS stages), with a ragged last
    column block, a K tail, a single stage and a K that wraps the ring many
    times: each row bitwise equal to the medium instance's row of the full
    64-row product, and the 64-row results within the oracle's bars."""
    A = wl.random_matrix((64, K), seed=N + K, sigma=2.0)
    W = wl.random_matrix((N, K), seed=N + 3 * K, sigma=0.02)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    Ad, Wd = to_dev(A), to_dev(W)
    W16 = heal.heal_pack_f16_weight(Wd, e)
    Bp = heal.heal_presplit_b(Wd, trans_b=True)
    for products in (1, 2):
        announce("stream tiles every M, f16w p%d N=%d K=%d" % (products, N, K))
        ref = heal.heal_gemm_f16w(Ad, W16, N, e, products, instance=heal.INSTANCE_MEDIUM)
        torch.cuda.synchronize()
        _, S = orc.gemm_f16w(A, W, e, products)
        check_tolerance(ref.cpu().numpy(), S, f16w_absprod(orc, A, W, e), "p%d" % products)
        for m in range(1, 65):
            C = heal.heal_gemm_f16w(Ad[:m], W16, N, e, products, instance=heal.INSTANCE_SKINNY)
            torch.cuda.synchronize()
            assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), \
                "p%d M=%d differs" % (products, m)
    announce("stream tiles every M, pre-split N=%d K=%d" % (N, K))
    ref = heal.heal_gemm_f32_presplit(Ad, Bp, N, instance=heal.INSTANCE_MEDIUM)
    torch.cuda.synchronize()
    for m in range(1, 65):
        C = heal.heal_gemm_f32_presplit(Ad[:m], Bp, N, instance=heal.INSTANCE_SKINNY)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), "pre-split M=%d" % m


@pytest.mark.parametrize("N,K", [(8196, 100), (16004, 68), (30724, 36)],
                         ids=["w32", "w32-w64", "w64-w128"])
def test_mid_width_tiles_every_m_bitwise(orc, N, K):
    """Every row count 1..64 through the skinny instance of the packed-weight
    products where the output is too wide for the streamed 16-column tiles
    and too narrow for 256-column ones: 32-, 64- and 128-column tiles (by
    row count as noted in the ids), ragged last tile, K tail.  Each row
    bitwise equal to the medium instance's, whose 64-row result is checked
    against the oracle."""
    A = wl.random_matrix((64, K), seed=2 * N + K, sigma=2.0)
    W = wl.random_matrix((N, K), seed=N + 7 * K, sigma=0.02)
    e = heal.heal_f16_weight_exponent(float(np.abs(W).max()))
    Ad, Wd = to_dev(A), to_dev(W)
    W16 = heal.heal_pack_f16_weight(Wd, e)
    Bp = heal.heal_presplit_b(Wd, trans_b=True)
    for products in (1, 2):
        announce("mid-width tiles every M, f16w p%d N=%d K=%d" % (products, N, K))
        ref = heal.heal_gemm_f16w(Ad, W16, N, e, products, instance=heal.INSTANCE_MEDIUM)
        torch.cuda.synchronize()
        _, S = orc.gemm_f16w(A, W, e, products)
        check_tolerance(ref.cpu().numpy(), S, f16w_absprod(orc, A, W, e), "p%d" % products)
        for m in range(1, 65):
            C = heal.heal_gemm_f16w(Ad[:m], W16, N, e, products, instance=heal.INSTANCE_SKINNY)
            torch.cuda.synchronize()
            assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), \
                "p%d M=%d differs" % (products, m)
    announce("mid-width tiles every M, pre-split N=%d K=%d" % (N, K))
    ref = heal.heal_gemm_f32_presplit(Ad, Bp, N, instance=heal.INSTANCE_MEDIUM)
    C3 = heal.heal_gemm_f32_instance(heal.INSTANCE_MEDIUM, Ad, Wd.t().contiguous())
    torch.cuda.synchronize()
    assert torch.equal(ref.view(torch.int32), C3.view(torch.int32)), "pre-split differs from bf16x3"
    for m in range(1, 65):
        C = heal.heal_gemm_f32_presplit(Ad[:m], Bp, N, instance=heal.INSTANCE_SKINNY)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), "pre-split M=%d" % m

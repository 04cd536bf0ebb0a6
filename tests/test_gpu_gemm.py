"""heal_gemm_f32 on the GPU against the CPU oracle, and its bitwise invariants.

Parity: element by element against the oracle's FP64 sum on the same seeded
inputs (tolerance bars in gpu_util), exact equality where every partial sum
is an integer below 2^24.  Invariants (GPU against itself): 10 repeated runs,
every M for the same row, every kernel instance, plain vs batched entry points.
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


def gpu_gemm(A, B, instance=None, alpha=1.0, trans_b=False):
    """Run on numpy inputs; B is K x N (or N x K when trans_b); returns numpy C."""
    Ad, Bd = to_dev(A), to_dev(B)
    if instance is None and alpha == 1.0 and not trans_b:
        C = heal.heal_gemm_f32(Ad, Bd)
    else:
        C = heal.heal_gemm_f32_instance(instance or heal.INSTANCE_AUTO, Ad, Bd, alpha=alpha,
                                        trans_b=trans_b)
    torch.cuda.synchronize()
    return C.cpu().numpy()


# ---------------------------------------------------------------------------
# exactness: integer inputs, any summation order gives the exact result
# ---------------------------------------------------------------------------
INT_SHAPES = [(1, 1, 1), (17, 33, 31), (300, 257, 32), (65, 129, 17), (16, 64, 32), (513, 70, 5)]


@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
@pytest.mark.parametrize("shape", INT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_integer_exact(orc, instance, shape):
    M, N, K = shape
    for (ba, bb, seed) in ((2048, 128, 10), (128, 2048, 11)):
        A = wl.integer_matrix((M, K), seed, ba)
        B = wl.integer_matrix((K, N), seed + 100, bb)
        announce("integer exact %s %s bounds %d/%d" % (INAME[instance], shape, ba, bb))
        C = gpu_gemm(A, B, instance)
        exact = (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float32)
        Co, _ = orc.gemm3(A, B)
        assert np.array_equal(Co, exact)
        assert np.array_equal(C, exact), "GPU differs from the exact integer GEMM"


# ---------------------------------------------------------------------------
# tolerance parity on small shapes spanning several tiles and ragged tails
# ---------------------------------------------------------------------------
SHAPES = [(1, 1, 1), (15, 16, 17), (16, 16, 32), (17, 31, 33), (31, 33, 255), (255, 257, 257),
          (257, 255, 129), (64, 300, 1000), (300, 64, 64), (129, 513, 96), (33, 1000, 70),
          (520, 530, 300)]


@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_parity_small(orc, instance, shape):
    M, N, K = shape
    A = wl.random_matrix((M, K), seed=M * 7 + K)
    B = wl.random_matrix((K, N), seed=N * 13 + K)
    announce("parity %s %s" % (INAME[instance], shape))
    C = gpu_gemm(A, B, instance)
    _, S = orc.gemm3(A, B)
    check_tolerance(C, S, abs_product(A, B), "%s %s" % (INAME[instance], shape))


@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
@pytest.mark.parametrize("shape", [(17, 31, 33), (255, 257, 257), (64, 300, 1000)],
                         ids=lambda s: "x".join(map(str, s)))
def test_parity_trans_b_alpha(orc, instance, shape):
    M, N, K = shape
    A = wl.random_matrix((M, K), seed=1 + M)
    Bt = wl.random_matrix((N, K), seed=2 + N)      # stored N x K
    alpha = float(wl.ATTN_SCALE)
    announce("parity trans_b alpha %s %s" % (INAME[instance], shape))
    C = gpu_gemm(A, Bt, instance, alpha=alpha, trans_b=True)
    B = np.ascontiguousarray(Bt.T)
    Co, S = orc.gemm3(A, B, alpha=alpha)
    check_tolerance(C, float(np.float32(alpha)) * S, float(np.float32(alpha)) * abs_product(A, B),
                    "trans_b alpha %s" % (shape,))


@pytest.mark.parametrize("instance", INSTANCES, ids=lambda i: INAME[i])
def test_parity_padded_and_misaligned(orc, instance):
    """Leading dimensions above the width and base pointers off 16 bytes."""
    M, N, K = 70, 90, 77
    lda, ldb, ldc = K + 5, N + 3, N + 7
    rng = np.random.default_rng(5)
    Abuf = rng.standard_normal(M * lda + 1).astype(np.float32)
    Bbuf = rng.standard_normal(K * ldb + 1).astype(np.float32)
    A = Abuf[1:].reshape(M, lda)[:, :K]
    B = Bbuf[1:].reshape(K, ldb)[:, :N]
    Ad = torch.from_numpy(Abuf).cuda()[1:].view(M, lda)[:, :K]
    Bd = torch.from_numpy(Bbuf).cuda()[1:].view(K, ldb)[:, :N]
    Cbuf = torch.full((M * ldc + 1,), float("nan"), device="cuda")
    Cd = Cbuf[1:].view(M, ldc)[:, :N]
    announce("parity padded/misaligned %s" % INAME[instance])
    heal.heal_gemm_f32_instance(instance, Ad, Bd, out=Cd)
    torch.cuda.synchronize()
    _, S = orc.gemm3(A, B)
    check_tolerance(Cd.cpu().numpy(), S, abs_product(A, B), "padded")
    # the padding columns of C are untouched
    assert torch.isnan(Cbuf[1:].view(M, ldc)[:, N:]).all()


def test_k_zero_writes_zero_and_empty_is_noop():
    announce("K=0 and empty products")
    A = torch.empty((5, 0), device="cuda")
    B = torch.empty((0, 7), device="cuda")
    C = torch.full((5, 7), float("nan"), device="cuda")
    heal.heal_gemm_f32(A, B, out=C)
    torch.cuda.synchronize()
    assert torch.equal(C, torch.zeros_like(C))
    assert not torch.signbit(C).any()
    A = torch.ones((0, 4), device="cuda")
    B = torch.ones((4, 3), device="cuda")
    C = heal.heal_gemm_f32(A, B)
    assert C.shape == (0, 3)


def test_nonfinite_inputs_match_oracle(orc):
    """inf/NaN inputs give the oracle's NaN pattern; other outputs stay in tolerance."""
    rng = np.random.default_rng(9)
    A = rng.standard_normal((40, 70)).astype(np.float32)
    B = rng.standard_normal((70, 50)).astype(np.float32)
    A[3, 5] = np.inf
    A[7, 9] = -np.inf
    A[11, 0] = np.nan
    B[20, 13] = np.inf
    B[2, 2] = np.float32(3.4e38)      # finite, but rounds to +inf in bf16
    Co, S = orc.gemm3(A, B)
    fin = np.isfinite(Co)
    assert 0 < fin.sum() < fin.size
    absAB = abs_product(np.where(np.isfinite(A), A, 0), np.where(np.abs(B) < 3e38, B, 0))
    for inst in INSTANCES:
        announce("non-finite inputs %s" % INAME[inst])
        C = gpu_gemm(A, B, inst)
        assert np.array_equal(np.isnan(C), np.isnan(Co)), "NaN pattern differs"
        assert np.array_equal(np.isinf(C), np.isinf(Co)), "inf pattern differs"
        err = np.abs(C[fin].astype(np.float64) - S[fin])
        assert np.all(err <= 1e-5 * absAB[fin])


# ---------------------------------------------------------------------------
# the LLM-layer workloads at full size (sampled rows against the oracle)
# ---------------------------------------------------------------------------
def _rows(M, n, seed):
    rng = np.random.default_rng(seed)
    r = {0, M - 1} | set(rng.choice(M, min(n, M), replace=False).tolist())
    return np.array(sorted(r), dtype=np.int64)


def test_config_square256_full(orc):
    w = wl.WORKLOADS["square256"]
    A, B = wl.make_inputs(w)
    announce("config square256")
    C = gpu_gemm(A, B)
    _, S = orc.gemm3(A, B)
    nw, ew = check_tolerance(C, S, abs_product(A, B), "square256")
    print("square256 normwise %.3g elementwise %.3g" % (nw, ew))


@pytest.mark.parametrize("name,nrows", [("decode", 16), ("prefill_up", 6), ("square8192", 4),
                                        ("lm_head", 3)])
def test_config_full_size_sampled(orc, name, nrows):
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    announce("config %s %dx%dx%d" % (name, w.M, w.N, w.K))
    Ad, Bd = to_dev(A), to_dev(B)
    C = heal.heal_gemm_f32(Ad, Bd)
    torch.cuda.synchronize()
    rows = _rows(w.M, nrows, w.seed)
    Cr = C[torch.from_numpy(rows).cuda()].cpu().numpy()
    del C, Ad, Bd
    _, S = orc.gemm3(A, B, rows=rows)
    nw, ew = check_tolerance(Cr, S, abs_product(A[rows], B), name)
    print("%s rows %s normwise %.3g elementwise %.3g" % (name, rows.tolist(), nw, ew))


def test_config_attention_sampled(orc):
    w = wl.WORKLOADS["attn_scores"]
    Q, Kh = wl.make_inputs(w)
    announce("config attn_scores batched")
    C = heal.heal_gemm_f32_strided_batched(to_dev(Q), to_dev(Kh), alpha=w.alpha, trans_b=True)
    torch.cuda.synchronize()
    alpha = float(np.float32(w.alpha))
    for h in (0, 13, 31):
        rows = _rows(w.M, 4, h)
        Cr = C[h][torch.from_numpy(rows).cuda()].cpu().numpy()
        B = np.ascontiguousarray(Kh[h].T)
        _, S = orc.gemm3(Q[h], B, alpha=w.alpha, rows=rows)
        nw, ew = check_tolerance(Cr, alpha * S, alpha * abs_product(Q[h][rows], B),
                                 "attn head %d" % h)
        print("attn_scores head %d rows %s normwise %.3g elementwise %.3g" % (h, rows.tolist(), nw,
                                                                            ew))


# ---------------------------------------------------------------------------
# bitwise invariants (GPU against itself)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["square8192", "decode", "attn_scores"])
def test_bitwise_repro_10_runs(name):
    w = wl.WORKLOADS[name]
    A, B = wl.make_inputs(w)
    Ad, Bd = to_dev(A), to_dev(B)
    announce("bit-repro x10 %s" % name)
    if name == "attn_scores":
        run = lambda: heal.heal_gemm_f32_strided_batched(Ad, Bd, alpha=w.alpha, trans_b=True)
    else:
        run = lambda: heal.heal_gemm_f32(Ad, Bd)
    ref = run()
    # a concurrent product on another stream must not change the bits
    side = torch.cuda.Stream()
    for r in range(10):
        if r % 2:
            with torch.cuda.stream(side):
                x = torch.randn(2048, 2048, device="cuda")
                heal.heal_gemm_f32(x, x)
        C = run()
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref.view(torch.int32)), "run %d differs" % r


def test_batch_invariance_attention_all_m():
    """Row i of C(Q[:M], K^T) is bitwise the same for every M = 1..2048 (head 0),
    and for a ladder of M on the other heads."""
    w = wl.WORKLOADS["attn_scores"]
    Q, Kh = wl.make_inputs(w)
    Qd, Kd = to_dev(Q), to_dev(Kh)
    announce("batch invariance head 0, M=1..2048")
    full = heal.heal_gemm_f32_strided_batched(Qd, Kd, alpha=w.alpha, trans_b=True)
    fb = full.view(torch.int32)
    for M in range(1, w.M + 1):
        C = heal.heal_gemm_f32_strided_batched(Qd[0:1, :M], Kd[0:1], alpha=w.alpha, trans_b=True)
        assert torch.equal(C.view(torch.int32)[0], fb[0, :M]), "head 0 differs at M=%d" % M
    ladder = [1, 2, 3, 5, 8, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 257,
              511, 512, 1023, 1024, 1025, 2047, 2048]
    announce("batch invariance other heads, ladder of M")
    for M in ladder:
        C = heal.heal_gemm_f32_strided_batched(Qd[:, :M].contiguous(), Kd, alpha=w.alpha,
                                               trans_b=True)
        assert torch.equal(C.view(torch.int32), fb[:, :M]), "heads differ at M=%d" % M


@pytest.mark.parametrize("shape", [(300, 257, 100), (64, 1000, 4096), (1000, 64, 513),
                                   (16, 4096, 512)], ids=lambda s: "x".join(map(str, s)))
def test_instances_bitwise_equal(shape):
    M, N, K = shape
    A = wl.random_matrix((M, K), seed=21)
    B = wl.random_matrix((K, N), seed=22)
    announce("instances bitwise %s" % (shape,))
    outs = [gpu_gemm(A, B, inst) for inst in INSTANCES]
    for inst, C in zip(INSTANCES[1:], outs[1:]):
        assert np.array_equal(C.view(np.int32), outs[0].view(np.int32)), \
            "%s differs from large" % INAME[inst]


# output widths and the strips the skinny kernel takes for them (the widest
# that still gives about one strip per CU at 64 rows, two at 16 or 32 rows),
# each with a ragged last strip and a K tail: 16 columns; 16; 32; 32 at up
# to 32 rows, else 64; 64, else 128; 128, else 256; 256 at every row count
SKINNY_WIDTHS = [(1040, 1028), (300, 520), (8196, 100), (16004, 68), (30724, 36), (61444, 36),
                 (122884, 12)]
SKINNY_WIDTH_IDS = ["s16-ktail", "s16-ragged-n", "s32", "s32-s64", "s64-s128", "s128-s256",
                    "s256"]


@pytest.mark.parametrize("N,K", SKINNY_WIDTHS, ids=SKINNY_WIDTH_IDS)
def test_skinny_every_m_bitwise(N, K):
    """Every row count 1..64 through the skinny instance (16-row, 32-row and
    64-row tiles; strips of 16 to 256 columns), B stored K x N with a K tail
    and a ragged last strip: each row bitwise equal to the medium instance's
    row of the full 64-row product."""
    A = wl.random_matrix((64, K), seed=N + K)
    B = wl.random_matrix((K, N), seed=N + 2 * K)
    Ad, Bd = to_dev(A), to_dev(B)
    announce("skinny every M %dx%d" % (N, K))
    ref = heal.heal_gemm_f32_instance(heal.INSTANCE_MEDIUM, Ad, Bd)
    torch.cuda.synchronize()
    for m in range(1, 65):
        C = heal.heal_gemm_f32_instance(heal.INSTANCE_SKINNY, Ad[:m], Bd)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), "M=%d differs" % m


# outputs the width rule leaves with 16-column strips, which run as 32-column
# strips with their rows in 1, 2 or 4 groups (up to 256 workgroups): ragged
# last strips, a K tail, and group counts that change with M's divisibility
ROW_GROUP_SHAPES = [(2052, 260), (3072, 100), (4100, 36), (5120, 68), (7168, 36)]


@pytest.mark.parametrize("alpha", [1.0, -0.75], ids=["alpha1", "alpha-0.75"])
@pytest.mark.parametrize("trans_b", [False, True], ids=["kxn", "nxk"])
@pytest.mark.parametrize("N,K", ROW_GROUP_SHAPES, ids=lambda v: str(v))
def test_skinny_row_groups_every_m(orc, N, K, trans_b, alpha):
    """Every row count 1..64 through the skinny instance where its rows run
    in groups (B stored K x N, or N x K where more than 32 rows or enough
    strips take them): each row bitwise equal to the medium instance's row of
    the full 64-row product; 16 and 64 rows element by element against the
    oracle."""
    A = wl.random_matrix((64, K), seed=5 * N + K)
    B = wl.random_matrix((K, N), seed=N + 3 * K)
    Ad = to_dev(A)
    Bd = to_dev(np.ascontiguousarray(B.T)) if trans_b else to_dev(B)
    announce("skinny row groups every M %dx%d trans_b %d alpha %g" % (N, K, trans_b, alpha))
    ref = heal.heal_gemm_f32_instance(heal.INSTANCE_MEDIUM, Ad, Bd, alpha=alpha, trans_b=trans_b)
    torch.cuda.synchronize()
    for m in range(1, 65):
        C = heal.heal_gemm_f32_instance(heal.INSTANCE_SKINNY, Ad[:m], Bd, alpha=alpha,
                                        trans_b=trans_b)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[:m].view(torch.int32)), "M=%d differs" % m
    a32 = float(np.float32(alpha))
    for m in (16, 64):
        _, S = orc.gemm3(A[:m], B, alpha=alpha)
        check_tolerance(ref[:m].cpu().numpy(), a32 * S, abs(a32) * abs_product(A[:m], B),
                        "row groups M=%d" % m)


@pytest.mark.parametrize("N,K", SKINNY_WIDTHS[2:], ids=SKINNY_WIDTH_IDS[2:])
def test_skinny_widths_trans_b_alpha(orc, N, K):
    """The wider strips with B stored N x K and alpha, at the row counts
    around the 16-, 32- and 64-row tiles: bitwise equal to the medium
    instance, and the 33-row product element by element against the oracle."""
    A = wl.random_matrix((64, K), seed=3 * N + K)
    Bt = wl.random_matrix((N, K), seed=N + 5 * K)
    alpha = 0.375
    Ad, Bd = to_dev(A)[None], to_dev(Bt)[None]
    announce("skinny widths trans_b %dx%d" % (N, K))
    ref = heal.heal_gemm_f32_instance(heal.INSTANCE_MEDIUM, Ad, Bd, alpha=alpha, trans_b=True)
    torch.cuda.synchronize()
    for m in (1, 15, 16, 17, 32, 33, 63, 64):
        C = heal.heal_gemm_f32_instance(heal.INSTANCE_SKINNY, Ad[:, :m], Bd, alpha=alpha,
                                        trans_b=True)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[:, :m].view(torch.int32)), "M=%d differs" % m
        if m == 33:
            B = np.ascontiguousarray(Bt.T)
            _, S = orc.gemm3(A[:m], B)
            check_tolerance(C[0].cpu().numpy(), alpha * S, alpha * abs_product(A[:m], B),
                            "skinny %d columns trans_b" % N)


@pytest.mark.parametrize("K", [8, 7], ids=["k8", "k7"])
@pytest.mark.parametrize("trans_b", [False, True], ids=["b", "bt"])
def test_batch_beyond_grid_limit(K, trans_b):
    """More batch entries than one grid dimension holds (65535 workgroups,
    two entries per workgroup in the medium instance): every instance walks
    the extra entries, each entry bitwise equal to the same product run in a
    batch of its own."""
    M, N, P, batch = 3, 5, 7, 140001
    rng = np.random.default_rng(K + 2 * trans_b)
    A7 = rng.standard_normal((P, M, K)).astype(np.float32)
    B7 = rng.standard_normal((P, N, K) if trans_b else (P, K, N)).astype(np.float32)
    idx = torch.arange(batch) % P
    Ad = to_dev(A7)[idx.cuda()].contiguous()
    Bd = to_dev(B7)[idx.cuda()].contiguous()
    for inst in INSTANCES:
        announce("batch %d %s K=%d trans_b=%d" % (batch, INAME[inst], K, trans_b))
        ref = heal.heal_gemm_f32_instance(inst, to_dev(A7), to_dev(B7), trans_b=trans_b)
        C = heal.heal_gemm_f32_instance(inst, Ad, Bd, trans_b=trans_b)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref[idx.cuda()].view(torch.int32)), INAME[inst]


@pytest.mark.parametrize("which", ["A", "B", "Bt"])
def test_operands_spanning_more_than_2gib(orc, which):
    """Leading dimensions that put operand byte offsets past 2^31, so that the
    kernels' 32-bit-offset paths have to step aside: every instance bitwise
    equal to the same product on compact operands, and within the bound of
    the oracle."""
    big = (1 << 23) + 32                   # 33.5 MB rows
    trans_b = which == "Bt"
    M, N, K = (65, 256, 64) if which == "A" else (300, 256, 72) if which == "B" else (300, 96, 64)
    A = wl.random_matrix((M, K), seed=91)
    B = wl.random_matrix((N, K) if trans_b else (K, N), seed=92)
    Ac, Bc = to_dev(A), to_dev(B)
    if which == "A":
        full = torch.zeros((M, big), device="cuda")
        full[:, :K] = Ac
        Aw, Bw = full[:, :K], Bc
    else:
        rows = B.shape[0]
        full = torch.zeros((rows, big), device="cuda")
        full[:, :B.shape[1]] = Bc
        Aw, Bw = Ac, full[:, :B.shape[1]]
    assert (Aw.shape[0] - 1) * Aw.stride(0) * 4 >= 2 ** 31 or (Bw.shape[0] - 1) * Bw.stride(0) * 4 >= 2 ** 31
    _, S = orc.gemm3(A, np.ascontiguousarray(B.T) if trans_b else B)
    for inst in INSTANCES:
        announce("operands past 2 GiB: %s %s" % (which, INAME[inst]))
        C = heal.heal_gemm_f32_instance(inst, Aw, Bw, trans_b=trans_b)
        C0 = heal.heal_gemm_f32_instance(inst, Ac, Bc, trans_b=trans_b)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), C0.view(torch.int32)), INAME[inst]
        check_tolerance(C.cpu().numpy(), S,
                        abs_product(A, np.ascontiguousarray(B.T) if trans_b else B),
                        "past 2 GiB %s %s" % (which, INAME[inst]))
    del full


def test_entry_points_bitwise_equal():
    M, N, K = 200, 300, 333
    A = wl.random_matrix((M, K), seed=31)
    B = wl.random_matrix((K, N), seed=32)
    Ad, Bd = to_dev(A), to_dev(B)
    announce("entry points bitwise")
    C0 = heal.heal_gemm_f32(Ad, Bd)
    C1 = heal.heal_gemm_f32_strided_batched(Ad[None], Bd[None], alpha=1.0, trans_b=False)[0]
    C2 = heal.heal_gemm_f32_strided_batched(Ad[None], Bd.t().contiguous()[None], alpha=1.0,
                                            trans_b=True)[0]
    torch.cuda.synchronize()
    assert torch.equal(C0.view(torch.int32), C1.view(torch.int32))
    assert torch.equal(C0.view(torch.int32), C2.view(torch.int32))
    # batch entries are independent products
    A3 = torch.stack([Ad, Ad.flip(0)])
    C3 = heal.heal_gemm_f32_strided_batched(A3, torch.stack([Bd, Bd]))
    torch.cuda.synchronize()
    assert torch.equal(C3[0].view(torch.int32), C0.view(torch.int32))
    assert torch.equal(C3[1].view(torch.int32), C0.flip(0).view(torch.int32))


@pytest.mark.parametrize("M,N,K", [(384, 256, 1000), (256, 384, 512), (300, 260, 640), (256, 256, 4096)],
                         ids=["ring-ktail", "ring-8-stages", "ring-edge-tiles", "ring-deep"])
@pytest.mark.parametrize("trans_b", [False, True], ids=["b", "bt"])
def test_medium_register_ring(orc, M, N, K, trans_b):
    """The medium tiles' register ring (loads two stages ahead, for at least
    8 full 64-deep stages): interior tiles with and without a K tail after
    the ring, edge tiles beside interior ones, both B layouts and alpha.
    Whole output against the oracle and bitwise against the large instance."""
    A = wl.random_matrix((M, K), seed=M + K)
    B = wl.random_matrix((N, K) if trans_b else (K, N), seed=N + 2 * K)
    alpha = 0.625
    Ad, Bd = to_dev(A)[None], to_dev(B)[None]
    announce("medium ring %dx%dx%d trans_b=%d" % (M, N, K, trans_b))
    C = heal.heal_gemm_f32_instance(heal.INSTANCE_MEDIUM, Ad, Bd, alpha=alpha, trans_b=trans_b)
    Cl = heal.heal_gemm_f32_instance(heal.INSTANCE_LARGE, Ad, Bd, alpha=alpha, trans_b=trans_b)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int32), Cl.view(torch.int32)), "medium differs from large"
    Bn = np.ascontiguousarray(B.T) if trans_b else B
    _, S = orc.gemm3(A, Bn)
    check_tolerance(C[0].cpu().numpy(), alpha * S, alpha * abs_product(A, Bn), "medium ring")

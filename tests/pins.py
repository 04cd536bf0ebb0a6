"""Pins for the CPU oracle: checks against what the paper and mathematics fix.

Each ``pin_*`` takes an ``oracle.oracle.Oracle`` and raises AssertionError on a
mismatch.  They never compare the oracle with itself or with the HIP path:

* golden cases derived by hand from the definition of the split and product
  (tests/golden/*.txt);
* the split against an independent RNE conversion (torch's float->bfloat16
  cast) and numpy's FP32 subtraction;
* closed forms: bf16-representable inputs give the plain product; a
  constructed split x = h + l gives exact(A*B) - S = sum lA*lB; small integers
  give the exact integer GEMM;
* a brute-force error bound against the exact rational product on tiny sizes.

The FP16 forms (HEAL-Base, HEAL-Full) and the INT16 score product (HEAL+)
have pins of the same kinds: binary16 rounding against numpy's float16 casts,
hand-derived golden pairs, the defining property of the weight exponent,
closed-form error bounds against exact rational products, integer inputs, the
exact identity hi + lo/2^10 = q of the INT16 unpack, INT16 codes against the
exact rational rounding (golden workload elements and values next to ties),
and the paper's INT16 error and MSE bounds.

The mutation tests run the same pins against oracles with planted mistakes.
"""
import os
from fractions import Fraction

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _bits_f32(x):
    return np.asarray(x, np.float32).view(np.uint32)


def _f32_from_bits(u):
    return np.asarray(u, np.uint32).view(np.float32)


def _bf16_to_f32(h):
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32)


def torch_rne_bf16(x):
    """Library RNE conversion FP32 -> bf16 bit patterns (torch CPU cast)."""
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def reference_split(x):
    """The split's definition evaluated with library primitives.

    hi = RNE_bf16(x) via torch; r = x - hi in numpy FP32 (IEEE, so inf - inf
    is NaN); lo = RNE_bf16(r) via torch.
    """
    x = np.ascontiguousarray(x, np.float32)
    hi = torch_rne_bf16(x)
    with np.errstate(invalid="ignore", over="ignore"):
        r = (x - _bf16_to_f32(hi)).astype(np.float32)
    lo = torch_rne_bf16(r)
    return hi, lo


def _nan16(h):
    return np.isnan(_bf16_to_f32(h))


def _check_split_equal(x, hi, lo, hi_ref, lo_ref, what):
    """Bitwise equality, except that NaNs are compared by NaN-ness only
    (payload and sign of a NaN are not part of the definition)."""
    for name, a, b in (("hi", hi, hi_ref), ("lo", lo, lo_ref)):
        na, nb = _nan16(a), _nan16(b)
        if not np.array_equal(na, nb):
            i = np.nonzero(na != nb)[0][0]
            raise AssertionError("%s: NaN-ness of %s differs at x=0x%08x" % (what, name,
                                                                            _bits_f32(x[i])))
    ok = ~(_nan16(hi_ref) | _nan16(lo_ref))
    bad = np.nonzero((hi[ok] != hi_ref[ok]) | (lo[ok] != lo_ref[ok]))[0]
    if bad.size:
        i = np.nonzero(ok)[0][bad[0]]
        raise AssertionError("%s: split mismatch at x=0x%08x: got (%04x,%04x), expected (%04x,%04x)"
                             % (what, _bits_f32(x[i]), hi[i], lo[i], hi_ref[i], lo_ref[i]))


# --------------------------------------------------------------------------
# split pins
# --------------------------------------------------------------------------

def load_split_golden():
    rows = []
    with open(os.path.join(GOLDEN, "split_cases.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                x, h, l = line.split()
                rows.append((int(x, 16), None if h == "nan" else int(h, 16),
                             None if l == "nan" else int(l, 16)))
    return rows


def pin_golden_split(orc):
    """Hand-derived cases; None (written "nan") accepts any NaN pattern."""
    rows = load_split_golden()
    x = _f32_from_bits(np.array([r[0] for r in rows], np.uint32))
    hi, lo = orc.split(x)
    for (xb, hb, lb), h, l in zip(rows, hi, lo):
        for exp, got, name in ((hb, int(h), "hi"), (lb, int(l), "lo")):
            if exp is None:
                assert _nan16(np.uint16(got)), "golden split x=0x%08x: %s=%04x is not NaN" % (
                    xb, name, got)
            else:
                assert got == exp, "golden split x=0x%08x: %s=%04x, expected %04x" % (
                    xb, name, got, exp)


def structured_patterns():
    """FP32 bit patterns covering every rounding class of the split.

    All 2^16 upper halves combined with lower halves at and around the tie
    (0x7fff, 0x8000, 0x8001), the extremes (0, 1, 0xffff) and a few others.
    """
    upper = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x1234, 0x7fff, 0x8000, 0x8001, 0xbeef, 0xffff], np.uint32)
    return (upper[:, None] | lows[None, :]).ravel()


def pin_split_vs_library(orc, bits=None):
    """The oracle split equals the definition evaluated with library RNE."""
    if bits is None:
        bits = structured_patterns()
    x = _f32_from_bits(bits)
    hi, lo = orc.split(x)
    hi_ref, lo_ref = reference_split(x)
    _check_split_equal(x, hi, lo, hi_ref, lo_ref, "split vs library RNE")


def check_split_range_exhaustive(orc, start, n):
    """Exhaustive form of pin_split_vs_library over bit patterns [start, start+n).

    The reference is evaluated with torch CPU ops (multi-threaded) for speed;
    it is the same definition as ``reference_split``.
    """
    hi, lo = orc.split_range(start, n)
    bits = torch.arange(n, dtype=torch.int64).add_(start).to(torch.int32)
    x = bits.view(torch.float32)
    hi_ref = x.to(torch.bfloat16)
    lo_ref = (x - hi_ref.to(torch.float32)).to(torch.bfloat16).view(torch.int16)
    hi_t = torch.from_numpy(hi.view(np.int16))
    lo_t = torch.from_numpy(lo.view(np.int16))
    what = "exhaustive split [0x%08x,+%d)" % (start, n)
    hn, ln = torch.isnan(hi_t.view(torch.bfloat16)), torch.isnan(lo_t.view(torch.bfloat16))
    hrn, lrn = torch.isnan(hi_ref), torch.isnan(lo_ref.view(torch.bfloat16))
    assert torch.equal(hn, hrn), "%s: NaN-ness of hi differs" % what
    assert torch.equal(ln, lrn), "%s: NaN-ness of lo differs" % what
    bad = ~(hrn | lrn) & ((hi_t != hi_ref.view(torch.int16)) | (lo_t != lo_ref))
    if torch.any(bad):
        i = int(torch.nonzero(bad)[0, 0])
        raise AssertionError("%s: split mismatch at x=0x%08x" % (what, (start + i) & 0xffffffff))


def pin_split_properties(orc, seed=0):
    """Mathematical properties of the split that hold for every finite input.

    * r = x - hi is exact (checked in FP64);
    * |x - hi - lo| <= 2^-17 |x| for normal-range inputs that do not round to inf;
    * bf16-representable x gives hi = x and lo = 0.
    """
    rng = np.random.default_rng(seed)
    # log-uniform magnitudes over the normal range, random signs and low bits
    e = rng.integers(-100, 127, size=200000)
    m = rng.random(200000) + 1.0
    x = (np.where(rng.random(200000) < 0.5, -1.0, 1.0) * m * np.exp2(e)).astype(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) < np.float32(3.3e38))]
    hi, lo = orc.split(x)
    hf = _bf16_to_f32(hi).astype(np.float64)
    lf = _bf16_to_f32(lo).astype(np.float64)
    x64 = x.astype(np.float64)
    assert np.all(np.isfinite(hf)), "hi overflowed on an in-range input"
    r32 = (x - _bf16_to_f32(hi)).astype(np.float64)
    assert np.array_equal(r32, x64 - hf), "x - hi is not exact in FP32"
    err = np.abs(x64 - hf - lf)
    assert np.all(err <= np.ldexp(np.abs(x64), -17)), \
        "split error exceeds 2^-17|x| (max ratio %g)" % np.max(err / np.abs(x64))
    # bf16-representable values
    xb = _bf16_to_f32(hi)
    hb, lb = orc.split(xb)
    assert np.array_equal(hb, hi), "split of a bf16 value changed it"
    assert np.all(lb == 0), "split of a bf16 value has nonzero lo"


# --------------------------------------------------------------------------
# product pins
# --------------------------------------------------------------------------

def pin_golden_gemm(orc):
    fields = {}
    with open(os.path.join(GOLDEN, "gemm_cases.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k, v = line.split(":")
                fields[k.strip()] = v.split()
    M, N, K = (int(v) for v in fields["M N K"])
    A = _f32_from_bits(np.array([int(v, 16) for v in fields["A"]], np.uint32)).reshape(M, K)
    B = _f32_from_bits(np.array([int(v, 16) for v in fields["B"]], np.uint32)).reshape(K, N)
    S_exp = sum(Fraction(2) ** int(t) for t in fields["S_terms"])
    C_exp = np.array([int(v, 16) for v in fields["C"]], np.uint32)
    C, S = orc.gemm3(A, B)
    assert Fraction(float(S[0, 0])) == S_exp, "golden GEMM S = %r, expected %r" % (S[0, 0], float(S_exp))
    assert np.array_equal(_bits_f32(C).ravel(), C_exp), \
        "golden GEMM C = 0x%08x, expected 0x%08x" % (_bits_f32(C).ravel()[0], C_exp[0])


def _short_bf16(shape, rng, emin=-4, emax=3):
    """bf16-representable values sign * (128..255)/128 * 2^e, e in [emin, emax]."""
    sig = rng.integers(128, 256, size=shape).astype(np.float64) / 128.0
    e = rng.integers(emin, emax + 1, size=shape)
    s = np.where(rng.random(shape) < 0.5, -1.0, 1.0)
    return (s * sig * np.exp2(e)).astype(np.float32)


def pin_bf16_inputs(orc, seed=1, shape=(13, 17, 40)):
    """bf16-representable A and B: lo = 0 and the result is the plain product.

    With 8-bit significands and exponents in [-4, 3] every partial sum is exact
    in FP64, so S must equal numpy's FP64 matmul exactly and C its FP32 rounding.
    """
    M, N, K = shape
    rng = np.random.default_rng(seed)
    A = _short_bf16((M, K), rng)
    B = _short_bf16((K, N), rng)
    assert np.all(orc.split(A)[1] == 0) and np.all(orc.split(B)[1] == 0)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    C, S = orc.gemm3(A, B)
    assert np.array_equal(S, ref), "bf16 inputs: S differs from the plain product"
    assert np.array_equal(C, ref.astype(np.float32)), "bf16 inputs: C is not RNE_fp32(S)"


def constructed_operand(shape, rng):
    """x = h + l with h bf16 and l bf16 whose exponent is 10..16 below h's.

    With h in [2^e, 2^(e+1)), |l| < 2^(e-9), which is below half a bf16 step
    on either side of h (2^(e-8) above, 2^(e-9) below a power of two), so
    RNE_bf16(x) = h with no tie; l's lowest bit is at least 2^(e-23), so x is
    exact in FP32 and x - h = l.  The split therefore returns (h, l) exactly.
    Returns (x, h, l) as float32 arrays.
    """
    h = _short_bf16(shape, rng, -3, 3)
    eh = np.floor(np.log2(np.abs(h.astype(np.float64))))
    el = eh - rng.integers(10, 17, size=shape)
    lsig = rng.integers(128, 256, size=shape).astype(np.float64) / 128.0
    ls = np.where(rng.random(shape) < 0.5, -1.0, 1.0)
    l = (ls * lsig * np.exp2(el)).astype(np.float32)
    x64 = h.astype(np.float64) + l.astype(np.float64)
    x = x64.astype(np.float32)
    assert np.array_equal(x.astype(np.float64), x64), "constructed x not exact in FP32"
    return x, h, l


def pin_constructed_split(orc, seed=2, shape=(9, 11, 37)):
    """Closed form: with x = h + l split exactly, exact(A*B) - S = sum lA*lB."""
    M, N, K = shape
    rng = np.random.default_rng(seed)
    A, hA, lA = constructed_operand((M, K), rng)
    B, hB, lB = constructed_operand((K, N), rng)
    ha, la = orc.split(A)
    assert np.array_equal(_bf16_to_f32(ha), hA) and np.array_equal(_bf16_to_f32(la), lA), \
        "constructed A did not split into (h, l)"
    C, S = orc.gemm3(A, B)
    exact = A.astype(np.float64) @ B.astype(np.float64)
    lolo = lA.astype(np.float64) @ lB.astype(np.float64)
    scale = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
    resid = np.abs(exact - S - lolo)
    assert np.all(resid <= 1e-13 * scale), \
        "exact - S != sum lA*lB (max rel %g)" % np.max(resid / scale)


def pin_integer_exact(orc, seed=3):
    """Small integers: every product and partial sum is exact, S = integer GEMM.

    Case 1: |a| <= 2^11 (hi and lo are exact integers), |b| <= 2^7 (bf16-exact).
    Case 2: the roles swapped, so each of the two correction terms is exercised.
    """
    rng = np.random.default_rng(seed)
    for (ba, bb, M, N, K) in ((2048, 128, 19, 23, 32), (128, 2048, 21, 17, 31)):
        A = rng.integers(-ba, ba + 1, size=(M, K)).astype(np.float32)
        B = rng.integers(-bb, bb + 1, size=(K, N)).astype(np.float32)
        ref = A.astype(np.int64) @ B.astype(np.int64)
        assert np.abs(ref).max() < 2 ** 24
        C, S = orc.gemm3(A, B)
        assert np.array_equal(S, ref.astype(np.float64)), "integer GEMM: S != exact"
        assert np.array_equal(C, ref.astype(np.float32)), "integer GEMM: C != exact"


def pin_bruteforce_tiny(orc, seed=4):
    """Tiny sizes against the exact rational product of the FP32 inputs.

    The split drops lo*lo and lo's rounding residual, so per element
    |S - exact| <= 2.1 * 2^-16 * (|A||B|)_ij; a dropped cross term or a wrong
    sign costs about 2^-9 and fails it.
    """
    rng = np.random.default_rng(seed)
    for (M, N, K) in ((1, 1, 1), (2, 3, 5), (4, 4, 8), (3, 7, 6)):
        A = rng.standard_normal((M, K)).astype(np.float32)
        B = rng.standard_normal((K, N)).astype(np.float32)
        C, S = orc.gemm3(A, B)
        for i in range(M):
            for j in range(N):
                ex = sum(Fraction(float(A[i, k])) * Fraction(float(B[k, j])) for k in range(K))
                mag = sum(abs(Fraction(float(A[i, k])) * Fraction(float(B[k, j])))
                          for k in range(K))
                err = abs(Fraction(float(S[i, j])) - ex)
                assert err <= Fraction(21, 10) * Fraction(1, 2 ** 16) * mag, \
                    "tiny brute force (%d,%d,%d) element (%d,%d): err %g > bound" % (
                        M, N, K, i, j, float(err))


def pin_alpha(orc, seed=5):
    """alpha scales the FP64 sum before the FP32 rounding.

    A power of two commutes with rounding, so C(2^-3) = C(1) * 2^-3 exactly;
    the attention scale 1/sqrt(128) gives one rounding of alpha*S.
    """
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((7, 33)).astype(np.float32)
    B = rng.standard_normal((33, 9)).astype(np.float32)
    C1, S1 = orc.gemm3(A, B)
    C8, S8 = orc.gemm3(A, B, alpha=0.125)
    assert np.array_equal(S1, S8)
    assert np.array_equal(C8, C1 * np.float32(0.125)), "alpha = 2^-3 is not an exact scale"
    a = np.float32(1.0 / np.sqrt(128.0))
    Ca, _ = orc.gemm3(A, B, alpha=a)
    ref = float(a) * S1
    assert np.all(np.abs(Ca.astype(np.float64) - ref) <= np.ldexp(np.abs(ref), -24)), \
        "alpha*S not correctly rounded"


def pin_row_subset(orc, seed=6):
    """Computing selected rows gives the same rows as the full product."""
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((40, 70)).astype(np.float32)
    B = rng.standard_normal((70, 30)).astype(np.float32)
    C, S = orc.gemm3(A, B)
    rows = np.array([39, 0, 17, 17, 5])
    Cr, Sr = orc.gemm3(A, B, rows=rows)
    assert np.array_equal(Sr, S[rows]) and np.array_equal(Cr, C[rows]), "row subset differs"


def pin_nonfinite_propagation(orc):
    """Non-finite inputs follow IEEE arithmetic of the split and products.

    An infinite element has lo = inf - inf = NaN, so every output it reaches
    is NaN, as is every output a NaN reaches; a finite element beyond the bf16
    range (hi = inf, lo = -inf) gives inf - inf = NaN too.  Rows and columns
    without such elements are untouched.
    """
    A = np.array([[1.0, np.inf], [1.0, np.nan], [2.0, 3.0], [np.float32(3.4e38), 0.0]],
                 np.float32)
    B = np.array([[1.0, 1.0], [1.0, -1.0]], np.float32)
    C, _ = orc.gemm3(A, B)
    assert np.all(np.isnan(C[0])) and np.all(np.isnan(C[1])) and np.all(np.isnan(C[3]))
    assert np.array_equal(C[2], np.array([5.0, -1.0], np.float32))


# --------------------------------------------------------------------------
# FP16 forms: binary16 rounding, the HEAL-Full pair, weight scaling, GEMM
# --------------------------------------------------------------------------

def _f16_to_f64(h):
    return np.asarray(h, np.uint16).view(np.float16).astype(np.float64)


def _nanh(h):
    return np.isnan(np.asarray(h, np.uint16).view(np.float16))


def _check_pairs_equal(x, hi, lo, hi_ref, lo_ref, what):
    """Bitwise equality of binary16 pairs; NaNs compared by NaN-ness only."""
    for name, a, b in (("hi", hi, hi_ref), ("lo", lo, lo_ref)):
        if not np.array_equal(_nanh(a), _nanh(b)):
            i = np.nonzero(_nanh(a) != _nanh(b))[0][0]
            raise AssertionError("%s: NaN-ness of %s differs at x=%r" % (what, name, x[i]))
    ok = ~(_nanh(hi_ref) | _nanh(lo_ref))
    bad = np.nonzero((hi[ok] != hi_ref[ok]) | (lo[ok] != lo_ref[ok]))[0]
    if bad.size:
        i = np.nonzero(ok)[0][bad[0]]
        raise AssertionError("%s: mismatch at x=%r: got (%04x,%04x), expected (%04x,%04x)"
                             % (what, x[i], hi[i], lo[i], hi_ref[i], lo_ref[i]))


def f16_boundary_doubles():
    """Doubles at, next to and halfway between every pair of adjacent binary16
    values (both signs), plus the overflow tie 65520 and its neighbours."""
    h = np.arange(0, 0x7c00, dtype=np.uint16)              # +0 .. 65504
    v = h.view(np.float16).astype(np.float64)
    nxt = np.append(v[1:], 65536.0)                        # next value up (65536 past the end)
    mid = (v + nxt) / 2.0                                  # exact in FP64
    pts = np.concatenate([v, mid, np.nextafter(mid, 0.0), np.nextafter(mid, np.inf),
                          np.nextafter(v, np.inf), [65520.0, np.nextafter(65520.0, 0.0),
                                                    1e6, np.inf]])
    return np.concatenate([pts, -pts, [np.nan]])


def pin_f16_rne_vs_library(orc):
    """binary16 rounding of doubles equals numpy's float64 -> float16 cast at
    every value, tie and near-tie of the format, and on FP32 inputs of every
    rounding class."""
    x = f16_boundary_doubles()
    got = orc.f16_rne(x)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    both_nan = _nanh(got) & _nanh(ref)
    bad = np.nonzero((got != ref) & ~both_nan)[0]
    assert bad.size == 0, "f16 RNE of %r: got %04x, numpy %04x" % (x[bad[0]], got[bad[0]],
                                                                     ref[bad[0]])
    xf = _f32_from_bits(structured_patterns())
    with np.errstate(over="ignore", invalid="ignore"):
        got = orc.f16_rne(xf.astype(np.float64))
        ref = xf.astype(np.float16).view(np.uint16)
    both_nan = _nanh(got) & _nanh(ref)
    bad = np.nonzero((got != ref) & ~both_nan)[0]
    assert bad.size == 0, "f16 RNE of FP32 %r: got %04x, numpy %04x" % (xf[bad[0]], got[bad[0]],
                                                                         ref[bad[0]])


def load_pair_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                x, h, l = line.split()
                rows.append((int(x, 16), None if h == "nan" else int(h, 16),
                             None if l == "nan" else int(l, 16)))
    return rows


def pin_golden_split_f16(orc):
    """Hand-derived HEAL-Full pairs; "nan" accepts any NaN pattern."""
    rows = load_pair_golden("split_f16_cases.txt")
    x = _f32_from_bits(np.array([r[0] for r in rows], np.uint32))
    hi, lo = orc.split_f16(x)
    for (xb, hb, lb), h, l in zip(rows, hi, lo):
        for exp, got, name in ((hb, int(h), "hi"), (lb, int(l), "lo")):
            if exp is None:
                assert _nanh(np.uint16(got)), "golden f16 pair x=0x%08x: %s=%04x is not NaN" % (
                    xb, name, got)
            else:
                assert got == exp, "golden f16 pair x=0x%08x: %s=%04x, expected %04x" % (
                    xb, name, got, exp)


def reference_split_f16(x):
    """The HEAL-Full pair evaluated with library primitives: numpy's
    float32 -> float16 cast for the head, FP64 for the shifted residual (exact)
    and numpy's float64 -> float16 cast for it."""
    x = np.ascontiguousarray(x, np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        hi = x.astype(np.float16)
        r = (x.astype(np.float64) - hi.astype(np.float64)) * 1024.0
        lo = r.astype(np.float16)
    return hi.view(np.uint16), lo.view(np.uint16)


def pin_split_f16_vs_library(orc):
    x = _f32_from_bits(structured_patterns())
    hi, lo = orc.split_f16(x)
    hr, lr = reference_split_f16(x)
    _check_pairs_equal(x, hi, lo, hr, lr, "f16 pair vs library")


def check_split_f16_range_exhaustive(orc, start, n):
    """Exhaustive form of pin_split_f16_vs_library over FP32 bit patterns
    [start, start+n), the reference evaluated with torch CPU casts (the same
    definition, multi-threaded)."""
    hi, lo = orc.split_f16_range(start, n)
    bits = torch.arange(n, dtype=torch.int64).add_(start).to(torch.int32)
    x = bits.view(torch.float32)
    hr = x.to(torch.float16)
    lr = ((x.to(torch.float64) - hr.to(torch.float64)) * 1024.0).to(torch.float16)
    hi_t = torch.from_numpy(hi.view(np.int16)).view(torch.float16)
    lo_t = torch.from_numpy(lo.view(np.int16)).view(torch.float16)
    what = "exhaustive f16 pair [0x%08x,+%d)" % (start, n)
    hrn, lrn = torch.isnan(hr), torch.isnan(lr)
    assert torch.equal(torch.isnan(hi_t), hrn), "%s: NaN-ness of hi differs" % what
    assert torch.equal(torch.isnan(lo_t), lrn), "%s: NaN-ness of lo differs" % what
    bad = ~(hrn | lrn) & ((hi_t.view(torch.int16) != hr.view(torch.int16)) |
                          (lo_t.view(torch.int16) != lr.view(torch.int16)))
    if torch.any(bad):
        i = int(torch.nonzero(bad)[0, 0])
        raise AssertionError("%s: mismatch at x=0x%08x" % (what, (start + i) & 0xffffffff))


def pin_split_f16_properties(orc, seed=7):
    """Properties of the HEAL-Full pair for finite inputs below the FP16 overflow.

    * x - hi is exact in FP32 (so a device may evaluate it in FP32);
    * |x - hi - 2^-10 lo| <= 2^-22 |x| + 2^-35: hi keeps 11 significant bits,
      |x - hi| is at most half a step of hi (2^-11 relative), and lo rounds
      2^10 (x - hi) to 11 more bits (or to the 2^-24 subnormal step);
    * FP16-representable x gives hi = x and lo = 0.
    """
    rng = np.random.default_rng(seed)
    n = 200000
    e = rng.integers(-40, 16, size=n)
    m = rng.random(n) + 1.0
    x = (np.where(rng.random(n) < 0.5, -1.0, 1.0) * m * np.exp2(e)).astype(np.float32)
    x = x[np.abs(x) < 65504.0]
    hi, lo = orc.split_f16(x)
    hf, lf = _f16_to_f64(hi), _f16_to_f64(lo)
    x64 = x.astype(np.float64)
    assert np.all(np.isfinite(hf)) and np.all(np.isfinite(lf)), "pair overflowed in range"
    r32 = (x - hf.astype(np.float32)).astype(np.float64)
    assert np.array_equal(r32, x64 - hf), "x - hi is not exact in FP32"
    err = np.abs(x64 - hf - lf / 1024.0)
    bound = np.ldexp(np.abs(x64), -22) + 2.0 ** -35
    assert np.all(err <= bound), "pair error exceeds 2^-22|x| + 2^-35 (max ratio %g)" % np.max(
        err / bound)
    hb, lb = orc.split_f16(hf.astype(np.float32))
    assert np.array_equal(hb, hi) and np.all(lb == 0), "pair of an FP16 value is not (x, 0)"


def pin_weight_exponent(orc, seed=8):
    """The weight exponent: golden values and its defining property
    maxabs * 2^e <= 65504 < maxabs * 2^(e+1), checked in exact rationals."""
    golden = [(1.0, 15), (65504.0, 0), (65505.0, -1), (0.0, 0), (0.01, 22), (2.0 ** -20, 35),
              (32752.0, 1), (32753.0, 0), (3.0e38, -112), (2.0 ** -149, 164)]
    for m, e in golden:
        got = orc.f16_weight_exponent(float(np.float32(m)))
        assert got == e, "weight exponent of %r: %d, expected %d" % (m, got, e)
    rng = np.random.default_rng(seed)
    ms = (np.exp2(rng.uniform(-140, 127, size=300)) * rng.uniform(1, 2, size=300)).astype(
        np.float32)
    top = Fraction(65504)
    for m in ms:
        if not np.isfinite(m) or m == 0:
            continue
        e = orc.f16_weight_exponent(float(m))
        fm = Fraction(float(m))
        assert fm * Fraction(2) ** e <= top < fm * Fraction(2) ** (e + 1), \
            "weight exponent %d of %r violates its definition" % (e, m)


def pin_f16_weights_vs_library(orc, seed=9):
    """RNE_f16(W * 2^e) equals numpy's float64 -> float16 cast of the exactly
    scaled weight, including weights that land in the FP16 subnormal range."""
    rng = np.random.default_rng(seed)
    W = (rng.standard_normal((37, 53)) * np.exp2(rng.integers(-30, 2, size=(37, 53)))).astype(
        np.float32)
    W[0, 0] = 0.0
    W[1, 1] = -0.0
    e = orc.f16_weight_exponent(float(np.abs(W).max()))
    got = orc.f16_weights(W, e)
    ref = np.ldexp(W.astype(np.float64), e).astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref), "f16 weights differ from the library cast"
    assert np.all(np.isfinite(_f16_to_f64(got))), "a scaled weight overflowed"


def pin_gemm_f16w_integer(orc, seed=10):
    """Integer activations |a| <= 2^11 are FP16-exact (lo = 0), integer weights
    |w| <= 32 scale exactly (e = 10): S is the exact integer GEMM for both
    forms, and C its FP32 rounding."""
    rng = np.random.default_rng(seed)
    M, N, K = 11, 13, 45
    A = rng.integers(-2048, 2049, size=(M, K)).astype(np.float32)
    W = rng.integers(-32, 33, size=(N, K)).astype(np.float32)
    W[0, 0] = 32.0
    e = orc.f16_weight_exponent(float(np.abs(W).max()))
    assert e == 10
    ref = A.astype(np.int64) @ W.astype(np.int64).T
    for products in (1, 2):
        C, S = orc.gemm_f16w(A, W, e, products)
        assert np.array_equal(S, ref.astype(np.float64)), "integer f16 GEMM: S != exact"
        assert np.array_equal(C, ref.astype(np.float32)), "integer f16 GEMM: C != exact"


def pin_gemm_f16w_bruteforce(orc, seed=11):
    """Tiny sizes against the exact rational product A * W16^T, W16 = the FP16
    weight values (numpy's cast of W * 2^e), scaled back by 2^-e:
      Full: |S - exact| <= 2^-e sum_k |w16| (2^-22 |a| + 2^-35) * (1 + 2^-40)
      Base: |S - exact| <= 2^-e sum_k |w16| (2^-11 |a| + 2^-25) * (1 + 2^-40)
    and Full must beat the Base bound by far, so a dropped or mis-scaled
    residual product, or a wrong exponent sign, fails."""
    rng = np.random.default_rng(seed)
    for (M, N, K) in ((1, 1, 1), (2, 3, 5), (3, 4, 9), (4, 2, 16)):
        A = (rng.standard_normal((M, K)) * 3.0).astype(np.float32)
        W = (rng.standard_normal((N, K)) * 0.05).astype(np.float32)
        e = orc.f16_weight_exponent(float(np.abs(W).max()))
        w16 = np.ldexp(W.astype(np.float64), e).astype(np.float16).astype(np.float64)
        Cf, Sf = orc.gemm_f16w(A, W, e, 2)
        Cb, Sb = orc.gemm_f16w(A, W, e, 1)
        scale = Fraction(2) ** (-e)
        for i in range(M):
            for j in range(N):
                ex = scale * sum(Fraction(float(A[i, k])) * Fraction(float(w16[j, k]))
                                 for k in range(K))
                bf = scale * sum(abs(Fraction(float(w16[j, k]))) *
                                 (abs(Fraction(float(A[i, k]))) / 2 ** 22 + Fraction(1, 2 ** 35))
                                 for k in range(K)) * (1 + Fraction(1, 2 ** 40))
                bb = scale * sum(abs(Fraction(float(w16[j, k]))) *
                                 (abs(Fraction(float(A[i, k]))) / 2 ** 11 + Fraction(1, 2 ** 25))
                                 for k in range(K)) * (1 + Fraction(1, 2 ** 40))
                ef = abs(Fraction(float(Sf[i, j])) - ex)
                eb = abs(Fraction(float(Sb[i, j])) - ex)
                assert ef <= bf, "Full (%d,%d,%d) (%d,%d): err %g > bound %g" % (
                    M, N, K, i, j, float(ef), float(bf))
                assert eb <= bb, "Base (%d,%d,%d) (%d,%d): err %g > bound %g" % (
                    M, N, K, i, j, float(eb), float(bb))
                assert np.float32(float(Sf[i, j])) == Cf[i, j], "Full C is not RNE_fp32(S)"


def pin_gemm_f16w_rows(orc, seed=12):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((30, 50)).astype(np.float32)
    W = rng.standard_normal((20, 50)).astype(np.float32)
    C, S = orc.gemm_f16w(A, W, 3, 2)
    rows = np.array([29, 0, 7, 7])
    Cr, Sr = orc.gemm_f16w(A, W, 3, 2, rows=rows)
    assert np.array_equal(Sr, S[rows]) and np.array_equal(Cr, C[rows]), "row subset differs"


# --------------------------------------------------------------------------
# INT16 codes and dual-FP16 scores (HEAL+)
# --------------------------------------------------------------------------

def exact_i16_code(x, m):
    """Round(32767 x / m) of the real quotient, ties to even (exact rationals)."""
    if float(m) == 0.0:
        return 0
    return round(Fraction(32767) * Fraction(float(x)) / Fraction(float(m)))


def load_quantize_golden():
    rows = []
    with open(os.path.join(GOLDEN, "quantize_i16_cases.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                xb, mb, q = line.split()
                rows.append((int(xb, 16), int(mb, 16), int(q)))
    return rows


def pin_quantize_i16_golden(orc):
    """Elements of the attention workload whose exactly rounded code differs
    from an FP32 decision (tests/golden/quantize_i16_cases.txt, derived in
    exact rationals): each is quantized together with an element equal to its
    tensor's maximum, so max|X| is the recorded m."""
    rows = load_quantize_golden()
    assert len(rows) >= 40
    for xb, mb, code in rows:
        x, m = _f32_from_bits(np.uint32(xb)), _f32_from_bits(np.uint32(mb))
        assert exact_i16_code(x, m) == code, "golden file entry 0x%08x is not Round" % xb
        q, mq = orc.quantize_i16(np.array([x, m, -x], np.float32))
        assert mq == m, "max|X| of the golden case"
        assert (int(q[0]), int(q[1]), int(q[2])) == (code, 32767, -code), \
            "golden x=0x%08x m=0x%08x: code %d, expected %d" % (xb, mb, int(q[0]), code)


def near_half_integer_inputs(rng, m, count):
    """FP32 x whose quotient 32767 x / m lies within a few ulps of a
    half-integer n + 1/2: the nearest float to (n + 1/2) m / 32767 and its two
    neighbours, for random n of both signs."""
    n = rng.integers(-32767, 32767, size=count)
    c = ((n + 0.5) * float(m) / 32767.0).astype(np.float32)
    xs = np.concatenate([c, np.nextafter(c, np.float32(np.inf)), np.nextafter(c, np.float32(-np.inf))])
    return xs[np.abs(xs) <= m]


def pin_quantize_i16(orc, seed=13):
    """INT16 codes by the definition Round(32767 x / max|X|) (Section 4, Q/K/V
    paragraph): golden ties, the range, the extremes, all-zero input, codes
    equal to the exact rational rounding on random values and on values whose
    quotient sits next to a half-integer, tiny and subnormal maxima, and the
    paper's INT16 error bound |x - q D| <= D/2 (D = max|X| / 32767) with no
    slack."""
    x = np.array([2.0, -1.0, 0.5, 1e-30, 0.0, -2.0, 1.5], np.float32)
    q, m = orc.quantize_i16(x)
    # 32767 x / 2: -1 -> -16383.5, a tie, to even -16384; 0.5 -> 8191.75 -> 8192;
    # 1.5 -> 24575.25 -> 24575
    assert m == 2.0 and list(q) == [32767, -16384, 8192, 0, 0, -32767, 24575], (list(q), m)
    # max|X| = 32767: the quotient is x itself, halves are ties to even
    q, m = orc.quantize_i16(np.array([32767.0, 2.5, -3.5, 0.5, 1.5, -0.5, 7.25], np.float32))
    assert m == 32767.0 and list(q) == [32767, 2, -4, 0, 2, 0, 7], (list(q), m)
    # max|X| = 3 (not a divisor of 32767): 32767 * 1 / 3 = 10922.33 -> 10922,
    # 32767 * 2.25 / 3 = 24575.25 -> 24575, 32767 * (-1.5) / 3 = -16383.5 -> -16384
    q, m = orc.quantize_i16(np.array([3.0, 1.0, 2.25, -1.5], np.float32))
    assert m == 3.0 and list(q) == [32767, 10922, 24575, -16384], (list(q), m)
    q0, m0 = orc.quantize_i16(np.zeros(9, np.float32))
    assert m0 == 0.0 and np.all(q0 == 0), "all-zero tensor"
    rng = np.random.default_rng(seed)
    cases = []
    for scale in (1e-3, 1.0, 300.0, 1e-36):
        x = (rng.standard_normal(50000) * scale).astype(np.float32)
        x[17] = np.float32(-40.0 * scale)  # an outlier sets max|X|
        cases.append((x, np.float32(40.0 * scale), 17))
        m = np.float32(40.0 * scale)
        near = near_half_integer_inputs(rng, m, 3000)
        cases.append((np.concatenate([np.array([m], np.float32), near]), m, 0))
    # subnormal maxima: the smallest subnormal and a few steps of it
    tiny = np.array([2.0 ** -149, -2.0 ** -149, 0.0], np.float32)
    cases.append((tiny, np.float32(2.0 ** -149), 0))
    sub = (rng.integers(-1000, 1001, size=2000) * 2.0 ** -149).astype(np.float32)
    sub[0] = np.float32(1000 * 2.0 ** -149)
    cases.append((sub, np.float32(1000 * 2.0 ** -149), 0))
    for x, mexp, imax in cases:
        q, m = orc.quantize_i16(x)
        assert m == mexp, "max|X| %r, expected %r" % (m, mexp)
        assert q.min() >= -32767 and q.max() <= 32767
        assert abs(int(q[imax])) == 32767, "the maximum's code"
        D = Fraction(float(m)) / 32767
        sample = np.arange(x.size) if x.size <= 4000 else rng.choice(x.size, 4000, replace=False)
        for i in sample:
            want = exact_i16_code(x[i], m)
            assert int(q[i]) == want, "x=%r m=%r: code %d, exact Round %d" % (
                float(x[i]), float(m), int(q[i]), want)
            assert abs(Fraction(float(x[i])) - int(q[i]) * D) <= D / 2, "INT16 error exceeds D/2"


def pin_int16_mse_ratio(orc, seed=14):
    """The paper's ratio bound E[MSE_fp16] / E[MSE_int16] > 256 sigma^2 / M^2
    (Section 4, Q/K/V paragraph), measured on Gaussian tensors with one
    outlier, against numpy's FP16 cast."""
    rng = np.random.default_rng(seed)
    for outlier in (4.0, 12.0, 40.0):
        x = rng.standard_normal(200000).astype(np.float32)
        x[0] = np.float32(outlier)
        q, m = orc.quantize_i16(x)
        deq = q.astype(np.float64) * (float(m) / 32767.0)
        mse_i16 = np.mean((deq - x) ** 2)
        mse_f16 = np.mean((x.astype(np.float16).astype(np.float64) - x) ** 2)
        sigma2, M = np.var(x.astype(np.float64)), float(m)
        assert mse_f16 / mse_i16 > 256.0 * sigma2 / M ** 2, (outlier, mse_f16 / mse_i16)


def pin_unpack_i16_exhaustive(orc):
    """Every INT16 code q unpacks to FP16 (hi, lo) with hi = numpy's float16 of
    q, hi + lo / 2^10 == q exactly, and |lo| / 2^10 <= 8."""
    q = np.arange(-32768, 32768, dtype=np.int64).astype(np.int16)
    hi, lo = orc.unpack_i16(q)
    assert np.array_equal(hi, q.astype(np.float16).view(np.uint16)), "hi is not f16(q)"
    hv, lv = _f16_to_f64(hi), _f16_to_f64(lo)
    assert np.array_equal(hv + lv / 1024.0, q.astype(np.float64)), "hi + lo/2^10 != q"
    assert np.abs(lv).max() <= 8 * 1024, "lo out of range"


def pin_scores_i16(orc, seed=15):
    """The four dual-FP16 products sum to the exact integer dot product of the
    codes (closed form); the factor is the dequantisation of both codes times
    alpha, alpha (maxQ / 32767)(maxK / 32767), within 2^-51 of its exact value;
    C is the FP32 rounding of factor * S (exact rationals)."""
    rng = np.random.default_rng(seed)
    M, N, K = 9, 7, 64
    Q = rng.integers(-32767, 32768, size=(M, K)).astype(np.int16)
    Kt = rng.integers(-32767, 32768, size=(N, K)).astype(np.int16)
    Q[0, :] = 32767
    Kt[0, :] = -32767
    for mq, mk, alpha in ((2.5, 0.75, 1.0 / np.sqrt(128.0)), (5.0978498, 5.571465, 0.125),
                          (1e-20, 3e-19, 0.7)):
        mq, mk, alpha = np.float32(mq), np.float32(mk), np.float32(alpha)
        C, S = orc.scores_i16(Q, Kt, mq, mk, alpha)
        exact = Q.astype(np.int64) @ Kt.astype(np.int64).T
        assert np.array_equal(S, exact.astype(np.float64)), "scores: S != integer dot product"
        f = orc.scores_factor(mq, mk, alpha)
        fx = Fraction(float(alpha)) * Fraction(float(mq)) * Fraction(float(mk)) / 32767 ** 2
        assert abs(Fraction(f) - fx) <= fx * Fraction(1, 2 ** 51), "scores factor"
        for i in range(M):
            for j in range(N):
                v = fx * int(exact[i, j])
                err = abs(Fraction(float(C[i, j])) - v)
                # half an FP32 step: 2^-24 |v| for normal results, 2^-150 below 2^-126
                half_step = max(abs(v) * Fraction(1, 2 ** 24), Fraction(1, 2 ** 150))
                assert err <= half_step * (1 + Fraction(1, 2 ** 20)), \
                    "scores: C != f32(factor * S) at (%d, %d)" % (i, j)
    rows = np.array([8, 0, 3])
    Cr, Sr = orc.scores_i16(Q, Kt, mq, mk, alpha, rows=rows)
    assert np.array_equal(Cr, C[rows]) and np.array_equal(Sr, S[rows]), "row subset differs"


SMALL_PINS = [pin_golden_split, pin_split_vs_library, pin_split_properties, pin_golden_gemm,
              pin_bf16_inputs, pin_constructed_split, pin_integer_exact, pin_bruteforce_tiny,
              pin_alpha, pin_row_subset, pin_nonfinite_propagation,
              pin_f16_rne_vs_library, pin_golden_split_f16, pin_split_f16_vs_library,
              pin_split_f16_properties, pin_weight_exponent, pin_f16_weights_vs_library,
              pin_gemm_f16w_integer, pin_gemm_f16w_bruteforce, pin_gemm_f16w_rows,
              pin_quantize_i16, pin_quantize_i16_golden, pin_int16_mse_ratio,
              pin_unpack_i16_exhaustive, pin_scores_i16]

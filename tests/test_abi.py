"""The C-ABI library: loads, exports what include/heal.h declares, and rejects
bad arguments before touching the device (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2606_21023_amd as heal

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "heal.h")

INVALID = 1


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(heal_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("heal_split_f32", "heal_gemm_f32", "heal_gemm_f32_strided_batched",
                     "heal_status_string"):
        assert required in names


def test_library_exports_every_declared_symbol():
    L = heal.lib()
    for name in declared_functions():
        assert hasattr(L, name), "libheal.so does not export %s" % name


def test_status_strings_and_version():
    L = heal.lib()
    for code, name in heal.STATUS.items():
        assert L.heal_status_string(code).decode() == name
    assert L.heal_status_string(99).decode() == "HEAL_ERR_UNKNOWN"
    assert L.heal_version() >= 100


def test_build_id_matches_the_sources():
    """The library reports the hash of the sources it was built from, and it
    is the hash of the sources in this tree; an edit of any source changes it."""
    from paper_2606_21023_amd import build as hbuild
    got = heal.build_id()
    assert re.fullmatch(r"[0-9a-f]{16}", got), got
    assert got == hbuild.source_hash()
    assert heal.check_build() == got


def test_select_instance_depends_on_m_and_n_only():
    assert heal.select_instance(1, 4096) == heal.INSTANCE_SKINNY
    assert heal.select_instance(64, 128256) == heal.INSTANCE_SKINNY
    assert heal.select_instance(65, 4096) in (heal.INSTANCE_MEDIUM, heal.INSTANCE_LARGE)
    assert heal.select_instance(8192, 8192) == heal.INSTANCE_LARGE


FAKE = 0x10000  # never dereferenced: every call below fails validation first


@pytest.mark.parametrize("args", [
    # M, N, K, A, B, C, lda, ldb, ldc
    (-1, 4, 4, FAKE, FAKE, FAKE, 4, 4, 4),       # negative M
    (4, -1, 4, FAKE, FAKE, FAKE, 4, 4, 4),       # negative N
    (4, 4, -1, FAKE, FAKE, FAKE, 4, 4, 4),       # negative K
    (4, 4, 8, FAKE, FAKE, FAKE, 7, 4, 4),        # lda < K
    (4, 8, 4, FAKE, FAKE, FAKE, 4, 7, 8),        # ldb < N
    (4, 8, 4, FAKE, FAKE, FAKE, 4, 8, 7),        # ldc < N
    (4, 4, 4, 0, FAKE, FAKE, 4, 4, 4),           # null A
    (4, 4, 4, FAKE, 0, FAKE, 4, 4, 4),           # null B
    (4, 4, 4, FAKE, FAKE, 0, 4, 4, 4),           # null C
    (4, 4, 4, FAKE + 2, FAKE, FAKE, 4, 4, 4),    # A not 4-byte aligned
    (4, 4, 4, FAKE, FAKE, FAKE + 1, 4, 4, 4),    # C not 4-byte aligned
])
def test_gemm_rejects_invalid_arguments(args):
    st = heal.lib().heal_gemm_f32(*args, None)
    assert st == INVALID


def test_empty_products_are_noops_without_device():
    L = heal.lib()
    assert L.heal_gemm_f32(0, 4, 4, 0, 0, 0, 4, 4, 4, None) == 0
    assert L.heal_gemm_f32(4, 0, 4, 0, 0, 0, 4, 1, 1, None) == 0
    assert L.heal_split_f32(0, 0, 0, 0, None) == 0
    f = L.heal_gemm_f32_strided_batched
    assert f(4, 4, 4, ctypes.c_float(1.0), 0, 4, 0, 0, 4, 0, 0, 0, 4, 0, 0, None) == 0  # batch 0


@pytest.mark.parametrize("bad", ["trans", "stride", "batch", "ldb_t"])
def test_batched_rejects_invalid_arguments(bad):
    f = heal.lib().heal_gemm_f32_strided_batched
    a = dict(M=4, N=8, K=16, alpha=ctypes.c_float(1.0), A=FAKE, lda=16, sA=64, B=FAKE, ldb=8,
             sB=128, tb=0, C=FAKE, ldc=8, sC=32, batch=2)
    if bad == "trans":
        a["tb"] = 2
    elif bad == "stride":
        a["sA"] = -1
    elif bad == "batch":
        a["batch"] = -3
    elif bad == "ldb_t":
        a["tb"] = 1
        a["ldb"] = 15   # B stored N x K needs ldb >= K
    st = f(a["M"], a["N"], a["K"], a["alpha"], a["A"], a["lda"], a["sA"], a["B"], a["ldb"],
           a["sB"], a["tb"], a["C"], a["ldc"], a["sC"], a["batch"], None)
    assert st == INVALID


def test_split_rejects_invalid_arguments():
    L = heal.lib()
    assert L.heal_split_f32(FAKE, FAKE, FAKE, -1, None) == INVALID
    assert L.heal_split_f32(0, FAKE, FAKE, 8, None) == INVALID
    assert L.heal_split_f32(FAKE, FAKE + 1, FAKE, 8, None) == INVALID


def test_forced_instance_out_of_range_rejected():
    f = heal.lib().heal_gemm_f32_instance
    st = f(17, 4, 4, 4, ctypes.c_float(1.0), FAKE, 4, 0, FAKE, 4, 0, 0, FAKE, 4, 0, 1, None)
    assert st == INVALID


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(heal, "_lib", None)
    monkeypatch.setattr(heal, "library_path", "/nonexistent/libheal.so")
    with pytest.raises(heal.HealError):
        heal.lib()


# ---- FP16 forms, pre-split operand, INT16 scores: validation without a GPU ----

def _f16w(products=2, M=4, N=8, K=16, A=FAKE, lda=16, W=FAKE, e=0, C=FAKE, ldc=8, inst=0):
    return heal.lib().heal_gemm_f16w_instance(inst, products, M, N, K, A, lda, W, e, C, ldc, None)


@pytest.mark.parametrize("kw", [
    dict(products=3), dict(products=0), dict(e=301), dict(e=-301), dict(M=-1), dict(K=-1),
    dict(K=(1 << 20) + 4, lda=(1 << 20) + 4), dict(lda=15), dict(ldc=7), dict(A=0), dict(W=0),
    dict(C=0), dict(A=FAKE + 2), dict(W=FAKE + 8), dict(C=FAKE + 1), dict(inst=17),
])
def test_gemm_f16w_rejects_invalid_arguments(kw):
    assert _f16w(**kw) == INVALID


def test_new_empty_calls_are_noops_without_device():
    L = heal.lib()
    assert _f16w(M=0, A=0, W=0, C=0) == 0
    assert _f16w(N=0, A=0, W=0, C=0, ldc=1) == 0
    assert L.heal_gemm_f32_presplit(0, 8, 16, 0, 16, 0, 0, 8, None) == 0
    assert L.heal_pack_f16_weight(0, 0, 16, 16, 0, 0, None) == 0
    assert L.heal_presplit_b(0, 16, 0, 1, 0, 0, None) == 0
    assert L.heal_split_f16(0, 0, 0, 0, None) == 0
    assert L.heal_scores_i16(0, 8, 16, 0, 16, 0, 0, 0, 16, 0, 0, ctypes.c_float(1.0), 0, 8, 0, 1,
                             None) == 0


def test_pack_and_presplit_reject_invalid_arguments():
    L = heal.lib()
    assert L.heal_pack_f16_weight(FAKE, 8, 16, 15, 0, FAKE, None) == INVALID      # ldw < K
    assert L.heal_pack_f16_weight(FAKE, 8, 16, 16, 301, FAKE, None) == INVALID    # |e| > 300
    assert L.heal_pack_f16_weight(FAKE, 8, 16, 16, 0, FAKE + 8, None) == INVALID  # W16 alignment
    assert L.heal_pack_f16_weight(FAKE, -8, 16, 16, 0, FAKE, None) == INVALID
    assert L.heal_presplit_b(FAKE, 16, 8, 8, 2, FAKE, None) == INVALID           # trans flag
    assert L.heal_presplit_b(FAKE, 16, 8, 7, 0, FAKE, None) == INVALID           # ldb < N
    assert L.heal_presplit_b(FAKE, 16, 8, 15, 1, FAKE, None) == INVALID          # ldb < K (N x K)
    assert L.heal_presplit_b(FAKE, 16, 8, 8, 0, FAKE + 4, None) == INVALID       # Bp alignment
    f = L.heal_gemm_f32_presplit
    assert f(4, 8, 16, FAKE, 15, FAKE, FAKE, 8, None) == INVALID                  # lda < K
    assert f(4, 8, 16, FAKE, 16, FAKE + 2, FAKE, 8, None) == INVALID              # Bp alignment
    assert L.heal_gemm_f32_presplit_instance(9, 4, 8, 16, FAKE, 16, FAKE, FAKE, 8, None) == INVALID


def test_scores_quantize_maxabs_split_f16_reject_invalid_arguments():
    L = heal.lib()
    one = ctypes.c_float(1.0)
    s = L.heal_scores_i16
    assert s(4, 8, 16, FAKE, 15, 0, FAKE, FAKE, 16, 0, FAKE, one, FAKE, 8, 0, 1, None) == INVALID
    assert s(4, 8, 16, FAKE, 16, 0, FAKE, FAKE, 16, 0, FAKE, one, FAKE, 7, 0, 1, None) == INVALID
    assert s(4, 8, 16, FAKE, 16, 0, 0, FAKE, 16, 0, FAKE, one, FAKE, 8, 0, 1, None) == INVALID
    assert s(4, 8, 16, FAKE + 1, 16, 0, FAKE, FAKE, 16, 0, FAKE, one, FAKE, 8, 0, 1,
             None) == INVALID
    assert s(4, 8, 16, FAKE, 16, -1, FAKE, FAKE, 16, 0, FAKE, one, FAKE, 8, 0, 2, None) == INVALID
    assert s(4, 8, 16, FAKE, 16, 0, FAKE, FAKE, 16, 0, FAKE, one, FAKE + 2, 8, 0, 1,
             None) == INVALID
    assert L.heal_quantize_i16(FAKE, -1, FAKE, FAKE, None) == INVALID
    assert L.heal_quantize_i16(FAKE, 8, FAKE, 0, None) == INVALID
    assert L.heal_quantize_i16(FAKE, 8, FAKE + 1, FAKE, None) == INVALID
    assert L.heal_maxabs_f32(FAKE, 4, 8, 7, FAKE, None) == INVALID
    assert L.heal_maxabs_f32(FAKE, 4, 8, 8, 0, None) == INVALID
    assert L.heal_maxabs_f32(0, 4, 8, 8, FAKE, None) == INVALID
    assert L.heal_split_f16(FAKE, FAKE, FAKE, -1, None) == INVALID
    assert L.heal_split_f16(FAKE, FAKE + 1, FAKE, 8, None) == INVALID


def test_oversized_products_rejected():
    """Outputs whose element count would overflow 64-bit tile arithmetic."""
    L = heal.lib()
    big = 1 << 40
    assert L.heal_gemm_f32(big, big, 4, FAKE, FAKE, FAKE, 4, big, big, None) == INVALID
    assert _f16w(M=big, N=1 << 39, ldc=1 << 39) == INVALID
    assert L.heal_maxabs_f32(FAKE, 1 << 40, 8, 1 << 40, FAKE, None) == INVALID


def test_header_is_plain_c_and_links(tmp_path):
    """include/heal.h compiles as C11 with a plain C compiler, and a C program
    linked against libheal.so sees the host-side contract (no GPU needed)."""
    import shutil
    import subprocess
    from paper_2606_21023_amd import build as hbuild
    gcc = shutil.which("gcc")
    if gcc is None or not os.path.exists(hbuild.LIBRARY):
        pytest.skip("gcc or libheal.so not available")
    src = os.path.join(ROOT, "tests", "c", "abi_check.c")
    exe = str(tmp_path / "abi_check")
    libdir = os.path.dirname(hbuild.LIBRARY)
    subprocess.run([gcc, "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", src,
                    "-L", libdir, "-lheal", "-Wl,-rpath," + libdir, "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    assert "abi_check: ok" in r.stdout

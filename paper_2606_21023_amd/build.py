"""Build libheal.so (the HIP kernels and their C ABI) for gfx950 with hipcc.

``build()`` always recompiles.  Objects go to ``_build/`` at the repository
root and the library to ``paper_2606_21023_amd/libheal.so``.
"""
import concurrent.futures as cf
import hashlib
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIBRARY = os.path.join(PKG, "libheal.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["heal_api.cpp", "heal_split.hip", "heal_gemm.hip", "heal_gemm_large.hip",
           "heal_gemm_skinny.hip", "heal_gemm_panel.hip", "heal_ops.hip", "heal_gemm_op.hip"]

# Packed FP32 instructions are disabled: only plain FP32 VALU code is emitted.
# The host pass of hipcc does not know this feature and says so; harmless.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC]


def source_hash():
    """Hash of everything the library is built from: every file under csrc/,
    the public header and the compiler flags (16 hex digits).  The built
    library returns the value it was built with from heal_build_id()."""
    h = hashlib.sha256()
    files = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp", ".h")))
    for name in files:
        h.update(name.encode() + b"\0")
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read() + b"\0")
    with open(os.path.join(INCLUDE, "heal.h"), "rb") as f:
        h.update(f.read() + b"\0")
    flags = [f for f in FLAGS if f not in ("-I", INCLUDE, CSRC)]  # paths differ by machine
    h.update(" ".join(flags + SOURCES).encode())
    return h.hexdigest()[:16]


def _compile(src, build_id):
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    ident = ['-DHEAL_BUILD_ID="%s"' % build_id] if src == "heal_api.cpp" else []
    cmd = [HIPCC, *FLAGS, *ident, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def build(verbose=False):
    """Compile every source and link ``libheal.so``; returns its path."""
    os.makedirs(OBJDIR, exist_ok=True)
    build_id = source_hash()
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_id), SOURCES))
    tmp = LIBRARY + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, LIBRARY)
    if verbose:
        print(LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

"""Build the oracle's shared library with the host C compiler.

Test infrastructure only.  ``build()`` compiles ``heal_oracle.c`` with
``gcc -O2 -fopenmp -ffp-contract=off`` (no fast-math, no FMA contraction) into
``liboracle.so`` beside it.  ``build_from_source`` compiles an arbitrary source
text, which the mutation tests use to check that the pins catch planted
mistakes.
"""
import os
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "heal_oracle.c")
LIBRARY = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-std=c11", "-Wall"]


def build_from_source(text, out_path, werror=True):
    """Compile C source ``text`` into the shared library ``out_path``."""
    with tempfile.NamedTemporaryFile("w", suffix=".c", delete=False) as f:
        f.write(text)
        src = f.name
    try:
        tmp_out = out_path + ".tmp%d" % os.getpid()
        flags = CFLAGS + (["-Werror"] if werror else ["-w"])
        subprocess.run(["gcc", *flags, src, "-o", tmp_out, "-lm"], check=True)
        os.replace(tmp_out, out_path)
    finally:
        os.unlink(src)
    return out_path


def build():
    """Compile the oracle library; always recompiles."""
    with open(SOURCE) as f:
        return build_from_source(f.read(), LIBRARY)


if __name__ == "__main__":
    print(build())

"""Write quantize_i16_cases.txt: INT16 codes q = Round(32767 x / max|X|).

Each expected code is derived in exact rational arithmetic (Python's
fractions): the real quotient 32767 x / m rounded to the nearest integer, ties
to even.  The cases are elements of the attention-score workload's Q and K
tensors (32 heads x 2048 x 128, N(0,1), the seeded generator of
paper_2606_21023_amd.workloads) whose exactly rounded code differs from a
decision taken in FP32 as rint(x * fl32(32767 / m)); the FP32 value is only
used to pick the cases.  Run from the repository root:
    python tests/golden/make_quantize_i16_cases.py
"""
import os
import sys
from fractions import Fraction

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
from paper_2606_21023_amd import workloads as wl  # noqa: E402

PER_TENSOR = 24


def exact_code(x, m):
    return round(Fraction(32767) * Fraction(float(x)) / Fraction(float(m)))


def main():
    Q, K = wl.make_inputs(wl.WORKLOADS["attn_scores"])
    lines = []
    for name, t in (("Q", Q), ("K", K)):
        x = t.ravel()
        m = np.float32(np.abs(x).max())
        inv32 = np.float32(32767.0) / m
        fp32 = np.rint(x * inv32)
        near = np.rint(32767.0 * x.astype(np.float64) / np.float64(m))
        idx = np.nonzero(fp32 != near)[0]
        print("%s: max|x| = %r, %d of %d codes differ from the FP32 decision"
              % (name, float(m), idx.size, x.size))
        for i in idx[:PER_TENSOR]:
            q = exact_code(x[i], m)
            lines.append("%08x %08x %d  # attention %s element %d; FP32 decision gives %d"
                         % (x[i].view(np.uint32), m.view(np.uint32), q, name, i, int(fp32[i])))
    with open(os.path.join(HERE, "quantize_i16_cases.txt"), "w") as f:
        f.write("# INT16 codes q = Round(32767 x / m), m = max|X| of the tensor the element\n"
                "# belongs to; Round is to the nearest integer, ties to even, of the real\n"
                "# quotient (HEAL Section 4, Q/K/V paragraph).  Expected codes derived in\n"
                "# exact rational arithmetic by make_quantize_i16_cases.py.\n"
                "# Each line: x_hex m_hex code  # origin\n")
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()

"""Helpers shared by the GPU parity tests: device checks, tolerance bars.

Bars (from the contract of the compensated GEMM): against the oracle's FP64
sum S, normwise ||C - S||_F / ||S||_F <= 2e-6 and elementwise
|C - S| <= 1e-5 * (|A||B|)_ij, with |A||B| formed in FP64 from the original
FP32 inputs; where (|A||B|)_ij = 0, C_ij must be zero.
"""
import sys

import numpy as np
import pytest
import torch

NORMWISE_BAR = 2e-6
ELEMENTWISE_BAR = 1e-5

needs_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="no GPU in this container")


def announce(msg):
    """Name the case before a GPU step, flushed, so a crash log shows it."""
    sys.stdout.write("[gpu-case] %s\n" % msg)
    sys.stdout.flush()


def to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def abs_product(A, B):
    return np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))


def check_tolerance(C, S, absAB, what="", normwise_min_elements=0):
    """Assert the bars; returns (normwise, max elementwise ratio).

    The normwise bar is a statement about a whole output: on a handful of
    elements, one sum that cancels to a small value (FP32 accumulation error
    relative to its terms, not to the result) can exceed it while every
    element meets the elementwise bar.  Callers that draw arbitrary shapes
    pass normwise_min_elements to apply it only to outputs at least that
    large; the elementwise bar always applies."""
    C = np.asarray(C, np.float64)
    S = np.asarray(S, np.float64)
    err = np.abs(C - S)
    nS = np.linalg.norm(S)
    normwise = np.linalg.norm(C - S) / nS if nS > 0 else np.linalg.norm(C - S)
    zero = absAB == 0
    assert np.all(C[zero] == 0), "%s: nonzero output where |A||B| = 0" % what
    ratio = np.where(zero, 0.0, err / np.where(zero, 1.0, absAB))
    worst = float(ratio.max()) if ratio.size else 0.0
    if C.size >= normwise_min_elements:
        assert normwise <= NORMWISE_BAR, "%s: normwise %.3g > %g" % (what, normwise, NORMWISE_BAR)
    assert worst <= ELEMENTWISE_BAR, "%s: elementwise %.3g > %g" % (what, worst, ELEMENTWISE_BAR)
    return normwise, worst

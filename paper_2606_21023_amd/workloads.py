"""Seeded synthetic inputs for the compensated GEMM.

This module only draws random numbers; it holds none of the method's
arithmetic.  The HIP path's tests, the benchmark and the CPU oracle's tests all
take their inputs from here, so both sides see identical bits.

Recipe (one ``numpy.random.default_rng(seed)`` stream per workload, PCG64):
  * A is drawn first, then B, each ``standard_normal(..., dtype=float32)``
    scaled by its sigma in float32;
  * "outlier channels" are 0.1% of A's K columns (``round(0.001*K)``, at least
    one), chosen with ``rng.choice(K, n, replace=False)`` after A and B are
    drawn, and scaled by 50 -- the fixed-channel outliers the paper describes
    for LLM activations (Section 4, GEMM compensation paragraph);
  * the attention-score workload draws Q then K per head, 2048 x 128 each,
    and multiplies Q by K^T with the 1/sqrt(128) scale applied after
    accumulation.

The shapes are those of a Llama-3.1-8B layer (hidden 4096, MLP 14336,
32 heads x 128, vocabulary 128256), one of the models the paper evaluates,
standing in for its ShareGPT serving workload.
"""
from dataclasses import dataclass, field

import numpy as np

ATTN_SCALE = np.float32(1.0 / np.sqrt(128.0))


@dataclass
class Workload:
    name: str
    M: int
    N: int
    K: int
    seed: int
    sigma_a: float = 1.0
    sigma_b: float = 1.0
    outlier_frac: float = 0.0
    outlier_scale: float = 50.0
    batch: int = 1
    trans_b: bool = False
    alpha: float = 1.0
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def flops(self):
        """FP32-equivalent flops, 2*M*N*K per batch entry."""
        return 2.0 * self.M * self.N * self.K * self.batch

    @property
    def algorithmic_bytes(self):
        """FP32 A and B read once plus FP32 C written once."""
        return 4.0 * self.batch * (self.M * self.K + self.K * self.N + self.M * self.N)


WORKLOADS = {
    "square256": Workload("square256", 256, 256, 256, seed=0,
                          note="M=N=K=256, A,B ~ N(0,1)"),
    "decode": Workload("decode", 16, 4096, 4096, seed=1, sigma_b=0.02, outlier_frac=0.001,
                       note="decode projection 16x4096 @ 4096x4096"),
    "prefill_up": Workload("prefill_up", 2048, 14336, 4096, seed=2, sigma_b=0.02,
                           outlier_frac=0.001,
                           note="prefill MLP up-projection 2048x4096 @ 4096x14336"),
    "attn_scores": Workload("attn_scores", 2048, 2048, 128, seed=3, batch=32, trans_b=True,
                            alpha=float(ATTN_SCALE),
                            note="32 heads of Q(2048x128) @ K^T(128x2048) / sqrt(128)"),
    "square8192": Workload("square8192", 8192, 8192, 8192, seed=4,
                           note="M=N=K=8192, A,B ~ N(0,1)"),
    "lm_head": Workload("lm_head", 64, 128256, 4096, seed=5, sigma_b=0.02,
                        note="lm_head 64x4096 @ 4096x128256"),
    # one GPU's column shard of a layer split 8 ways by N (tensor parallel:
    # B sliced by columns, A replicated)
    "lm_head_tp8": Workload("lm_head_tp8", 64, 16032, 4096, seed=6, sigma_b=0.02,
                            note="lm_head column shard 64x4096 @ 4096x16032 (1/8 of 128256)"),
    "prefill_up_tp8": Workload("prefill_up_tp8", 2048, 1792, 4096, seed=7, sigma_b=0.02,
                               outlier_frac=0.001,
                               note="prefill up-projection column shard 2048x4096 @ 4096x1792 "
                                    "(1/8 of 14336)"),
}


def _normal(rng, shape, sigma):
    x = rng.standard_normal(shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return x


def make_inputs(w, seed=None):
    """Return (A, B) as float32 numpy arrays for workload ``w``.

    Dense workloads: A is M x K and B is K x N, row-major.  The attention
    workload returns Q as (batch, M, K) and K as (batch, N, K): B is K's
    transpose, which the GEMM reads through its transposed-B layout.
    """
    rng = np.random.default_rng(w.seed if seed is None else seed)
    if w.name == "attn_scores" or w.trans_b:
        q = np.empty((w.batch, w.M, w.K), np.float32)
        k = np.empty((w.batch, w.N, w.K), np.float32)
        for h in range(w.batch):
            q[h] = _normal(rng, (w.M, w.K), w.sigma_a)
            k[h] = _normal(rng, (w.N, w.K), w.sigma_b)
        return q, k
    A = _normal(rng, (w.M, w.K), w.sigma_a)
    B = _normal(rng, (w.K, w.N), w.sigma_b)
    if w.outlier_frac > 0:
        n_out = max(1, int(round(w.outlier_frac * w.K)))
        ch = rng.choice(w.K, n_out, replace=False)
        A[:, ch] *= np.float32(w.outlier_scale)
    return A, B


def random_matrix(shape, seed, sigma=1.0):
    """A seeded N(0, sigma^2) float32 array, for tests of arbitrary shapes."""
    return _normal(np.random.default_rng(seed), shape, sigma)


def integer_matrix(shape, seed, bound):
    """Seeded integers in [-bound, bound] stored as float32."""
    rng = np.random.default_rng(seed)
    return rng.integers(-bound, bound + 1, size=shape).astype(np.float32)

"""A seeded sweep of random shapes through the INT16 dual-FP16 score product.

Each case draws a batch of 1 to 3, M and N (half of them 130..600, half
log-uniform over 1..130), the head size K (1..200: the short-K panel kernel
up to 128, the tiled kernels beyond), padded rows and batch gaps for Q, K
and S, the two maxima and alpha (either sign).  Every batch entry must
meet the oracle's bars (the normwise one on outputs of 256 elements or
more), the padding of S must stay untouched, and a slice of the rows (a
smaller M, which can take another kernel) must give the same bits as those
rows of the whole product.
"""
import numpy as np
import pytest
import torch

from gpu_util import announce, check_tolerance, needs_gpu
import paper_2606_21023_amd as heal

pytestmark = [pytest.mark.gpu, needs_gpu]

CASES = 96


def _draw(i):
    rng = np.random.default_rng(11000 + i)

    def size():
        if rng.random() < 0.5:
            return int(rng.integers(130, 601))
        return max(1, int(np.exp(rng.uniform(0.0, np.log(130.0)))))

    bat = int(rng.integers(1, 4))
    M, N = size(), size()
    K = int(rng.integers(1, 201))
    pads = [int(x) for x in rng.integers(0, 9, size=3)]
    gaps = [int(x) for x in rng.integers(0, 9, size=3)]
    mq = np.float32(np.exp(rng.uniform(-4.0, 6.0)))
    mk = np.float32(np.exp(rng.uniform(-4.0, 6.0)))
    alpha = float(np.float32(rng.choice([1.0, 0.0883883, -0.5])))
    return rng, bat, M, N, K, pads, gaps, mq, mk, alpha


def _strided(buf, bat, rows, cols, ld, stride):
    return buf.as_strided((bat, rows, cols), (stride, ld, 1), 0)


@pytest.mark.parametrize("case", range(CASES))
def test_random_scores(orc, case):
    rng, bat, M, N, K, pads, gaps, mq, mk, alpha = _draw(case)
    ldq, ldk, lds = K + pads[0], K + pads[1], N + pads[2]
    sq, sk, ss = M * ldq + gaps[0], N * ldk + gaps[1], M * lds + gaps[2]
    Qbuf = rng.integers(-32767, 32768, size=bat * sq).astype(np.int16)
    Kbuf = rng.integers(-32767, 32768, size=bat * sk).astype(np.int16)
    what = "case %d: %d x %dx%dx%d, ld %d/%d/%d, max %g/%g, alpha %g" % (
        case, bat, M, N, K, ldq, ldk, lds, mq, mk, alpha)
    announce(what)
    Qd = _strided(torch.from_numpy(Qbuf).cuda(), bat, M, K, ldq, sq)
    Kd = _strided(torch.from_numpy(Kbuf).cuda(), bat, N, K, ldk, sk)
    mqd, mkd = torch.tensor([mq], device="cuda"), torch.tensor([mk], device="cuda")
    Sbuf = torch.full((bat * ss,), float("nan"), device="cuda")
    Sd = _strided(Sbuf, bat, M, N, lds, ss)
    heal.heal_scores_i16(Qd, Kd, mqd, mkd, alpha, out=Sd)
    torch.cuda.synchronize()
    mask = torch.zeros(bat * ss, dtype=torch.bool, device="cuda")
    _strided(mask, bat, M, N, lds, ss).fill_(True)
    assert torch.isnan(Sbuf[~mask]).all(), "%s: padding of S written" % what

    # a slice of the rows, as its own (smaller) call
    r0 = int(rng.integers(0, M))
    r1 = int(rng.integers(r0 + 1, M + 1))
    Ss = heal.heal_scores_i16(Qd[:, r0:r1], Kd, mqd, mkd, alpha)
    torch.cuda.synchronize()
    assert torch.equal(Ss.contiguous().view(torch.int32), Sd[:, r0:r1].contiguous().view(torch.int32)), \
        "%s: rows %d..%d alone differ" % (what, r0, r1)

    S = Sd.cpu().numpy()
    f = orc.scores_factor(mq, mk, alpha)
    for b in range(bat):
        Q = np.lib.stride_tricks.as_strided(Qbuf[b * sq:], (M, K), (2 * ldq, 2))
        Kt = np.lib.stride_tricks.as_strided(Kbuf[b * sk:], (N, K), (2 * ldk, 2))
        Q, Kt = np.ascontiguousarray(Q), np.ascontiguousarray(Kt)
        _, So = orc.scores_i16(Q, Kt, mq, mk, alpha)
        absprod = abs(f) * (np.abs(Q.astype(np.float64)) @ np.abs(Kt.astype(np.float64)).T)
        check_tolerance(S[b], f * So, absprod, "%s, entry %d" % (what, b),
                        normwise_min_elements=256)

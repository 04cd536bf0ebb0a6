"""Host-side logic of the library that needs no GPU: the weight exponent and
the packed sizes, against the oracle and the layout's definition."""
import numpy as np
import pytest

import paper_2606_21023_amd as heal
from paper_2606_21023_amd import build as hbuild
import os


pytestmark = pytest.mark.skipif(not os.path.exists(hbuild.LIBRARY), reason="libheal.so not built")


def test_weight_exponent_matches_oracle(orc):
    rng = np.random.default_rng(3)
    vals = list((np.exp2(rng.uniform(-140, 127, 2000)) * rng.uniform(1, 2, 2000)).astype(np.float32))
    vals += [np.float32(v) for v in (0.0, 1.0, 65504.0, 65505.0, 32752.0, 32753.0, 2.0 ** -149,
                                     3.4e38)]
    for m in vals:
        if not np.isfinite(m):
            continue
        assert heal.heal_f16_weight_exponent(float(m)) == orc.f16_weight_exponent(float(m)), m


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -1.0])
def test_weight_exponent_rejects(bad):
    with pytest.raises(heal.HealError):
        heal.heal_f16_weight_exponent(bad)


def test_packed_size():
    for K, N, P in ((1, 1, 1), (32, 16, 2), (33, 17, 1), (4096, 128256, 1), (0, 5, 2)):
        assert heal.heal_packed_size(K, N, P) == ((N + 15) // 16) * ((K + 31) // 32) * P * 512
    assert heal.lib().heal_packed_size(10, 10, 3) == -1
    assert heal.lib().heal_packed_size(-1, 10, 1) == -1
    assert heal.lib().heal_packed_size((1 << 20) + 1, 10, 1) == -1

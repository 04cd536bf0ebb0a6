"""The CPU oracle against its pins (no GPU)."""
import numpy as np
import pytest

import pins


@pytest.mark.parametrize("pin", pins.SMALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_split_exhaustive_all_fp32(orc):
    """Every one of the 2^32 FP32 bit patterns splits as the library RNE says."""
    chunk = 1 << 26
    for start in range(0, 1 << 32, chunk):
        pins.check_split_range_exhaustive(orc, start, chunk)


def test_split_f16_exhaustive_all_fp32(orc):
    """Every FP32 bit pattern gives the HEAL-Full pair the library casts give."""
    chunk = 1 << 26
    for start in range(0, 1 << 32, chunk):
        pins.check_split_f16_range_exhaustive(orc, start, chunk)


def test_structured_patterns_cover_rounding_classes():
    bits = pins.structured_patterns()
    low = bits & 0xffff
    for v in (0x7fff, 0x8000, 0x8001):
        assert np.count_nonzero(low == v) == 1 << 16

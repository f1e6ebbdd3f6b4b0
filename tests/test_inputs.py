"""Pins of the seeded input module's storage rounding and stream layout.

The 16-bit patterns are checked against values fixed by the formats themselves
(IEEE 754 binary16; bfloat16 = the upper half of a binary32), not against NumPy's
own conversion, including the round-to-nearest-even ties, overflow, subnormals and
NaN handling.
"""

import numpy as np
import pytest

from paper_2511_01385_amd import inputs

# (value, bfloat16 bits): exact, ties to even both ways, the largest finite, overflow
BF16 = [
    (1.0, 0x3F80),
    (-2.0, 0xC000),
    (1.0 + 2.0**-8, 0x3F80),  # tie, rounds down to the even mantissa
    (1.0 + 3 * 2.0**-8, 0x3F82),  # tie, rounds up to the even mantissa
    (1.0 + 2.0**-8 + 2.0**-20, 0x3F81),  # above the tie
    (3.3895313892515355e38, 0x7F7F),  # largest finite bfloat16
    (np.inf, 0x7F80),
    (-np.inf, 0xFF80),
    (0.0, 0x0000),
    (-0.0, 0x8000),
    (2.0**-133, 0x0001),  # smallest subnormal
]

# (value, binary16 bits)
F16 = [
    (1.0, 0x3C00),
    (-2.0, 0xC000),
    (1.0 / 3.0, 0x3555),
    (1.0 + 2.0**-11, 0x3C00),  # tie, down to even
    (1.0 + 3 * 2.0**-11, 0x3C02),  # tie, up to even
    (65504.0, 0x7BFF),  # largest finite
    (65520.0, 0x7C00),  # halfway to 2^16 rounds to infinity
    (2.0**-24, 0x0001),  # smallest subnormal
    (2.0**-14, 0x0400),  # smallest normal
    (2.0**-26, 0x0000),  # below half the smallest subnormal
    (-0.0, 0x8000),
]


@pytest.mark.parametrize("value,bits", BF16)
def test_bf16_rounding(value, bits):
    got = inputs.round_to(np.array([value]), "bf16")
    assert got.dtype == np.uint16 and int(got[0]) == bits


@pytest.mark.parametrize("value,bits", F16)
def test_f16_rounding(value, bits):
    got = inputs.round_to(np.array([value]), "f16")
    assert got.dtype == np.uint16 and int(got[0]) == bits


@pytest.mark.filterwarnings("ignore:invalid value encountered in cast")
def test_widening_is_exact():
    # every 16-bit pattern widens to the value its fields encode
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    sign = np.where(bits >> 15, -1.0, 1.0)
    e = ((bits >> 10) & 0x1F).astype(np.int64)
    m = (bits & 0x3FF).astype(np.float64)
    fin = e < 31
    want = np.where(e == 0, sign * m * 2.0**-24, sign * (1 + m / 1024) * np.exp2(e - 15.0))
    got = inputs.to_f64(bits, "f16")
    assert np.array_equal(got[fin], want[fin])
    assert np.isinf(got[(e == 31) & (m == 0)]).all() and np.isnan(got[(e == 31) & (m != 0)]).all()
    e8 = ((bits >> 7) & 0xFF).astype(np.int64)
    m8 = (bits & 0x7F).astype(np.float64)
    fin8 = e8 < 255
    want8 = np.where(e8 == 0, sign * m8 * 2.0**-133, sign * (1 + m8 / 128) * np.exp2(e8 - 127.0))
    assert np.array_equal(inputs.to_f64(bits, "bf16")[fin8], want8[fin8])


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_round_trip_of_every_pattern(dtype):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = inputs.to_f64(bits, dtype)
    fin = np.isfinite(v)
    back = inputs.round_to(v[fin], dtype)
    assert np.array_equal(back, bits[fin])


def test_bf16_nan_stays_nan():
    got = inputs.round_to(np.array([np.nan, -np.nan]), "bf16")
    assert np.isnan(inputs.to_f64(got, "bf16")).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_normal_rows_block_draw_is_one_stream(dtype):
    # drawing in row blocks consumes the stream exactly as one draw of the whole array
    rows, n = 3000, 512  # crosses the 2^20-element block boundary
    got = inputs.normal_rows(11, rows, n, dtype, sigma=0.5)
    want = inputs.round_to(inputs.generator(11).standard_normal((rows, n)) * 0.5, dtype)
    assert np.array_equal(got, want)

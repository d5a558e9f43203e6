"""Pins for the oracle's bfloat16 rounding (round to nearest, ties to even)."""
import numpy as np
import pytest

from oracle.bf16 import round_bf16


def _bits_round_f32(x32):
    """Independent check: round float32 bit patterns to bf16 by integer arithmetic.

    Keep the top 16 bits; look at the dropped 16 bits: above half rounds up,
    below half rounds down, exactly half rounds to the even kept pattern.
    """
    u = x32.view(np.uint32).astype(np.uint64)
    keep = u >> 16
    drop = u & 0xFFFF
    up = (drop > 0x8000) | ((drop == 0x8000) & ((keep & 1) == 1))
    keep = keep + up.astype(np.uint64)
    return (keep << 16).astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("x,expect", [
    (1.0 + 2.0 ** -8, 1.0),                       # tie -> even (1.0)
    (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),       # tie -> even (mantissa ...10)
    (1.0 + 2.0 ** -8 + 2.0 ** -20, 1.0 + 2.0 ** -7),  # just above the tie
    (-(1.0 + 3 * 2.0 ** -8), -(1.0 + 2.0 ** -6)),
    (2.0 ** -133, 2.0 ** -133),                   # smallest subnormal is on the grid
    (2.0 ** -134, 0.0),                           # tie between 0 and 2^-133 -> 0
    (3 * 2.0 ** -134, 2.0 ** -132),               # tie -> even
    ((2.0 - 2.0 ** -7) * 2.0 ** 127, (2.0 - 2.0 ** -7) * 2.0 ** 127),  # max finite
    (2.0 ** 128 * (1 - 2.0 ** -9), np.inf),       # the tie above max rounds to inf
    (0.1, 0.10009765625),
    (3.14159265358979, 3.140625),
])
def test_round_bf16_cases(x, expect):
    assert round_bf16(np.array([x]))[0] == expect


def test_round_bf16_specials():
    r = round_bf16(np.array([np.nan, np.inf, -np.inf, 0.0, -0.0]))
    assert np.isnan(r[0]) and r[1] == np.inf and r[2] == -np.inf
    assert r[3] == 0.0 and np.signbit(r[4])


def test_round_bf16_matches_bit_rounding_of_float32():
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
        # exact ties and their neighbours
        (rng.integers(1, 2 ** 16, 5000).astype(np.uint32) << 16 | 0x8000).view(np.float32),
    ]).astype(np.float32)
    x = x[np.isfinite(x)]
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), _bits_round_f32(x))


def test_round_bf16_idempotent_and_monotone():
    rng = np.random.default_rng(2)
    x = np.sort(rng.standard_normal(10000))
    r = round_bf16(x)
    np.testing.assert_array_equal(round_bf16(r), r)
    assert np.all(np.diff(r) >= 0)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0 ** -8)

"""Pins for the oracle's number formats (no GPU).

The bf16 format's facts are fixed by its definition (1 sign, 8 exponent and
7 fraction bits, IEEE round to nearest even); the float32 -> bf16 special case
is checked against torch's own conversion, a library routine the oracle does
not call.
"""
import numpy as np
import pytest
import torch

from oracle import decode_bf16, encode_bf16, round_bf16, round_f32


def test_decode_known_patterns():
    bits = np.array([0x3F80, 0xBF80, 0x4000, 0x7F80, 0xFF80, 0x0001, 0x0080, 0x7F7F, 0x8000],
                    dtype=np.uint16)
    v = decode_bf16(bits)
    assert v[0] == 1.0 and v[1] == -1.0 and v[2] == 2.0
    assert np.isposinf(v[3]) and np.isneginf(v[4])
    assert v[5] == 2.0 ** -133                      # smallest subnormal
    assert v[6] == 2.0 ** -126                      # smallest normal
    assert v[7] == (2 - 2.0 ** -7) * 2.0 ** 127     # largest finite
    assert v[8] == 0.0 and np.signbit(v[8])


def test_ties_to_even_and_single_rounding():
    one = 1.0
    ulp = 2.0 ** -7                                  # bf16 spacing in [1, 2)
    x = np.array([one + ulp / 2,                     # tie, 1.0 is even -> 1.0
                  one + 3 * ulp / 2,                 # tie, odd below -> up
                  one + ulp / 2 + 2.0 ** -40,        # just above the tie -> up
                  -(one + ulp / 2 + 2.0 ** -40)])
    r = round_bf16(x)
    assert r[0] == 1.0
    assert r[1] == one + 2 * ulp
    # A float64 -> float32 -> bf16 chain would first land exactly on the tie
    # (2**-40 is below float32's half spacing) and then round down to 1.0.
    assert r[2] == one + ulp
    assert r[3] == -(one + ulp)
    assert float(np.float32(x[2])) == one + ulp / 2   # the double-rounding trap is real


def test_overflow_subnormal_zero_nan():
    big = (2 - 2.0 ** -7) * 2.0 ** 127
    half_ulp = 2.0 ** 119
    x = np.array([big, big + half_ulp * 0.99, big + half_ulp, -(big + half_ulp),
                  2.0 ** -133, 2.0 ** -134, 0.75 * 2.0 ** -133, 1.5 * 2.0 ** -133,
                  -0.0, np.inf, np.nan])
    r = round_bf16(x)
    assert r[0] == big and r[1] == big
    assert np.isposinf(r[2]) and np.isneginf(r[3])   # tie at the top rounds to even = 2**128
    assert r[4] == 2.0 ** -133
    assert r[5] == 0.0                               # tie between 0 and 2**-133 -> 0 (even)
    assert r[6] == 2.0 ** -133
    assert r[7] == 2.0 ** -132                       # tie between 1 and 2 quanta -> 2 (even)
    assert r[8] == 0.0 and np.signbit(r[8])
    assert np.isposinf(r[9]) and np.isnan(r[10])
    assert encode_bf16(np.array([np.nan]))[0] == 0x7FC0


@pytest.mark.parametrize("seed", [0, 1])
def test_matches_torch_for_float32_inputs(seed):
    rng = np.random.default_rng(seed)
    # random bit patterns cover every binade incl. subnormals; drop NaNs
    u = rng.integers(0, 2 ** 32, size=200_000, dtype=np.uint64).astype(np.uint32)
    f = u.view(np.float32)
    f = f[~np.isnan(f)]
    ours = encode_bf16(f.astype(np.float64))
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_roundtrip_exact_for_representable():
    bits = np.arange(0, 2 ** 16, dtype=np.uint32).astype(np.uint16)
    v = decode_bf16(bits)
    ok = ~np.isnan(v)
    assert np.array_equal(encode_bf16(v[ok]), bits[ok])


def test_round_f32():
    x = np.array([1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24, 0.1])
    r = round_f32(x)
    assert r[0] == 1.0 and r[1] == 1.0 + 2.0 ** -22
    assert r[2] == float(np.float32(0.1))

"""Pins for the FP8 E4M3 codec of the oracle: the format's fixed points,
agreement with an independent implementation (torch.float8_e4m3fn casts)
on every code and on random and tie-point inputs, and the power-of-two
scale rule."""
import math

import numpy as np
import pytest

from oracle import fp8


def test_fixed_points():
    t = fp8.e4m3_table()
    assert t[0x38] == 1.0 and t[0x7E] == 448.0 and t[0xFE] == -448.0
    assert t[0x01] == 2.0 ** -9 and t[0x08] == 2.0 ** -6 and t[0x07] == 7 * 2.0 ** -9
    assert math.isnan(t[0x7F]) and math.isnan(t[0xFF])
    assert t[0x00] == 0.0 and t[0x80] == 0.0
    finite = t[np.isfinite(t)]
    assert finite.size == 254 and np.max(finite) == 448.0


def test_every_code_round_trips():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF, 0x80)], dtype=np.uint8)
    np.testing.assert_array_equal(fp8.encode(fp8.decode(codes)), codes)


def _torch_codes(x):
    import torch
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_agrees_with_torch_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * s for s in (1e-3, 1e-1, 1.0, 30.0, 200.0)])
    x = np.clip(x, -448, 448).astype(np.float32)
    np.testing.assert_array_equal(fp8.encode(x), _torch_codes(x))
    # midpoints between neighbouring values: ties go to the even code
    v = fp8.e4m3_table()[: 0x7E]
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    np.testing.assert_array_equal(fp8.encode(mids), _torch_codes(mids))
    np.testing.assert_array_equal(fp8.encode(-mids), _torch_codes(-mids))
    assert np.all(fp8.encode(mids) % 2 == 0)


def test_saturation_and_signed_zero():
    assert fp8.encode(np.array([500.0, -1e9]))[0] == 0x7E
    assert fp8.encode(np.array([-1e9]))[0] == 0xFE
    assert fp8.encode(np.array([-1e-6]))[0] == 0x80 and fp8.encode(np.array([1e-6]))[0] == 0x00


@pytest.mark.parametrize("amax", [1.0, 448.0, 449.0, 3.5, 0.001, 1e-15, 7e4, 1e18, 2.0 ** -52, 2.0 ** 68])
def test_pow2_scale(amax):
    s = fp8.pow2_scale(amax)
    assert math.log2(s) == int(math.log2(s))                 # a power of two
    assert amax * s <= 448.0 < amax * s * 2                  # the largest one
    assert fp8.pow2_scale(0.0) == 1.0


def test_pow2_scale_clamp():
    # exponents outside [-60, 60] are clamped, so that s and the inverse of a
    # product of two scales, 1 / (s s'), stay finite normal fp32 numbers
    assert fp8.pow2_scale(2.0 ** -52) == 2.0 ** 60          # 2^-52 2^60 = 256 <= 448 < 512: not clamped
    assert fp8.pow2_scale(2.0 ** -53) == 2.0 ** 60          # would be 2^61: clamped
    assert fp8.pow2_scale(1e-30) == 2.0 ** 60
    assert fp8.pow2_scale(2.0 ** 68) == 2.0 ** -60          # 2^68 2^-60 = 256: not clamped
    assert fp8.pow2_scale(2.0 ** 69) == 2.0 ** -60          # would be 2^-61: clamped
    assert fp8.pow2_scale(1e30) == 2.0 ** -60
    tiny = np.finfo(np.float32).tiny
    for s1, s2 in [(2.0 ** 60, 2.0 ** 60), (2.0 ** -60, 2.0 ** -60)]:
        inv = np.float32(1.0) / (np.float32(s1) * np.float32(s2))
        assert np.isfinite(inv) and inv >= tiny
    # at the lower clamp the codes saturate instead of overflowing
    codes, s = fp8.quantize(np.array([1e30, -1e30, 1.0], dtype=np.float32))
    assert s == 2.0 ** -60 and list(codes[:2]) == [0x7E, 0xFE]


def test_quantize_exact_scaling():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((64, 48)) * 3).astype(np.float32)
    codes, s = fp8.quantize(x)
    back = fp8.dequantize(codes, s)
    # every element within half an E4M3 step (relative 2^-4 for normals)
    rel = np.abs(back - x) / np.maximum(np.abs(x), 2.0 ** -6 / s)
    assert np.max(rel) <= 2.0 ** -4 + 1e-12
    assert np.max(np.abs(x)) * s <= 448.0

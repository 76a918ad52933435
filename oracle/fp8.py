"""OCP FP8 E4M3 ("e4m3fn") codec and per-tensor power-of-two scaling for the
mixed-precision layer (test infrastructure only).

The appendix on mixed-precision training runs the contractions that involve
the batch dimension in FP8 and keeps the batch-free ones in full precision;
it fixes neither the FP8 format nor the scaling.  Readings used here (the
same on the GPU side):

* format: E4M3 with 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits,
  no infinities, code 0x7F / 0xFF = NaN; normal values 2^(e-7) (1 + m/8) for
  e = 1..15 (but not e = 15, m = 7), subnormals 2^-6 m/8; largest 448;
* rounding: to the nearest representable value, ties to the even code
  (mantissa LSB 0), magnitudes above 448 saturate to 448;
* scaling: one power of two per tensor, s = 2^e with e the largest integer
  such that amax * s <= 448 (amax = max |x| of the fp32 values; s = 1 when
  amax = 0), e clamped to [-60, 60] so that s and the product scales
  1 / (s s') of two tensors stay finite normal fp32 numbers.  x * s is then
  exact in fp32, so the only rounding decision is the FP8 one, taken on the
  fp32 value x * s.

Written from the format's definition with numpy; pinned against an
independent implementation (torch.float8_e4m3fn casts) and the format's
fixed points in tests/test_oracle_fp8.py.
"""
from __future__ import annotations

import math

import numpy as np

E4M3_MAX = 448.0


def e4m3_table() -> np.ndarray:
    """Value of each of the 256 codes (NaN for 0x7F and 0xFF), float64."""
    vals = np.empty(256)
    for code in range(256):
        s = -1.0 if code & 0x80 else 1.0
        e = (code >> 3) & 0xF
        m = code & 0x7
        if e == 0xF and m == 0x7:
            vals[code] = np.nan
        elif e == 0:
            vals[code] = s * 2.0 ** -6 * (m / 8.0)
        else:
            vals[code] = s * 2.0 ** (e - 7) * (1.0 + m / 8.0)
    return vals


_TABLE = e4m3_table()
_POS_CODES = np.arange(0, 0x7F)                 # 0x00 .. 0x7E: the non-negative finite codes, increasing
_POS_VALS = _TABLE[_POS_CODES]


def decode(codes) -> np.ndarray:
    return _TABLE[np.asarray(codes, dtype=np.uint8)]


def encode(x) -> np.ndarray:
    """Round to the nearest E4M3 value (ties to the even code), saturating."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.searchsorted(_POS_VALS, a, side="left")          # first value >= a
    hi = np.minimum(hi, _POS_VALS.size - 1)
    lo = np.maximum(hi - 1, 0)
    dlo = a - _POS_VALS[lo]
    dhi = _POS_VALS[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (_POS_CODES[hi] % 2 == 0) & (hi != lo))
    code = np.where(pick_hi, _POS_CODES[hi], _POS_CODES[lo]).astype(np.uint8)
    code = np.where(a == _POS_VALS[hi], _POS_CODES[hi], code).astype(np.uint8)
    # the sign bit is kept, also for values that round to zero (-0 = 0x80)
    return (code | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)


E_MIN, E_MAX = -60, 60


def pow2_scale(amax: float) -> float:
    """Largest power of two s = 2^e with amax * s <= 448, e clamped to
    [E_MIN, E_MAX] (1 when amax is 0)."""
    amax = float(amax)
    if amax == 0.0 or not math.isfinite(amax):
        return 1.0
    f, k = math.frexp(amax)                      # amax = f 2^k, 0.5 <= f < 1
    e = 9 - k if f <= 0.875 else 8 - k           # 448 = 0.875 2^9
    return math.ldexp(1.0, min(max(e, E_MIN), E_MAX))


def quantize(x) -> tuple:
    """(codes, s) for a tensor: s from the fp32 amax, codes of the fp32 x * s."""
    x32 = np.asarray(x, dtype=np.float32)
    s = pow2_scale(float(np.max(np.abs(x32))) if x32.size else 0.0)
    return encode((x32 * np.float32(s)).astype(np.float64)), s


def dequantize(codes, s: float) -> np.ndarray:
    return decode(codes) / s

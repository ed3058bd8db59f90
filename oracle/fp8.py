"""OCP FP8 E4M3 quantization (oracle; test infrastructure only).

What it serves: the fp8 inference variant of the cached chunk attention, which
follows the deployment direction the paper names at its end (Sec. 6,
"Efficient deployment": quantization to cut inference latency and cost).  The
paper fixes no format; the reading taken here:

- The format is E4M3 of the OCP 8-bit floating point specification (the
  "fn" variant): 1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits.
  Exponent field 0 holds the subnormals m * 2^-9; exponent field e > 0 holds
  (1 + m/8) * 2^(e-7); the single code pair S.1111.111 is NaN and there are no
  infinities, so the largest finite magnitude is 1.75 * 2^8 = 448.
- One scale per tensor, value = decode(code) * scale.  A bf16 tensor x is
  quantized as code = RNE(clamp(fl32(x * fl32(1 / scale)), -448, 448)):
  fl32 is rounding to fp32 (nearest even), 1/scale is an fp32 division, and
  RNE takes the nearest finite E4M3 value, a tie going to the code with the
  even (zero) last mantissa bit.  The sign of the code is the sign bit of the
  clamped product (so -0 and negative values that round to zero give 0x80).

Encoding is done by brute force over the table of all finite E4M3 values, so
it can be read against the definition above without any bit tricks.
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    """float64 value of each E4M3 code (uint8); NaN for 0x7F and 0xFF."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = c >> 7
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(sign == 1, -mag, mag)


# non-negative finite values, indexed by code 0x00 .. 0x7E (increasing with the code)
_POS = e4m3_decode(np.arange(0x7F))


def e4m3_encode(x) -> np.ndarray:
    """Nearest E4M3 code (ties to even) of finite values with |x| <= 448."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)) or np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("e4m3_encode takes finite values within +-448 (clamp first)")
    a = np.abs(x).ravel()
    hi = np.clip(np.searchsorted(_POS, a, side="left"), 0, len(_POS) - 1)  # first table value >= a
    lo = np.maximum(hi - 1, 0)
    d_hi = _POS[hi] - a
    d_lo = a - _POS[lo]
    take_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(take_lo, lo, hi)
    code = np.where(a == _POS[hi], hi, code)  # exact values
    sign = np.signbit(x).ravel().astype(np.int64)
    return (code | (sign << 7)).astype(np.uint8).reshape(x.shape)


def quantize_fp8(x, scale: float) -> np.ndarray:
    """Codes of x (bf16 values, any float dtype holding them) at per-tensor `scale`."""
    inv = np.float32(1.0) / np.float32(scale)
    y = np.asarray(x, dtype=np.float32) * inv                      # fl32(x * fl32(1/scale))
    y = np.clip(y, np.float32(-E4M3_MAX), np.float32(E4M3_MAX))
    return e4m3_encode(y)


def dequantize_fp8(codes, scale: float) -> np.ndarray:
    """float64 value of each code at per-tensor `scale`."""
    return e4m3_decode(codes) * float(np.float32(scale))

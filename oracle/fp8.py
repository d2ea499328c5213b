"""8-bit floating-point KV cache codes (E4M3) for the oracle.

TEST INFRASTRUCTURE ONLY: only tests, the package smoke check and the
benchmark's CPU-baseline leg call this.  It shares no code with the HIP path.

The paper runs its engine in BF16 (Sec. 4.1 "Implementation"); an 8-bit KV
cache is this build's variant on the same path (it halves the bytes a decode
step streams, the cost the paper attributes to decode attention: Sec. 1,
App. A.2).  The format is the public OCP 8-bit floating point E4M3 encoding:

  bit 7 sign, bits 6..3 exponent e (bias 7), bits 2..0 mantissa m;
  e = 0:           value = m * 2^-9            (subnormals, and +-0)
  1 <= e <= 15:    value = (1 + m / 8) * 2^(e - 7)
  e = 15, m = 7:   NaN (the only non-finite codes: 0x7F, 0xFF); no infinity
  largest finite:  0x7E = 448.

Cache semantics used throughout: the code of a value is
e4m3(bf16(value) / scale) with the division in float32, rounded to nearest
(ties to even) and saturated to +-448 beyond the largest finite value (also
for +-inf); NaN encodes as 0x7F with the input's sign.  A cached code reads
back as decode(code) * scale.

8-bit weights: a projection W [out, in] is held as codes with one scale per
output row; the weight it stands for is decode(code[n][k]) * scale[n].
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
MIN_NORMAL = 2.0 ** -6


def e4m3_decode(codes) -> np.ndarray:
    """Value (float64) of each E4M3 code (uint8 array)."""
    c = np.asarray(codes).astype(np.int64) & 0xFF
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0))
    mag = np.where((e == 15) & (c & 0x7 == 7), np.nan, mag)
    return sign * mag


def e4m3_encode(x) -> np.ndarray:
    """Nearest E4M3 code (ties to even, saturating) of each value of x."""
    x = np.asarray(x, dtype=np.float64)
    sign = np.signbit(x).astype(np.int64) << 7
    a = np.abs(x)
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        # normal range: a = (1 + f) 2^e with e = floor(log2 a); 3 mantissa bits
        mant, ex = np.frexp(np.where(a > 0, a, 1.0))     # a = mant 2^ex, mant in [0.5, 1)
        e = ex - 1
        q = np.rint((2.0 * mant - 1.0) * 8.0).astype(np.int64)   # 0..8, 8 carries into e
        normal = ((e + 7) << 3) + q
        # subnormal range: multiples of 2^-9
        sub = np.rint(a * 2.0 ** 9).astype(np.int64)               # 0..8 (8 = smallest normal)
    code = np.where(a < MIN_NORMAL, sub, normal)
    code = np.where(a >= E4M3_MAX, 0x7E, np.minimum(code, 0x7E))
    code = np.where(np.isnan(x), 0x7F, code)
    return (code | sign).astype(np.uint8)


def quantize_cache_value(bf16_value_f32, scale: float) -> np.ndarray:
    """Cache code of values that are already bf16 numbers (float32 array):
    e4m3(value / scale), the division rounded in float32."""
    v = np.asarray(bf16_value_f32, dtype=np.float32)
    return e4m3_encode((v / np.float32(scale)).astype(np.float32))


def dequantize(codes, scale: float) -> np.ndarray:
    """Values a cached code stands for: decode(code) * scale (float64)."""
    return e4m3_decode(codes) * float(scale)


def dequantize_rows(codes, scales) -> np.ndarray:
    """Weights 8-bit codes [out, in] with one scale per output row stand for:
    decode(code[n][k]) * scales[n] (float64)."""
    return e4m3_decode(codes) * np.asarray(scales, np.float64)[:, None]

"""FP8 KV-cache quantization on top of DMS.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module; the GPU library never calls it and shares no code with it.

The paper lists KV quantization (per-channel / per-token schemes such as KIVI
and KVQuant) among methods orthogonal to DMS that could be combined with it
(App. B, related work on KV cache size reduction).  The combination built
here stores every retained key and value row in OCP FP8 E4M3 with one
power-of-two scale per (token, KV head) row for K and one for V:

* E4M3 (OCP 8-bit floating point, "FN" variant): sign, 4 exponent bits with
  bias 7, 3 mantissa bits; exponent field 0 encodes subnormals m * 2^-9;
  S.1111.111 is NaN; there are no infinities; the largest finite value is
  448 = 1.75 * 2^8.  Encoding rounds to nearest, ties to even.
* Row scale 2^e with e the smallest integer such that amax * 2^-e <= 448,
  amax = max |x| over the row (e = 0 for an all-zero row): the row's largest
  element lands in (224, 448] and no element overflows.  The code of x is
  E4M3(x * 2^-e) (exact scaling, then one rounding); the stored value is
  decode(code) * 2^e.  A power-of-two scale keeps dequantization exact in
  any binary format wide enough, which is why it is used (as in OCP MX).

Readings (not fixed by the paper, which only names quantization as
orthogonal): per-token scales for both K and V; every key and value is
attended in its stored (quantized) form, including the token appended by the
same decode step.
"""
from __future__ import annotations

import numpy as np

__all__ = ["E4M3_MAX", "e4m3_decode", "e4m3_encode", "fp8_row_exponent", "quantize_rows_fp8",
           "dequantize_rows_fp8", "fake_quantize_fp8"]

E4M3_MAX = 448.0


def e4m3_decode(codes):
    """uint8 codes -> float64 values (NaN for S.1111.111)."""
    c = np.asarray(codes, np.int64) & 0xFF
    sign = np.where(c & 0x80, -1.0, 1.0)
    exp = (c >> 3) & 0xF
    man = c & 0x7
    mag = np.where(exp == 0, man * 2.0 ** -9, (1.0 + man / 8.0) * np.exp2(exp - 7.0))
    mag = np.where((exp == 0xF) & (man == 0x7), np.nan, mag)
    return sign * mag


def e4m3_encode(x):
    """Finite values with |x| <= 448 -> uint8 codes, round to nearest even.

    Normal range (|x| >= 2^-6): |x| = (1 + f) 2^E with E = floor(log2 |x|);
    the 3-bit mantissa is rint(8 f) (half to even), a carry to 8 moves to the
    next binade.  Below 2^-6 the code is the subnormal rint(|x| 2^9)
    (a result of 8 is the smallest normal, code 0x08).  The sign bit is kept,
    also for zero.
    """
    x = np.asarray(x, np.float64)
    if np.any(~np.isfinite(x)) or np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("e4m3_encode takes finite values with |x| <= 448")
    a = np.abs(x)
    sign = np.where(np.signbit(x), 0x80, 0)
    # subnormal branch
    sub = np.rint(a * 2.0 ** 9).astype(np.int64)          # 0 .. 8 (8 = 0x08, the smallest normal)
    # normal branch
    m, E = np.frexp(np.where(a > 0, a, 1.0))                 # a = m 2^E, m in [0.5, 1)
    E = E - 1                                                # a = (2m) 2^E, 2m in [1, 2)
    frac = 2.0 * m - 1.0
    mant = np.rint(frac * 8.0).astype(np.int64)
    carry = mant == 8
    mant = np.where(carry, 0, mant)
    E = np.where(carry, E + 1, E)
    normal = (E + 7) * 8 + mant
    code = np.where(a < 2.0 ** -6, sub, normal)
    return (code | sign).astype(np.uint8)


def fp8_row_exponent(amax):
    """Smallest integer e with amax * 2^-e <= 448 (0 for amax = 0)."""
    a = np.asarray(amax, np.float64)
    m, E = np.frexp(np.where(a > 0, a, 1.0))                 # a = m 2^E, m in [0.5, 1)
    # 448 = 0.875 * 2^9: m <= 0.875 -> a * 2^-(E-9) = m 2^9 <= 448, else one more
    e = np.where(m <= 0.875, E - 9, E - 8)
    return np.where(a > 0, e, 0).astype(np.int64)


def quantize_rows_fp8(x):
    """Rows of the last axis -> (codes uint8, exponent e per row) with the row
    scale 2^e (x is taken as float32 values, e.g. bf16 inputs)."""
    x = np.asarray(x, np.float32).astype(np.float64)
    e = fp8_row_exponent(np.max(np.abs(x), axis=-1))
    q = x * np.exp2(-e.astype(np.float64))[..., None]
    return e4m3_encode(q), e


def dequantize_rows_fp8(codes, e):
    return e4m3_decode(codes) * np.exp2(np.asarray(e, np.float64))[..., None]


def fake_quantize_fp8(x):
    """x -> decode(encode(x * 2^-e)) * 2^e row by row (float64)."""
    codes, e = quantize_rows_fp8(x)
    return dequantize_rows_fp8(codes, e)

"""Storage formats of the KV cache, decoded to fp64.  Test infrastructure only.

bf16: sign, 8 exponent bits (bias 127), 7 fraction bits; the value is the
float32 whose upper 16 bits are the pattern.

OCP 8-bit floating point E4M3FN (the fp8 KV format): sign, 4 exponent bits
(bias 7), 3 mantissa bits; no infinities; S.1111.111 is NaN; exponent field
0 encodes subnormals m * 2^-9.  Largest finite magnitude 1.75 * 2^8 = 448.

Encoding (quantise-on-append of a decode step's K/V into an fp8 block): the
code of a finite value y is the E4M3FN value nearest to |y|, ties to the code
with an even mantissa, magnitudes beyond 448 saturating to 448, with y's
sign (so -0 gives 0x80).  The value quantised is y = x / s rounded to fp32 (x
the bf16 element, s the block's fp32 scale): a rounding decides an integer
here, so the oracle takes it in the precision the kernel computes in.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def e4m3fn_to_f64(codes: np.ndarray) -> np.ndarray:
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    normal = sign * (1.0 + m / 8.0) * np.exp2(e - 7.0)
    sub = sign * (m / 8.0) * 2.0 ** -6
    out = np.where(e == 0, sub, normal)
    nan = (e == 0xF) & (m == 0x7)
    return np.where(nan, np.nan, out)


def decode(codes: np.ndarray, kv_dtype: str) -> np.ndarray:
    if kv_dtype == "bf16":
        return bf16_to_f64(codes)
    if kv_dtype == "fp8_e4m3":
        return e4m3fn_to_f64(codes)
    raise ValueError(kv_dtype)


# The 127 non-negative finite E4M3FN values, indexed by code 0x00 .. 0x7E.
_E4M3_POS = None


def _e4m3_table() -> np.ndarray:
    global _E4M3_POS
    if _E4M3_POS is None:
        _E4M3_POS = e4m3fn_to_f64(np.arange(0x7F, dtype=np.uint8))
    return _E4M3_POS


def f64_to_e4m3fn(y: np.ndarray) -> np.ndarray:
    """Codes of finite values y: nearest value, ties to the even code, saturating."""
    y = np.asarray(y, dtype=np.float64)
    if not np.isfinite(y).all():
        raise ValueError("E4M3FN encoding of a non-finite value")
    vals = _e4m3_table()
    a = np.abs(y).reshape(-1)
    hi = np.minimum(np.searchsorted(vals, a, side="left"), len(vals) - 1)  # vals[hi] >= a below 448
    lo = np.maximum(hi - 1, 0)
    dlo, dhi = a - vals[lo], vals[hi] - a
    tie_even = np.where(lo % 2 == 0, lo, hi)
    out = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, tie_even))
    out = np.where(vals[hi] == a, hi, out)
    out = np.where(a >= vals[-1], 0x7E, out).astype(np.uint8)
    out |= np.where(np.signbit(y).reshape(-1), 0x80, 0).astype(np.uint8)
    return out.reshape(y.shape)


def quantise_e4m3fn(x: np.ndarray, scale: float) -> np.ndarray:
    """Codes of x / scale, the quotient rounded to fp32 first (x: fp64 values of bf16)."""
    q = np.asarray(x, dtype=np.float32) / np.float32(scale)
    return f64_to_e4m3fn(q.astype(np.float64))

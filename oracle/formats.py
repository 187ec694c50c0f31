"""Storage formats of the KV cache, decoded to fp64.  Test infrastructure only.

bf16: sign, 8 exponent bits (bias 127), 7 fraction bits; the value is the
float32 whose upper 16 bits are the pattern.

OCP 8-bit floating point E4M3FN (the fp8 KV format): sign, 4 exponent bits
(bias 7), 3 mantissa bits; no infinities; S.1111.111 is NaN; exponent field
0 encodes subnormals m * 2^-9.  Largest finite magnitude 1.75 * 2^8 = 448.
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

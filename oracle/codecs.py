"""Bit-pattern decoders used by the oracle.

bf16 is the upper half of an IEEE-754 binary32, so decoding is a 16-bit left
shift. OCP FP8 E4M3FN (the OCP 8-bit floating point specification, "E4M3"
variant with finite-only encoding): 1 sign bit, 4 exponent bits with bias 7, 3
mantissa bits; exponent field 0 encodes subnormals m * 2^-9; S.1111.111 is NaN;
there is no infinity, so S.1111.110 = +-448 is the largest finite value.
"""

import numpy as np


def bf16_bits_to_f64(u16: np.ndarray) -> np.ndarray:
    u32 = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def e4m3fn_value(code: int) -> float:
    """Value of one E4M3FN code, read field by field."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    exp_field = (code >> 3) & 0xF
    mant = code & 0x7
    if exp_field == 0xF and mant == 0x7:
        return float("nan")
    if exp_field == 0:
        return sign * mant * 2.0 ** -9
    return sign * (1.0 + mant / 8.0) * 2.0 ** (exp_field - 7)


E4M3FN_TABLE = np.array([e4m3fn_value(c) for c in range(256)], dtype=np.float64)


def e4m3fn_bits_to_f64(u8: np.ndarray) -> np.ndarray:
    return E4M3FN_TABLE[np.asarray(u8, dtype=np.uint8)]


def storage_to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(x)
    if dtype == "fp8":
        return e4m3fn_bits_to_f64(x)
    raise ValueError(dtype)


# Finite non-negative E4M3FN values in code order (codes 0x00 .. 0x7E); the
# value grows with the code, so nearest-value search is a sorted search.
_POS_VALUES = E4M3FN_TABLE[:0x7F]


def e4m3fn_encode(y: np.ndarray) -> np.ndarray:
    """float32 -> E4M3FN codes: the nearest finite value, ties to the code with
    an even mantissa (round to nearest even), magnitudes beyond 448 saturate
    to +-448, the sign of zero is kept. Found by searching the value table,
    not by manipulating bits."""
    y = np.asarray(y, dtype=np.float32).astype(np.float64)
    a = np.minimum(np.abs(y), 448.0)
    hi = np.searchsorted(_POS_VALUES, a, side="left")          # first value >= a
    hi = np.minimum(hi, 0x7E)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _POS_VALUES[lo]
    d_hi = _POS_VALUES[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo)
    code = np.where(a == _POS_VALUES[hi], hi, code)             # exact hits
    sign = np.signbit(y)
    return (code | (sign.astype(np.int64) << 7)).astype(np.uint8)

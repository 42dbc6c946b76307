"""Exponent / sign / mantissa of bf16 values derived from their *value*.

Used by the tests to pin the oracle to something other than itself: the
oracle extracts fields with bit masks; here the fields come from IEEE-754
semantics (bf16 is binary32 with the low 16 bits dropped) through frexp and
magnitude comparisons. A transposed shift, a wrong mask or a wrong packing
order in the oracle disagrees with these on some value.
"""
import numpy as np


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def _to_f64(bits):
    # signalling-NaN patterns raise a harmless "invalid" flag in the cast
    with np.errstate(invalid="ignore"):
        return bf16_to_f32(bits).astype(np.float64)


def exponent_field(bits: np.ndarray) -> np.ndarray:
    """Biased 8-bit exponent: 0 for zero and subnormals, 255 for Inf/NaN,
    otherwise floor(log2|x|) + 127 (frexp returns |m| in [0.5, 1))."""
    x = _to_f64(bits)
    out = np.zeros(x.shape, np.int64)
    special = ~np.isfinite(x)
    out[special] = 255
    ax = np.abs(np.where(special, 0.0, x))
    normal = ax >= 2.0 ** -126
    _, ex = np.frexp(ax[normal])
    out[normal] = ex + 126
    return out.astype(np.uint8)


def sign_bit(bits: np.ndarray) -> np.ndarray:
    return np.signbit(bf16_to_f32(bits)).astype(np.uint8)


def mantissa7(bits: np.ndarray) -> np.ndarray:
    """The 7 stored fraction bits of finite values, from the magnitude:
    normal |x| = (1 + m/128) 2^(e-127), subnormal |x| = (m/128) 2^-126.
    Non-finite values return -1 (their payload is not a magnitude)."""
    x = _to_f64(bits)
    out = np.full(x.shape, -1, np.int64)
    fin = np.isfinite(x)
    ax = np.abs(np.where(fin, x, 0.0))
    e = exponent_field(bits).astype(np.int64)
    normal = fin & (e > 0)
    sub = fin & (e == 0)
    out[normal] = np.rint((ax[normal] / np.exp2(e[normal] - 127.0) - 1.0)
                          * 128.0).astype(np.int64)
    out[sub] = np.rint(ax[sub] * 2.0 ** 133).astype(np.int64)
    return out


def all_bf16_patterns() -> np.ndarray:
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


# ---- binary16 (fp16) ----

def f16_values(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits).astype(np.uint16)
    return b.view(np.float16).astype(np.float64)


def exponent_field_f16(bits: np.ndarray) -> np.ndarray:
    """Biased 5-bit exponent from the value: 0 for zero and subnormals, 31
    for Inf/NaN, otherwise floor(log2|x|) + 15."""
    with np.errstate(invalid="ignore"):
        x = f16_values(bits)
    out = np.zeros(x.shape, np.int64)
    special = ~np.isfinite(x)
    out[special] = 31
    ax = np.abs(np.where(special, 0.0, x))
    normal = ax >= 2.0 ** -14
    _, ex = np.frexp(ax[normal])
    out[normal] = ex - 1 + 15
    return out.astype(np.uint8)


def mantissa10_f16(bits: np.ndarray) -> np.ndarray:
    """The 10 stored fraction bits of finite values, from the magnitude
    (normal: (1 + m/1024) 2^(e-15); subnormal: m 2^-24); -1 otherwise."""
    with np.errstate(invalid="ignore"):
        x = f16_values(bits)
    out = np.full(x.shape, -1, np.int64)
    fin = np.isfinite(x)
    ax = np.abs(np.where(fin, x, 0.0))
    e = exponent_field_f16(bits).astype(np.int64)
    normal = fin & (e > 0)
    sub = fin & (e == 0)
    out[normal] = np.rint((ax[normal] / 2.0 ** (e[normal] - 15) - 1.0) * 1024)
    out[sub] = np.rint(ax[sub] * 2.0 ** 24)
    return out


def sign_f16(bits: np.ndarray) -> np.ndarray:
    with np.errstate(invalid="ignore"):
        return np.signbit(f16_values(bits)).astype(np.uint8)

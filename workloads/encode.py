"""Storage encodings of drawn values.

Values are drawn in float64 and then stored either as IEEE binary32 or as
bfloat16 (1 sign, 8 exponent, 7 mantissa bits) rounded to nearest, ties to
even, directly from float64 (no double rounding through binary32). bfloat16
arrays are held as their raw uint16 bit patterns; widening them back to float64
is exact.
"""
import numpy as np

_F64_MANT = 52
_BF16_MANT = 7


def bf16_bits_from_f64(x):
    """Round float64 values to bfloat16 (RNE) and return the uint16 bit patterns.

    NaN stays NaN (quiet), +-Inf stays Inf, overflow past the largest finite
    bfloat16 becomes Inf, and values below the binary32 normal range go through
    a binary32 conversion first (they do not occur in the drawn workloads).
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    shift = _F64_MANT - _BF16_MANT                      # 45 dropped mantissa bits
    bits = x.view(np.uint64)
    lsb = (bits >> np.uint64(shift)) & np.uint64(1)
    rounded = (bits + (np.uint64(1) << np.uint64(shift - 1)) - np.uint64(1) + lsb)
    rounded &= ~((np.uint64(1) << np.uint64(shift)) - np.uint64(1))
    y = rounded.view(np.float64)
    with np.errstate(over="ignore"):
        y32 = y.astype(np.float32)                      # exact: <= 8 significant bits
    tiny = np.abs(x) < np.float64(2.0 ** -126)
    if tiny.any():                                      # binary32-subnormal range
        y32 = np.where(tiny, x.astype(np.float32), y32)
        t = y32.view(np.uint32)
        t_l = (t >> np.uint32(16)) & np.uint32(1)
        t = np.where(tiny, (t + np.uint32(0x7FFF) + t_l) & np.uint32(0xFFFF0000), t)
        y32 = t.astype(np.uint32).view(np.float32)
    out = (y32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out = np.where(nan, np.uint16(0x7FC0), out)
    return out.reshape(x.shape)


def f64_from_bf16_bits(b):
    """Widen bfloat16 bit patterns (uint16) to float64, exactly."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    with np.errstate(invalid="ignore"):
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def f32_from_f64(x):
    """Round float64 values to binary32 (RNE, numpy's conversion)."""
    return np.ascontiguousarray(x, dtype=np.float64).astype(np.float32)


def encode(x, dtype):
    """Encode float64 values in storage dtype 'bf16' (uint16 bits) or 'f32'."""
    if dtype == "bf16":
        return bf16_bits_from_f64(x)
    if dtype == "f32":
        return f32_from_f64(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def decode(raw, dtype):
    """Widen stored values (bf16 bits or binary32) to float64, exactly."""
    if dtype == "bf16":
        return f64_from_bf16_bits(raw)
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")

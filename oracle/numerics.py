"""Exact rounding of float64 values to the bf16 and fp16 formats.

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests, the smoke check and
the benchmark's CPU-baseline leg may import it; the product path never does.

Each function rounds the exact float64 input once, straight from the IEEE 754
definition of the target format (significand width, minimum normal exponent,
largest finite value).  Nothing goes through an intermediate float32 cast, so
there is no double rounding.
"""
from __future__ import annotations

import numpy as np

__all__ = ["round_to_format", "rne_bf16", "rne_fp16", "rd_fp16", "ru_fp16",
           "FP16_MAX", "BF16_MAX", "fp16_bits", "bf16_bits", "from_fp16_bits", "from_bf16_bits"]

# (significand bits including the implicit one, exponent of the smallest normal, largest finite)
_BF16 = (8, -126, float.fromhex("0x1.fep127"))
_FP16 = (11, -14, 65504.0)
BF16_MAX = _BF16[2]
FP16_MAX = _FP16[2]


def round_to_format(x, fmt, mode: str) -> np.ndarray:
    """Round float64 ``x`` to the binary format ``fmt``.

    mode: "rne" (nearest, ties to even), "down" (toward -inf), "up" (toward +inf).
    The unit in the last place of a normal value with frexp exponent e is
    2^(e - p); below the normal range it is fixed at 2^(emin - p + 1).  Scaling
    by a power of two is exact, so rint/floor/ceil see the exact quotient.
    """
    p, emin, vmax = fmt
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.maximum(e - p, emin - p + 1)
    y = np.ldexp(x, -q)
    if mode == "rne":
        r = np.rint(y)
    elif mode == "down":
        r = np.floor(y)
    elif mode == "up":
        r = np.ceil(y)
    else:
        raise ValueError(mode)
    out = np.ldexp(r, q)
    big = np.abs(out) > vmax
    if np.any(big):
        out = np.array(out, dtype=np.float64, copy=True)
        if mode == "rne":
            out[big] = np.copysign(np.inf, out[big])
        elif mode == "down":
            out[big] = np.where(out[big] > 0, vmax, -np.inf)
        else:
            out[big] = np.where(out[big] > 0, np.inf, -vmax)
    return out


def rne_bf16(x) -> np.ndarray:
    return round_to_format(x, _BF16, "rne")


def rne_fp16(x) -> np.ndarray:
    return round_to_format(x, _FP16, "rne")


def rd_fp16(x) -> np.ndarray:
    """Largest fp16 value <= x."""
    return round_to_format(x, _FP16, "down")


def ru_fp16(x) -> np.ndarray:
    """Smallest fp16 value >= x."""
    return round_to_format(x, _FP16, "up")


def fp16_bits(x) -> np.ndarray:
    """Bit patterns of float64 values that are exactly fp16-representable."""
    x = np.asarray(x, dtype=np.float64)
    h = x.astype(np.float16)
    if not np.array_equal(h.astype(np.float64), x, equal_nan=True):
        raise ValueError("value not representable in fp16")
    return h.view(np.uint16)


def from_fp16_bits(b) -> np.ndarray:
    return np.asarray(b, dtype=np.uint16).view(np.float16).astype(np.float64)


def bf16_bits(x) -> np.ndarray:
    """Bit patterns of float64 values that are exactly bf16-representable."""
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    if not np.array_equal(f.astype(np.float64), x, equal_nan=True):
        raise ValueError("value not representable in bf16")
    b = f.view(np.uint32)
    if np.any(b & 0xFFFF):
        raise ValueError("value not representable in bf16")
    return (b >> 16).astype(np.uint16)


def from_bf16_bits(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)

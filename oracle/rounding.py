"""Round-to-nearest-even into narrow binary floating-point formats (fp64 oracle).

The stored formats of the method use fp16 for the low-rank factors and the
quantiser scales (the paper's serialisation convention, section 9) and bf16
for the cache itself and the Gaussian sketch.  Rounding here is written from
the IEEE-754 definition: a value x = f * 2^e with 0.5 <= |f| < 1 is rounded to
a multiple of the quantum 2^(e - p), p = significand bits, where the quantum is
floored at the subnormal spacing; ties go to the even multiple.  Results above
the largest finite value become +-inf.
"""
from __future__ import annotations

import numpy as np

# (significand bits incl. hidden bit, log2 of subnormal spacing, largest finite)
FP16 = (11, -24, 65504.0)
BF16 = (8, -133, float.fromhex("0x1.fep127"))
FP32 = (24, -149, float.fromhex("0x1.fffffep127"))


def round_to(x, fmt) -> np.ndarray:
    """Round float64 values to the format ``fmt``; result returned as float64."""
    p, qmin, fmax = fmt
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.maximum(e - p, qmin)
    # ldexp by a power of two is exact; np.rint is round-half-to-even
    y = np.ldexp(np.rint(np.ldexp(x, -q)), q)
    y = np.where(np.abs(y) > fmax, np.copysign(np.inf, x), y)
    return np.where(np.isfinite(x), y, x)


def to_fp16(x) -> np.ndarray:
    return round_to(x, FP16)


def to_bf16(x) -> np.ndarray:
    return round_to(x, BF16)


def to_fp32(x) -> np.ndarray:
    return round_to(x, FP32)


def fp16_bits(x) -> np.ndarray:
    """IEEE binary16 bit patterns of values already representable in fp16."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def bf16_bits(x) -> np.ndarray:
    """bf16 bit patterns of values already representable in bf16."""
    v = np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32)
    return (v >> 16).astype(np.uint16)


def bf16_from_bits(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def ceil_log2(x: float) -> int:
    """ceil(log2(x)) for x > 0, exactly (via frexp, no logarithm)."""
    f, e = np.frexp(float(x))
    return int(e - 1) if f == 0.5 else int(e)

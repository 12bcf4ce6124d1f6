"""Rotated low-bit residual (fp64 oracle).

Section 4, "Rotated residual": the truncation residual R = X - X~ is rotated
by a random orthogonal matrix and quantised uniformly at b in {0, 2, 4, 8}
bits per entry (b = 0 stores nothing); decoding inverts the rotation.  Eq. (1)
prices it at b/8 bytes per entry "up to a negligible per-row scale term".

Readings adopted where the paper is silent:

* rotation = randomized Hadamard on the feature axis, r' = H_d (s * r) / sqrt(d)
  with H_d the Sylvester Hadamard matrix and s a seeded sign vector (one per
  cell); its inverse is r = s * (H_d r') / sqrt(d) because H_d is symmetric
  and H_d H_d = d I;
* quantiser = symmetric, scale-only, mid-rise, over contiguous groups of g
  rotated-row entries: a = max |r'|, Delta = fp16(2 a / (2^b - 1)) (clamped to
  the largest finite fp16), code = clip(rint(r'/Delta + (2^b-1)/2), 0, 2^b-1)
  with rint = round half to even; Delta = 0 gives code 2^(b-1) everywhere;
  dequantised value (code - (2^b-1)/2) * Delta;
* codes are packed LSB-first, 8/b codes per byte, in flattened (slice, token,
  feature) order; one fp16 scale per group in the same order.
"""
from __future__ import annotations

import numpy as np

from .rounding import to_fp16

FP16_MAX = 65504.0


def sylvester_hadamard(d: int) -> np.ndarray:
    """H_1 = [1], H_2k = [[H_k, H_k], [H_k, -H_k]]."""
    if d < 1 or d & (d - 1):
        raise ValueError("d must be a power of two")
    H = np.ones((1, 1))
    while H.shape[0] < d:
        H = np.block([[H, H], [H, -H]])
    return H


def rotate(r: np.ndarray, signs: np.ndarray) -> np.ndarray:
    """r' = H_d (s * r) / sqrt(d) applied to every feature row (last axis)."""
    d = r.shape[-1]
    H = sylvester_hadamard(d)
    return ((r * signs) @ H.T) / np.sqrt(d)


def unrotate(rp: np.ndarray, signs: np.ndarray) -> np.ndarray:
    """Inverse rotation: r = s * (H_d r') / sqrt(d)."""
    d = rp.shape[-1]
    H = sylvester_hadamard(d)
    return signs * ((rp @ H.T) / np.sqrt(d))


def quantize(rp: np.ndarray, bits: int, group: int):
    """Quantise rotated rows; returns (codes uint8 with rp's shape, scales fp64).

    ``scales`` has shape rp.shape[:-1] + (d // group,) and holds fp16-exact values.
    """
    if bits not in (2, 4, 8):
        raise ValueError("bits must be 2, 4 or 8 (b = 0 stores no residual)")
    d = rp.shape[-1]
    if group < 1 or d % group:
        raise ValueError("group must divide d")
    levels = (1 << bits) - 1
    g = rp.reshape(rp.shape[:-1] + (d // group, group))
    a = np.max(np.abs(g), axis=-1)
    delta = to_fp16(np.minimum(2.0 * a / levels, FP16_MAX))
    with np.errstate(divide="ignore", invalid="ignore"):
        code = np.rint(g / delta[..., None] + levels / 2.0)
    code = np.clip(code, 0, levels)
    code = np.where(delta[..., None] == 0.0, float(1 << (bits - 1)), code)
    return code.reshape(rp.shape).astype(np.uint8), delta


def dequantize(codes: np.ndarray, scales: np.ndarray, bits: int, group: int) -> np.ndarray:
    levels = (1 << bits) - 1
    d = codes.shape[-1]
    c = codes.reshape(codes.shape[:-1] + (d // group, group)).astype(np.float64)
    return ((c - levels / 2.0) * scales[..., None]).reshape(codes.shape)


def pack(codes: np.ndarray, bits: int) -> np.ndarray:
    """Pack codes (flattened C order) LSB-first into bytes."""
    flat = codes.reshape(-1).astype(np.uint8)
    per = 8 // bits
    if flat.size % per:
        raise ValueError("number of codes must fill whole bytes")
    flat = flat.reshape(-1, per).astype(np.uint16)
    out = np.zeros(flat.shape[0], dtype=np.uint16)
    for k in range(per):
        out |= flat[:, k] << (bits * k)
    return out.astype(np.uint8)


def unpack(packed: np.ndarray, bits: int, n: int) -> np.ndarray:
    per = 8 // bits
    p = np.asarray(packed, dtype=np.uint8).reshape(-1, 1).astype(np.uint16)
    shifts = (bits * np.arange(per, dtype=np.uint16))[None, :]
    codes = (p >> shifts) & ((1 << bits) - 1)
    return codes.reshape(-1)[:n].astype(np.uint8)


def residual_roundtrip(r: np.ndarray, signs: np.ndarray, bits: int, group: int) -> np.ndarray:
    """Rotate, quantise, dequantise and unrotate r (b = 0 returns zeros)."""
    if bits == 0:
        return np.zeros_like(r)
    codes, scales = quantize(rotate(r, signs), bits, group)
    return unrotate(dequantize(codes, scales, bits, group), signs)

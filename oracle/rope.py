"""Rotary position embedding re-applied at decode time (fp64 oracle; test infrastructure).

Appendix B: keys are compressed before RoPE, and the rotation is re-applied when the
cache is decoded.  RoPE (Su et al. 2021) rotates feature pairs of a token row by
position-dependent angles; with the half-split pairing of the Mistral / LLaMA
checkpoints, pair j < d/2 is (j, j + d/2) and token position p turns it by
p * base^(-2 j / d):

    x'_j       = x_j cos(p w_j) - x_{j+d/2} sin(p w_j)
    x'_{j+d/2} = x_{j+d/2} cos(p w_j) + x_j sin(p w_j),   w_j = base^(-2 j / d).
"""
from __future__ import annotations

import numpy as np


def rope(X: np.ndarray, base: float, positions) -> np.ndarray:
    """Rotate the last axis (d features) of every token row; the token axis is -2 and
    ``positions`` gives one position per token (array of length T)."""
    d = X.shape[-1]
    if d % 2:
        raise ValueError("d must be even")
    h = d // 2
    w = base ** (-2.0 * np.arange(h, dtype=np.float64) / d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * w[None, :]     # T x d/2
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = X[..., :h], X[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)

"""Decode-time attention over a decompressed cache (fp64 oracle; test infrastructure).

Section 8 and the conclusion name the deployable decode path: attention evaluated on the
compressed factors, without materialising the cache.  Whatever route a kernel takes, the
result it must reproduce is plain softmax attention of the new queries over the cache that
decompression would produce; this module is that definition.

Grouped-query layout (Mistral / LLaMA convention): with H key-value heads per layer and
n_q query heads, n_q a multiple of H, query head j reads key-value head j // (n_q / H).
For layer l of a cell, key-value head h is slice s = l * H + h.

    o_j = sum_t softmax_t(scale * q_j . K[s][t]) V[s][t]
"""
from __future__ import annotations

import numpy as np


def softmax(x: np.ndarray) -> np.ndarray:
    z = np.exp(x - np.max(x))
    return z / z.sum()


def attend(K: np.ndarray, V: np.ndarray, layer: int, n_heads: int, Q: np.ndarray,
           scale: float) -> np.ndarray:
    """K, V: decoded cells [m][T][d]; Q: [n_q][d]; returns [n_q][d] (fp64)."""
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    n_q = Q.shape[0]
    if n_q % n_heads:
        raise ValueError("n_q must be a multiple of the key-value heads")
    rep = n_q // n_heads
    out = np.zeros_like(Q)
    for j in range(n_q):
        s = layer * n_heads + j // rep
        p = softmax(scale * (K[s] @ Q[j]))
        out[j] = p @ V[s]
    return out

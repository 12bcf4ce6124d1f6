"""Counter-based random numbers for the method's seeded draws (fp64 oracle).

The method draws two kinds of random numbers: the sign vector of the random
orthogonal rotation of the residual (section 4, "Rotated residual") and the
Gaussian test matrix of FlashJoLT's randomized SVD (section 5).  Both sides of
the parity check (this oracle and the GPU library) implement the same
published counter-based generator, Philox4x32-10 (Salmon, Moraes, Dror and
Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011), so that a draw
is a pure function of (seed, counter) and needs no shared state.

Conventions (the generator is the published one; the counter layout is this
library's):

* key = (seed mod 2^32, seed div 2^32);
* counter = (i, j, 0, stream) with ``stream`` 1 = rotation signs,
  2 = sketch matrix, 3 = calibration samples;
* uniform from a 32-bit word w: u = (w + 1/2) * 2^-32, in (0, 1);
* Gaussian (Box-Muller, cosine branch) in float64 from words (w0, w1):
  z = sqrt(-2 ln u0) * cos(2 pi u1);
* rotation sign for feature j: +1 if bit 0 of word 0 of philox((j,0,0,1)) is
  0, else -1;
* sketch entry Omega[c, j]: bf16(z(philox((c, j, 0, 2)))) (round to nearest
  even), c indexing columns of the token unfolding and j sketch columns;
* calibration sample k: fp32(z(philox((k, 0, 0, 3)))).
"""
from __future__ import annotations

import numpy as np

from .rounding import to_bf16, to_fp32

M0, M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK = np.uint64(0xFFFFFFFF)

STREAM_SIGN, STREAM_SKETCH, STREAM_CALIB = 1, 2, 3


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Ten Philox-4x32 rounds; arrays of uint32 counters -> four uint32 arrays."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & MASK for c in (c0, c1, c2, c3))
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    k0, k1 = int(k0) & 0xFFFFFFFF, int(k1) & 0xFFFFFFFF
    for r in range(10):
        key0 = np.uint64((k0 + r * W0) & 0xFFFFFFFF)
        key1 = np.uint64((k1 + r * W1) & 0xFFFFFFFF)
        p0 = M0 * c0                 # < 2^64: exact in uint64
        p1 = M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK
        c0, c1, c2, c3 = (hi1 ^ c1 ^ key0), lo1, (hi0 ^ c3 ^ key1), lo0
    return tuple(x.astype(np.uint32) for x in (c0, c1, c2, c3))


def _key(seed: int):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & 0xFFFFFFFF, seed >> 32


def uniform(w) -> np.ndarray:
    return (np.asarray(w, dtype=np.float64) + 0.5) * 2.0 ** -32


def box_muller(w0, w1) -> np.ndarray:
    u0, u1 = uniform(w0), uniform(w1)
    return np.sqrt(-2.0 * np.log(u0)) * np.cos((2.0 * np.pi) * u1)


def rotation_signs(seed: int, d: int) -> np.ndarray:
    """Sign vector s in {+1, -1}^d of the randomized Hadamard rotation."""
    j = np.arange(d, dtype=np.uint64)
    w0, _, _, _ = philox4x32_10(j, 0, 0, STREAM_SIGN, *_key(seed))
    return np.where((w0 & 1) == 0, 1.0, -1.0)


def sketch_matrix(seed: int, n_rows: int, n_cols: int) -> np.ndarray:
    """Gaussian test matrix Omega (n_rows x n_cols), entries rounded to bf16."""
    c = np.arange(n_rows, dtype=np.uint64)[:, None]
    j = np.arange(n_cols, dtype=np.uint64)[None, :]
    w0, w1, _, _ = philox4x32_10(c, j, 0, STREAM_SKETCH, *_key(seed))
    return to_bf16(box_muller(w0, w1))


def calibration_samples(seed: int, n: int) -> np.ndarray:
    """n standard-normal samples rounded to fp32 (the epsilon^2 calibration input)."""
    k = np.arange(n, dtype=np.uint64)
    w0, w1, _, _ = philox4x32_10(k, 0, 0, STREAM_CALIB, *_key(seed))
    return to_fp32(box_muller(w0, w1))

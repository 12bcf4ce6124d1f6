"""Three-mode spectral diagnostics of a cache tensor (fp64 oracle; test infrastructure).

Section 3 (spectral motivation) and appendix A: the cache of one layer (or of a cell of
several layers) is a third-order tensor X[s][t][f] (s = slice: head, or layer x head;
t = token; f = feature).  Each of its three unfoldings has singular values sigma_1 >= ...;
the appendix tabulates, per mode, the dynamic range sigma_1 / sigma_min and the smallest
ranks r whose truncation error is at most 10% and at most 20%.

Reading (the paper gives no formula): the error of keeping the top r singular values of a
mode is the relative Frobenius error sqrt(sum_{i>r} sigma_i^2 / sum_i sigma_i^2), the
metric the paper reports everywhere else.  The appendix's head rows (8/8 at both
thresholds for eight heads of similar energy) agree with this reading and not with a
threshold on the discarded energy fraction itself.  sigma_min is the smallest of the n
singular values of the n-row unfolding (0 when the unfolding is rank deficient, which
makes the range infinite).
"""
from __future__ import annotations

import numpy as np

MODES = ("slices", "tokens", "features")


def unfold(X: np.ndarray, mode: int) -> np.ndarray:
    """Mode unfolding of X[s][t][f]: rows are the given mode's index (0 = slices,
    1 = tokens, 2 = features), columns the other two in their natural order."""
    X = np.asarray(X, dtype=np.float64)
    return np.moveaxis(X, mode, 0).reshape(X.shape[mode], -1)


def mode_spectrum(X: np.ndarray, mode: int) -> np.ndarray:
    """Squared singular values of the mode unfolding (eigenvalues of its Gram), all n of
    them, descending, clipped at zero."""
    A = unfold(X, mode)
    lam = np.linalg.eigvalsh(A @ A.T)[::-1]
    return np.maximum(lam, 0.0)


def truncation_error(lam: np.ndarray, r: int) -> float:
    """Relative Frobenius error of keeping the top r of the squared singular values lam."""
    lam = np.asarray(lam, dtype=np.float64)
    total = lam.sum()
    if total <= 0.0:
        return 0.0
    return float(np.sqrt(lam[r:].sum() / total))


def rank_for_error(lam: np.ndarray, err: float) -> int:
    """Smallest r in 0..n with truncation_error(lam, r) <= err."""
    for r in range(len(lam) + 1):
        if truncation_error(lam, r) <= err:
            return r
    return len(lam)


def sigma_range(lam: np.ndarray) -> float:
    """sigma_1 / sigma_min (infinite when sigma_min is zero)."""
    lam = np.asarray(lam, dtype=np.float64)
    if lam[-1] <= 0.0:
        return float("inf")
    return float(np.sqrt(lam[0] / lam[-1]))


def mode_summary(lam: np.ndarray, errs=(0.10, 0.20)) -> dict:
    """One appendix-A row: n, sigma_1 / sigma_min and the ranks at each error threshold."""
    return {"n": int(len(lam)), "sigma_range": sigma_range(lam),
            "ranks": [rank_for_error(lam, e) for e in errs]}


def three_mode_table(X: np.ndarray, errs=(0.10, 0.20)) -> dict:
    """Appendix-A rows for the three modes of X[s][t][f]."""
    return {MODES[k]: mode_summary(mode_spectrum(X, k), errs) for k in range(3)}

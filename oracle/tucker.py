"""Partial Tucker backbone of one cell (fp64 oracle).

A cell is X in R^{m x T x d}: the m = |g| * n_h (layer, head) slices of one
layer group's keys or values (section 4; eq. (1) defines m).  The head and
layer modes keep identity factors, so the cell is treated as m slices X_s of
size T x d and only the token mode (T) and feature mode (d) are truncated.

* token unfolding X_(2) in R^{T x N}, N = m d, column s*d + f holds X[s, :, f];
* exact token spectrum: eigen-decomposition of C = X_(2) X_(2)^T
  (section 4, "Partial Tucker backbone"; section 3 takes mode spectra of the
  unfoldings);
* FlashJoLT token spectrum: randomized SVD (Halko et al. 2011) of X_(2) that
  keeps the top q directions, with the discarded energy appended as one
  synthetic eigenvalue ("tail-mass accounting", section 5);
* feature spectrum: eigen-decomposition of F = sum_s X_s^T X_s, kept exact in
  both variants (section 5);
* ST-HOSVD (Vannieuwenhoven et al. 2012, cited in section 4): truncate the
  token mode first with U_T, then take the feature factor from the projected
  tensor Y = X x_2 U_T^T, core G = Y x_3 U_d^T;
* truncated feature spectra: the eigenvalues of Y's feature Gram at every grid
  token rank, from which the exact discarded mass of every (r_T, r_d) follows;
* serialisation: fp16 factors (c = 2 bytes per scalar, section 9) with one
  power-of-two exponent per core slice, or fp32 factors (c = 4);
* reconstruction X~_s = U^_T G^_s U^_d^T from the *stored* factors.
"""
from __future__ import annotations

import numpy as np

from .philox import sketch_matrix
from .rounding import to_fp16, to_fp32, ceil_log2


def unfold_tokens(X: np.ndarray) -> np.ndarray:
    """X (m, T, d) -> X_(2) (T, m*d), column s*d + f = X[s, :, f]."""
    m, T, d = X.shape
    return X.transpose(1, 0, 2).reshape(T, m * d)


def energy(X: np.ndarray) -> float:
    return float(np.sum(X * X))


def _eigh_desc(A: np.ndarray):
    w, V = np.linalg.eigh(A)
    order = np.argsort(w)[::-1]
    return w[order], V[:, order]


def token_spectrum_exact(X: np.ndarray):
    """All T eigenvalues of C = X_(2) X_(2)^T (descending, clipped at 0) and eigenvectors."""
    X2 = unfold_tokens(X)
    lam, U = _eigh_desc(X2 @ X2.T)
    return np.maximum(lam, 0.0), U


def feature_spectrum(X: np.ndarray):
    """All d eigenvalues of F = sum_s X_s^T X_s (descending, clipped at 0) and eigenvectors."""
    m, T, d = X.shape
    Xf = X.reshape(m * T, d)
    mu, V = _eigh_desc(Xf.T @ Xf)
    return np.maximum(mu, 0.0), V


def _orth(A: np.ndarray) -> np.ndarray:
    q, _ = np.linalg.qr(A, mode="reduced")
    return q


def sketch_width(q: int, p: int, T: int, N: int) -> int:
    """l = min(q + p, T, N)."""
    return int(min(q + p, T, N))


def token_spectrum_flash(X: np.ndarray, *, q: int, p: int, power_iters: int, seed: int,
                         omega: np.ndarray | None = None):
    """FlashJoLT randomized token spectrum with tail-mass accounting (section 5).

    Returns (lam, U_T, extras): lam has q_eff + 1 entries, the last being the
    synthetic tail E - sum(captured), and U_T is T x q_eff.
    """
    m, T, d = X.shape
    N = m * d
    X2 = unfold_tokens(X)
    ell = sketch_width(q, p, T, N)
    q_eff = min(q, ell)
    if omega is None:
        omega = sketch_matrix(seed, N, ell)
    Q = _orth(X2 @ omega)                       # range finder
    for _ in range(power_iters):                # power (subspace) iteration
        Qp = _orth(X2.T @ Q)
        Q = _orth(X2 @ Qp)
    B = Q.T @ X2                                # ell x N
    Lam, W = _eigh_desc(B @ B.T)
    Lam = np.maximum(Lam, 0.0)
    U = Q @ W[:, :q_eff]
    captured = Lam[:q_eff]
    E = energy(X)
    tail = max(E - float(np.sum(captured)), 0.0)
    lam = np.concatenate([captured, [tail]])
    return lam, U, dict(Q=Q, B=B, W=W, Lam=Lam, ell=ell, q_eff=q_eff, omega=omega)


def tail_fractions(lam: np.ndarray, E: float) -> np.ndarray:
    """tau[r] = (sum of lam[i] for i >= r) / E for r = 0..len(lam).

    The suffix sums are accumulated one term at a time from the smallest
    index upward (i = n-1 down to 0) so that the tail is summed directly
    rather than formed as E minus a head sum.  E = 0 gives tau = 0.
    """
    n = len(lam)
    suf = np.zeros(n + 1)
    acc = 0.0
    for i in range(n - 1, -1, -1):
        acc += float(lam[i])
        suf[i] = acc
    if E <= 0.0:
        return np.zeros(n + 1)
    return suf / E


def truncated_feature_spectra(X: np.ndarray, U_T: np.ndarray, r_list) -> np.ndarray:
    """Feature spectra of the token-truncated cell, one row per token rank.

    The token-first ST-HOSVD (section 4) takes its feature factor from the
    projected cell Y = X x_2 U_r^T, U_r = the first r columns of U_T, i.e. from
    F_Y(r) = sum_s Y_s^T Y_s = sum_s X_s^T U_r U_r^T X_s.  Row k of the result
    holds the d eigenvalues of F_Y(r_list[k]), descending, clipped at 0.  With
    orthonormal U_r and U_d the truncation keeps ||G||^2 = the sum of the top
    r_d of them, so these rows give the exact discarded mass at every (r, r_d).
    """
    m, T, d = X.shape
    out = np.zeros((len(r_list), d))
    for k, r in enumerate(r_list):
        U = U_T[:, :r]
        F = np.zeros((d, d))
        for s in range(m):
            Ys = U.T @ X[s]                     # r x d
            F += Ys.T @ Ys
        mu, _ = _eigh_desc(F)
        out[k] = np.maximum(mu, 0.0)
    return out


def st_hosvd(X: np.ndarray, U_T: np.ndarray, r_T: int, r_d: int):
    """Token-first ST-HOSVD at (r_T, r_d); returns (U, U_d, G, mu_Y)."""
    m, T, d = X.shape
    if (r_T == 0) != (r_d == 0):
        raise ValueError("r_T = 0 if and only if r_d = 0")
    if r_T == 0:
        return np.zeros((T, 0)), np.zeros((d, 0)), np.zeros((m, 0, 0)), np.zeros(d)
    U = U_T[:, :r_T]
    Y = np.stack([U.T @ X[s] for s in range(m)])         # Y_s = U^T X_s  (r_T x d)
    Yf = Y.reshape(m * r_T, d)
    mu_Y, V = _eigh_desc(Yf.T @ Yf)             # feature spectrum of Y
    U_d = V[:, :r_d]
    G = np.stack([Y[s] @ U_d for s in range(m)])         # G_s = Y_s U_d  (r_T x r_d)
    return U, U_d, G, mu_Y


def serialize(U: np.ndarray, U_d: np.ndarray, G: np.ndarray, factor_bytes: int):
    """Round factors to the stored precision; fp16 cores get one exponent per slice.

    Returns (U_hat, Ud_hat, G_hat, gexp) with G_s = G_hat_s * 2^gexp[s] up to rounding.
    The exponent is e_s = max(-128, ceil(log2 max|G_s|) - 15) (0 for an all-zero slice):
    the blob keeps it in one signed byte, and the floor only matters for cores below
    2^-113, whose scaled values then stay below 2^15 as well.
    """
    m = G.shape[0]
    gexp = np.zeros(m, dtype=np.int64)
    if factor_bytes == 4:
        return to_fp32(U), to_fp32(U_d), to_fp32(G), gexp
    if factor_bytes != 2:
        raise ValueError("factor_bytes must be 2 (fp16) or 4 (fp32)")
    G_hat = np.empty_like(G)
    for s in range(m):
        M = float(np.max(np.abs(G[s]))) if G[s].size else 0.0
        e = max(-128, ceil_log2(M) - 15) if M > 0.0 else 0
        gexp[s] = e
        G_hat[s] = to_fp16(np.ldexp(G[s], -e))
    return to_fp16(U), to_fp16(U_d), G_hat, gexp


def reconstruct(U_hat: np.ndarray, Ud_hat: np.ndarray, G_hat: np.ndarray,
                gexp: np.ndarray, T: int, d: int) -> np.ndarray:
    """X~_s = U_hat (2^gexp[s] G_hat_s) Ud_hat^T for every slice, in fp64."""
    m = G_hat.shape[0]
    if U_hat.shape[1] == 0:
        return np.zeros((m, T, d))
    G = np.ldexp(G_hat, gexp[:, None, None])
    W = [G[s] @ Ud_hat.T for s in range(m)]              # W_s = G_s U_d^T  (r_T x d)
    return np.stack([U_hat @ W[s] for s in range(m)])    # X~_s = U_T W_s  (T x d)

"""Pins of the oracle's partial Tucker backbone (section 4) and FlashJoLT (section 5).

The pins are closed forms and textbook reductions: exactness at full rank,
the ST-HOSVD error bounds by discarded mode energy, Pythagoras for orthogonal
projections, Eckart-Young for a single slice, brute force against SVDs of the
unfoldings, exactness of the randomized range finder when the sketch covers
the whole range, and tail-mass conservation.
"""
import numpy as np
import pytest

from conftest import lowrank_cell
from oracle import tucker as tk
from oracle.rounding import to_fp16


def _unrounded_xtilde(X, U_T, r_T, r_d):
    U, U_d, G, _ = tk.st_hosvd(X, U_T, r_T, r_d)
    return np.einsum("tr,srk,dk->std", U, G, U_d), U, U_d, G


def test_unfolding_layout():
    X = np.arange(2 * 3 * 4, dtype=float).reshape(2, 3, 4)
    X2 = tk.unfold_tokens(X)
    assert X2.shape == (3, 8)
    for s in range(2):
        for t in range(3):
            for f in range(4):
                assert X2[t, s * 4 + f] == X[s, t, f]


def test_full_rank_is_exact(rng):                                     # P1
    X = rng.standard_normal((3, 20, 16))
    lam, U_T = tk.token_spectrum_exact(X)
    Xt, *_ = _unrounded_xtilde(X, U_T, 20, 16)
    np.testing.assert_allclose(Xt, X, atol=1e-12 * np.abs(X).max())


@pytest.mark.parametrize("rT,rd", [(4, 3), (10, 8), (1, 16), (20, 1), (7, 7)])
def test_sthosvd_error_bounds(rng, rT, rd):                           # P2, P3
    X = lowrank_cell(rng, 3, 20, 16, 6, noise=0.3)
    E = tk.energy(X)
    lam, U_T = tk.token_spectrum_exact(X)
    mu, _ = tk.feature_spectrum(X)
    tauT = tk.tail_fractions(lam, E)[rT]
    taud = tk.tail_fractions(mu, E)[rd]
    Xt, U, U_d, G = _unrounded_xtilde(X, U_T, rT, rd)
    err2 = np.sum((X - Xt) ** 2)
    assert max(tauT, taud) * E <= err2 * (1 + 1e-10)
    assert err2 <= (tauT + taud) * E * (1 + 1e-10)
    np.testing.assert_allclose(err2, E - np.sum(G * G), rtol=1e-9)     # Pythagoras


def test_single_slice_is_eckart_young(rng):                           # P4
    X = rng.standard_normal((1, 30, 12)) @ np.diag(np.linspace(3, 0.1, 12))
    sv = np.linalg.svd(X[0], compute_uv=False)
    lam, U_T = tk.token_spectrum_exact(X)
    np.testing.assert_allclose(lam[:12], sv ** 2, rtol=1e-10)
    for r in (1, 3, 7):
        Xt, *_ = _unrounded_xtilde(X, U_T, r, 12)
        np.testing.assert_allclose(np.sum((X - Xt) ** 2), np.sum(sv[r:] ** 2), rtol=1e-9)


def test_brute_force_against_unfolding_svds(rng):                     # P5
    for trial in range(20):
        m, T, d = rng.integers(1, 4), rng.integers(3, 9), rng.integers(3, 9)
        X = rng.standard_normal((m, T, d)) * np.exp(rng.uniform(-1, 1, (1, 1, d)))
        rT = int(rng.integers(1, min(T, m * d) + 1))
        rd = int(rng.integers(1, min(d, m * rT) + 1))
        # literal ST-HOSVD from numpy SVDs of the mode unfoldings
        Uy, sy, _ = np.linalg.svd(X.transpose(1, 0, 2).reshape(T, m * d), full_matrices=False)
        sy_full = np.zeros(T); sy_full[:len(sy)] = sy
        gap_ok = rT >= min(T, m * d) or sy_full[rT - 1] - sy_full[rT] > 1e-6 * sy_full[0]
        U1 = Uy[:, :rT]
        Y = np.einsum("std,tr->srd", X, U1)
        Uf, sf, _ = np.linalg.svd(Y.transpose(2, 0, 1).reshape(d, -1), full_matrices=False)
        sf_full = np.zeros(d); sf_full[:len(sf)] = sf
        gap_ok &= rd >= min(d, m * rT) or sf_full[rd - 1] - sf_full[rd] > 1e-6 * sf_full[0]
        if not gap_ok:
            continue
        U2 = Uf[:, :rd]
        ref = np.einsum("tr,srk,dk->std", U1, np.einsum("srd,dk->srk", Y, U2), U2)
        lam, U_T = tk.token_spectrum_exact(X)
        np.testing.assert_allclose(lam[:len(sy)], sy ** 2, rtol=1e-9, atol=1e-12)
        Xt, U, U_d, _ = _unrounded_xtilde(X, U_T, rT, rd)
        np.testing.assert_allclose(U @ U.T, U1 @ U1.T, atol=1e-9)   # projectors, not factors
        np.testing.assert_allclose(U_d @ U_d.T, U2 @ U2.T, atol=1e-9)
        np.testing.assert_allclose(Xt, ref, atol=1e-9 * np.abs(X).max())


def test_factors_orthonormal(rng):                                    # P14
    X = lowrank_cell(rng, 4, 40, 16, 5, noise=0.1)
    lam, U_T = tk.token_spectrum_exact(X)
    _, U, U_d, _ = _unrounded_xtilde(X, U_T, 12, 9)
    np.testing.assert_allclose(U.T @ U, np.eye(12), atol=1e-12)
    np.testing.assert_allclose(U_d.T @ U_d, np.eye(9), atol=1e-12)


def test_exact_spectrum_sums_to_energy(rng):
    X = rng.standard_normal((3, 30, 8))
    lam, _ = tk.token_spectrum_exact(X)
    mu, _ = tk.feature_spectrum(X)
    E = tk.energy(X)
    np.testing.assert_allclose(lam.sum(), E, rtol=1e-12)
    np.testing.assert_allclose(mu.sum(), E, rtol=1e-12)
    tau = tk.tail_fractions(lam, E)
    assert tau[-1] == 0.0 and abs(tau[0] - 1) < 1e-12
    assert (np.diff(tau) <= 1e-15).all()


def test_flash_exact_when_sketch_covers_range(rng):                   # P12, P13
    X = lowrank_cell(rng, 4, 60, 16, 5, noise=0.0)     # rank(X_(2)) <= 5 * ... <= l
    E = tk.energy(X)
    lam_e, U_e = tk.token_spectrum_exact(X)
    rank = int(np.sum(lam_e > 1e-10 * lam_e[0]))
    q = rank + 2
    lam_f, U_f, ex = tk.token_spectrum_flash(X, q=q, p=10, power_iters=1, seed=5)
    assert ex["ell"] >= rank
    np.testing.assert_allclose(lam_f[:rank], lam_e[:rank], rtol=1e-9)
    np.testing.assert_allclose(lam_f[:-1].sum() + lam_f[-1], E, rtol=1e-12)   # tail mass
    assert lam_f[-1] <= 1e-9 * E
    P_e, P_f = U_e[:, :rank] @ U_e[:, :rank].T, U_f[:, :rank] @ U_f[:, :rank].T
    np.testing.assert_allclose(P_f, P_e, atol=1e-8)


def test_flash_tail_mass_is_uncaptured_energy(rng):                   # P13
    X = lowrank_cell(rng, 3, 80, 16, 6, noise=0.5)
    E = tk.energy(X)
    q = 10
    lam_f, U_f, _ = tk.token_spectrum_flash(X, q=q, p=5, power_iters=1, seed=1)
    assert len(lam_f) == q + 1
    proj = np.einsum("std,tr->srd", X, U_f)
    captured = np.sum(proj ** 2)
    np.testing.assert_allclose(lam_f[:q].sum(), captured, rtol=1e-10)
    np.testing.assert_allclose(lam_f[q], E - captured, rtol=1e-9)


def test_flash_converges_to_exact_with_many_power_iterations(rng):    # P12
    X = lowrank_cell(rng, 3, 50, 16, 8, noise=0.05, decay=0.5)
    lam_e, U_e = tk.token_spectrum_exact(X)
    lam_f, U_f, _ = tk.token_spectrum_flash(X, q=6, p=4, power_iters=25, seed=2)
    np.testing.assert_allclose(lam_f[:6], lam_e[:6], rtol=1e-8)
    np.testing.assert_allclose(U_f @ U_f.T, U_e[:, :6] @ U_e[:, :6].T, atol=1e-7)


def test_serialize_fp16_exponents(rng):
    G = rng.standard_normal((4, 5, 3)) * np.array([1e-7, 1.0, 7e4, 3e9])[:, None, None]
    U = rng.standard_normal((10, 5)) / 3
    Ud = rng.standard_normal((6, 3)) / 3
    Uh, Udh, Gh, e = tk.serialize(U, Ud, G, 2)
    np.testing.assert_array_equal(Uh, to_fp16(U))
    for s in range(4):
        mx = np.abs(Gh[s]).max()
        assert 2.0 ** 14 < mx <= 2.0 ** 15
        np.testing.assert_allclose(np.ldexp(Gh[s], e[s]), G[s], rtol=2 ** -11)
    Xt = tk.reconstruct(Uh, Udh, Gh, e, 10, 6)
    ref = np.einsum("tr,srk,dk->std", Uh, np.ldexp(Gh, e[:, None, None]), Udh)
    np.testing.assert_allclose(Xt, ref, rtol=1e-12)


def test_core_exponent_fits_a_signed_byte():
    """The blob keeps one int8 exponent per core slice: e_s = max(-128, ceil(log2 max|G_s|) - 15).
    Ordinary cores get the unclamped value (stored maxima in (2^14, 2^15]); cores below 2^-113
    take the floor -128 and still scale to below 2^15; an all-zero slice stores 0."""
    from oracle.rounding import to_fp16
    rng = np.random.default_rng(3)
    G = rng.standard_normal((4, 6, 5))
    G[1] *= 2.0 ** -120          # below the range the byte can express unclamped
    G[2] *= 2.0 ** 100
    G[3] = 0.0
    U = np.linalg.qr(rng.standard_normal((9, 6)))[0]
    Ud = np.linalg.qr(rng.standard_normal((5, 5)))[0]
    _, _, G_hat, gexp = tk.serialize(U, Ud, G, factor_bytes=2)
    assert gexp.min() >= -128 and gexp.max() <= 127
    assert gexp[1] == -128 and gexp[3] == 0
    for s in (0, 2):
        M = np.abs(G[s]).max()
        assert 2.0 ** 14 < M * 2.0 ** -gexp[s] <= 2.0 ** 15
    assert np.abs(G_hat[1]).max() < 2.0 ** 15
    # stored values are the fp16 rounding of the scaled core (exact powers of two)
    for s in range(4):
        np.testing.assert_array_equal(G_hat[s], to_fp16(np.ldexp(G[s], -int(gexp[s]))))
    # the scaled-back core of the clamped slice keeps fp16 relative accuracy
    back = np.ldexp(G_hat[1], int(gexp[1]))
    assert np.abs(back - G[1]).max() <= 2.0 ** -11 * np.abs(G[1]).max()

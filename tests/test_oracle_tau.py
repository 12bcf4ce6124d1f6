"""Pins of the exact ST-HOSVD truncation error (section 4, eq. (2)'s tau) and of the
allocator run on it.

tau(r_T, r_d) is the relative Frobenius mass that the token-first ST-HOSVD truncation
discards.  The oracle forms it from the feature spectra of the token-truncated cell,
mu_k = eig(sum_s X_s^T U_r U_r^T X_s), as (E - sum_{i < r_d} mu_k[i]) / E.  These tests
tie that to quantities fixed independently of it: the error of the explicit
reconstruction, a closed form for a separable cell, the one-mode special cases and the
two-sided mode-tail bounds of the sequentially truncated HOSVD.
"""
import itertools

import numpy as np
import pytest

from conftest import lowrank_cell
from oracle import alloc, pipeline, tucker as tk

EPS2 = {0: 1.0, 2: 0.26, 4: 0.0101, 8: 3.5e-5}


def _tau_table(X, U_T, step):
    E = tk.energy(X)
    T = X.shape[1]
    rs = list(range(step, T + 1, step))
    mu = tk.truncated_feature_spectra(X, U_T, rs)
    return rs, mu, alloc.st_tau_table(E, mu), E


def _explicit_error(X, U_T, rT, rd):
    """||X - X~||^2 of the truncation, by projecting every slice in both modes."""
    U = U_T[:, :rT]
    Y = np.einsum("tr,std->srd", U, X)
    F = sum(Y[s].T @ Y[s] for s in range(X.shape[0]))
    w, V = np.linalg.eigh(F)
    Vd = V[:, np.argsort(w)[::-1][:rd]]
    Xt = np.einsum("tr,srd,ed->ste", U, Y @ Vd, Vd)
    return float(np.sum((X - Xt) ** 2))


def test_tau_equals_the_explicit_reconstruction_error(rng):
    X = lowrank_cell(rng, 3, 20, 8, 5, noise=0.05)
    _, U_T = tk.token_spectrum_exact(X)
    rs, mu, tab, E = _tau_table(X, U_T, 2)
    for k, rT in enumerate(rs):
        for rd in range(1, 9):
            assert tab[k][rd] == pytest.approx(_explicit_error(X, U_T, rT, rd) / E, abs=1e-12)


def test_separable_cell_closed_form(rng):
    """X_s = w_s A with A = P diag(sigma) Q^T: the token and feature spectra are
    W^2 sigma^2, and the truncation keeps the first min(r_T, r_d) singular triplets, so
    tau = sum_{i >= min(r_T, r_d)} sigma_i^2 / sum_i sigma_i^2."""
    m, T, d = 4, 12, 6
    P, _ = np.linalg.qr(rng.standard_normal((T, d)))
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    sig = np.array([5.0, 3.0, 2.0, 1.2, 0.7, 0.3])
    A = P @ np.diag(sig) @ Q.T
    w = np.array([1.0, -0.5, 2.0, 0.25])
    X = np.stack([w[s] * A for s in range(m)])
    _, U_T = tk.token_spectrum_exact(X)
    rs, mu, tab, E = _tau_table(X, U_T, 1)
    W2 = float(np.sum(w * w))
    for k, rT in enumerate(rs):
        expect_mu = np.zeros(d)
        n = min(rT, d)
        expect_mu[:n] = W2 * sig[:n] ** 2
        np.testing.assert_allclose(mu[k], expect_mu, rtol=0, atol=1e-11 * W2 * sig[0] ** 2)
        for rd in range(1, d + 1):
            r = min(rT, rd)
            assert tab[k][rd] == pytest.approx(np.sum(sig[r:] ** 2) / np.sum(sig ** 2), abs=1e-12)


def test_full_token_rank_gives_the_feature_tail_and_full_feature_rank_the_token_tail(rng):
    X = lowrank_cell(rng, 2, 16, 8, 4, noise=0.1)
    lam_T, U_T = tk.token_spectrum_exact(X)
    lam_d, _ = tk.feature_spectrum(X)
    rs, mu, tab, E = _tau_table(X, U_T, 1)
    tauT = tk.tail_fractions(lam_T, E)
    taud = tk.tail_fractions(lam_d, E)
    # r_T = T keeps the whole cell in the token mode: mu is the feature spectrum of X
    np.testing.assert_allclose(mu[-1], lam_d, rtol=0, atol=1e-10 * lam_d[0])
    np.testing.assert_allclose(tab[-1][1:], taud[1:], rtol=0, atol=1e-12)
    # r_d = d keeps everything in the feature mode: only the token tail is discarded
    for k, rT in enumerate(rs):
        assert tab[k][8] == pytest.approx(tauT[rT], abs=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_two_sided_mode_tail_bounds(seed):
    """max(tau_T(r_T), tau_d(r_d)) <= tau <= min(1, tau_T(r_T) + tau_d(r_d)): a rank-r
    mode projection cannot beat the best rank-r approximation of that unfolding, and the
    sequential truncation is within the sum of the mode tails (Vannieuwenhoven et al.)."""
    rng = np.random.default_rng(100 + seed)
    X = lowrank_cell(rng, 3, 18, 10, 6, noise=0.3)
    lam_T, U_T = tk.token_spectrum_exact(X)
    lam_d, _ = tk.feature_spectrum(X)
    rs, mu, tab, E = _tau_table(X, U_T, 1)
    tauT = tk.tail_fractions(lam_T, E)
    taud = tk.tail_fractions(lam_d, E)
    for k, rT in enumerate(rs):
        for rd in range(1, 11):
            t = tab[k][rd]
            assert t >= max(tauT[rT], taud[rd]) - 1e-12
            assert t <= min(1.0, tauT[rT] + taud[rd]) + 1e-12
    # monotone: more rank never discards more
    assert (np.diff(tab[:, 1:], axis=0) <= 1e-12).all()
    assert (np.diff(tab[:, 1:], axis=1) <= 1e-12).all()


def test_flash_factor_tau_is_the_explicit_error(rng):
    """The table holds for any orthonormal token factor, the FlashJoLT one included
    (its mass outside the sketch is counted automatically)."""
    X = lowrank_cell(rng, 4, 40, 8, 6, noise=0.2)
    sp = pipeline.spectrum(X, method="flash", q=12, p=4, power_iters=1, seed=3)
    U_T = sp["U_T"]
    E = sp["E"]
    rs = list(range(2, sp["rT_max"] + 1, 2))
    tab = alloc.st_tau_table(E, tk.truncated_feature_spectra(X, U_T, rs))
    for k, rT in enumerate(rs):
        for rd in (1, 3, 8):
            assert tab[k][rd] == pytest.approx(_explicit_error(X, U_T, rT, rd) / E, abs=1e-12)


def test_tau_table_degenerate_cases():
    mu = np.array([[3.0, 1.0], [4.0, 0.0]])
    tab = alloc.st_tau_table(4.0, mu)
    np.testing.assert_array_equal(tab, [[1.0, 0.25, 0.0], [1.0, 0.0, 0.0]])
    assert (alloc.st_tau_table(0.0, mu) == 0.0).all()
    # a head sum past E (possible only through rounding of measured spectra) clips at 0
    assert alloc.st_tau_table(1.0, np.array([[0.75, 0.5]]))[0][2] == 0.0


# ------------------------------------------------------------------ the allocator on exact tau
def _exact_cells(rng, n, step, m=2, T=24, d=16):
    out = []
    for i in range(n):
        X = lowrank_cell(rng, m, T, d, 4, noise=0.2 + 0.3 * i, decay=0.5 + i)
        sp = pipeline.spectrum(X)
        rs = list(range(step, T + 1, step))
        mu = tk.truncated_feature_spectra(X, sp["U_T"], rs)
        out.append(alloc.CellSpectrum(m=m, T=T, d=d, c=2, g=8, E=sp["E"], lam_T=sp["lam_T"],
                                      lam_d=sp["lam_d"], rT_max=T, mu=mu))
    return out


def test_exact_tau_allocation_is_optimal_against_brute_force(rng):
    step = 8
    cells = _exact_cells(rng, 3, step)
    per = []
    for c in cells:
        tab = alloc.st_tau_table(c.E, c.mu)
        pts = [(alloc.byte_cost(c.m, c.T, c.d, 0, 0, b, c.c, c.g), EPS2[b] * 1.0, (0, 0, b))
               for b in alloc.BIT_GRID]
        pts += [(alloc.byte_cost(c.m, c.T, c.d, rT, rd, b, c.c, c.g), EPS2[b] * tab[rT // step - 1][rd],
                 (rT, rd, b)) for rT in range(step, c.rT_max + 1, step)
                for rd in range(step, c.d + 1, step) for b in alloc.BIT_GRID]
        per.append(pts)
    total_in = sum(c.m * c.T * c.d * 2 for c in cells)
    for ratio in (1.5, 2.0, 3.0, 6.0):
        res = alloc.allocate(cells, total_in / ratio, EPS2, step=step)
        assert res["total_bytes"] <= total_in / ratio
        best = min(sum(p[1] for p in combo) for combo in itertools.product(*per)
                   if sum(p[0] for p in combo) <= res["total_bytes"])
        assert res["model_error"] <= best + 1e-15


def test_exact_tau_never_models_more_error_than_the_bound(rng):
    """Each grid point's exact tau is at most the additive bound, so at the same budget the
    allocation on exact tau reaches a summed model error no larger than the bound's."""
    step = 8
    ex = _exact_cells(rng, 3, step)
    bd = [alloc.CellSpectrum(m=c.m, T=c.T, d=c.d, c=c.c, g=c.g, E=c.E, lam_T=c.lam_T,
                             lam_d=c.lam_d, rT_max=c.rT_max) for c in ex]
    for c_ex, c_bd in zip(ex, bd):
        s1, e1, P1 = alloc.cell_grid(c_ex, EPS2, step=step)
        s2, e2, P2 = alloc.cell_grid(c_bd, EPS2, step=step)
        np.testing.assert_array_equal(P1, P2)
        assert (e1 <= e2 + 1e-15).all()
    total_in = sum(c.m * c.T * c.d * 2 for c in ex)
    for ratio in (2.0, 4.0):
        a = alloc.allocate(ex, total_in / ratio, EPS2, step=step)
        # the bound's allocation, scored with exact tau, is feasible for the exact problem
        b = alloc.allocate(bd, total_in / ratio, EPS2, step=step)
        e_b = 0.0
        for c, (rT, rd, bits) in zip(ex, b["alloc"]):
            tab = alloc.st_tau_table(c.E, c.mu)
            e_b += EPS2[bits] * (1.0 if rT == 0 else tab[rT // step - 1][rd])
        if b["total_bytes"] <= a["total_bytes"]:
            assert a["model_error"] <= e_b + 1e-15


def test_table_shorter_than_rT_max_caps_the_grid(rng):
    step = 8
    c = _exact_cells(rng, 1, step)[0]
    c.mu = c.mu[:1]                       # only r_T = 8 tabulated
    s, e, P = alloc.cell_grid(c, EPS2, step=step)
    assert set(P[:, 2]) == {0, 8}


def test_compress_cells_on_exact_tau_meets_the_budget_and_its_model(rng):
    cells = [lowrank_cell(rng, 2, 24, 16, 4, noise=0.1 + 0.2 * i) for i in range(2)]
    out = pipeline.compress_cells(cells, ratio=3.0, eps2=EPS2, tau="exact", bits=(0,))
    assert out["allocation"]["total_bytes"] <= out["budget"]
    # with no residual the model error is the exact relative truncation error, so the
    # stored-factor reconstruction lands on it up to the fp16 rounding of the factors
    for X, c, part, (rT, rd, b) in zip(cells, out["cells"], out["parts"], out["allocation"]["alloc"]):
        tab = alloc.st_tau_table(c.E, c.mu)
        model = 1.0 if rT == 0 else tab[rT // 8 - 1][rd]
        got = float(np.sum((X - part["Xhat"]) ** 2)) / c.E
        assert got == pytest.approx(model, abs=2e-3)

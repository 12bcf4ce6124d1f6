"""Pins of the oracle's three-mode spectral diagnostics (section 3, appendix A).

Each test checks the oracle against something other than itself: tensors whose mode
singular values are known in closed form, the energy identity shared by the three
unfoldings, invariances of the definition, hand-computed ranks, and the best low-rank
approximation error of each unfolding formed explicitly from its SVD.
"""
import math

import numpy as np
import pytest

from oracle import diagnostics as dg


def _orth(rng, n, k):
    q, _ = np.linalg.qr(rng.standard_normal((n, k)))
    return q


def test_unfoldings_have_the_mode_index_as_rows(rng):
    X = rng.standard_normal((3, 5, 4))
    assert dg.unfold(X, 0).shape == (3, 20)
    assert dg.unfold(X, 1).shape == (5, 12)
    assert dg.unfold(X, 2).shape == (4, 15)
    # the token unfolding is the token-major matrix whose Gram is the token Gram
    np.testing.assert_array_equal(dg.unfold(X, 1), X.transpose(1, 0, 2).reshape(5, 12))
    assert dg.unfold(X, 2)[1, 7] == X[1, 2, 1]            # column (s, t) = s * T + t, T = 5


def test_rank_one_tensor(rng):
    a, b, c = rng.standard_normal(6), rng.standard_normal(9), rng.standard_normal(5)
    X = np.einsum("s,t,f->stf", a, b, c)
    energy = (a @ a) * (b @ b) * (c @ c)
    for mode in range(3):
        lam = dg.mode_spectrum(X, mode)
        assert lam[0] == pytest.approx(energy, rel=1e-12)
        assert np.all(lam[1:] <= 1e-12 * energy)
        s = dg.mode_summary(lam)
        assert s["ranks"] == [1, 1]
    assert dg.sigma_range(np.array([2.0, 0.0])) == math.inf


def test_orthogonal_rank_k_tensor_has_the_core_values_in_every_mode(rng):
    # X = sum_k g_k u_k (x) v_k (x) w_k with orthonormal {u}, {v}, {w}: every unfolding has
    # singular values |g_k| (and zeros)
    k = 4
    g = np.array([3.0, -2.0, 1.5, 0.25])
    U, V, W = _orth(rng, 7, k), _orth(rng, 11, k), _orth(rng, 6, k)
    X = np.einsum("k,sk,tk,fk->stf", g, U, V, W)
    want = np.sort(g ** 2)[::-1]
    for mode, n in zip(range(3), (7, 11, 6)):
        lam = dg.mode_spectrum(X, mode)
        assert len(lam) == n
        np.testing.assert_allclose(lam[:k], want, rtol=1e-12)
        assert np.all(lam[k:] < 1e-12)
    # ranks by hand: energies 9, 4, 2.25, 0.0625 of 15.3125; errors after r = 1, 2, 3:
    # sqrt(6.3125/15.3125) = 0.642, sqrt(2.3125/15.3125) = 0.389, sqrt(0.0625/15.3125) = 0.0639
    s = dg.mode_summary(dg.mode_spectrum(X, 1), errs=(0.10, 0.20, 0.40, 0.70))
    assert s["ranks"] == [3, 3, 2, 1]


def test_threshold_is_on_the_relative_frobenius_error():
    # eight slices of equal energy (the appendix's head rows): dropping one slice leaves an
    # error of sqrt(1/8) = 0.354 > 0.2, so both thresholds need all eight; a threshold on
    # the discarded energy fraction would keep seven at 20% (1/8 <= 0.2)
    lam = np.full(8, 2.0)
    s = dg.mode_summary(lam)
    assert s["ranks"] == [8, 8] and s["sigma_range"] == 1.0
    # hand-made spectrum: errors after r = 0..4 are 1, 0.7071, 0.4472, 0.2236, 0
    lam = np.array([0.5, 0.3, 0.15, 0.05])
    assert [dg.rank_for_error(lam, e) for e in (0.1, 0.2, 0.25, 0.5, 0.71, 1.0)] == [4, 4, 3, 2, 1, 0]
    assert dg.truncation_error(lam, 3) == pytest.approx(math.sqrt(0.05))
    assert dg.sigma_range(lam) == pytest.approx(math.sqrt(10.0))


def test_the_three_modes_share_the_energy(rng):
    X = rng.standard_normal((5, 33, 8)) * rng.uniform(0.1, 3.0, (5, 1, 1))
    E = float(np.sum(X ** 2))
    for mode in range(3):
        assert dg.mode_spectrum(X, mode).sum() == pytest.approx(E, rel=1e-12)


def test_slice_spectrum_is_invariant_to_rotations_of_the_other_modes(rng):
    X = rng.standard_normal((6, 20, 16))
    Qt, Qf = _orth(rng, 20, 20), _orth(rng, 16, 16)
    Y = np.einsum("stf,tu,fg->sug", X, Qt, Qf)
    np.testing.assert_allclose(dg.mode_spectrum(Y, 0), dg.mode_spectrum(X, 0), rtol=1e-10)
    # and the token spectrum does not depend on the order of the slices
    np.testing.assert_allclose(dg.mode_spectrum(X[::-1], 1), dg.mode_spectrum(X, 1), rtol=1e-10, atol=1e-10)


def test_truncation_error_equals_the_best_low_rank_approximation_error(rng):
    X = rng.standard_normal((4, 9, 6)) @ np.diag(np.geomspace(1.0, 0.01, 6))
    for mode in range(3):
        A = dg.unfold(X, mode)
        u, s, vt = np.linalg.svd(A, full_matrices=False)
        lam = dg.mode_spectrum(X, mode)
        for r in range(A.shape[0] + 1):
            Ar = (u[:, :r] * s[:r]) @ vt[:r]
            want = np.linalg.norm(A - Ar) / np.linalg.norm(A)
            assert dg.truncation_error(lam, r) == pytest.approx(want, rel=1e-8, abs=1e-12)

"""GPU checks of the boundary's error paths and degenerate inputs, through the C-ABI.

* non-finite input: every entry point that computes a spectrum reports JOLT_E_NONFINITE
  (jolt_spectrum, jolt_compress without a reused spectrum, jolt_truncated_spectra), and
  the context keeps working afterwards;
* rank-deficient and all-zero cells are not solver failures (clamped CholeskyQR pivots of
  a first pass and zero eigenvalues are the designed treatment) and still match the oracle;
* JOLT_E_NOCONV: forced from the host with the inverse-iteration limit set to zero sweeps
  (the growth check then fails on any input) and with the two-stage reduction's bulge-chase
  wait bound set to zero, never on the same input with the defaults;
* the int8 core exponent: a core below 2^-113 stores the floor -128 (identically to the
  oracle's serialisation rule), and the oracle's decode of that blob equals the GPU's.
"""
import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from conftest import lowrank_cell
from gpu_util import blob_bytes, ctx, decompress, device_cells, note, workspace
from oracle import pipeline as opl, tucker as otk

pytestmark = pytest.mark.gpu


def keys(T=256, H=4, d=128, seed=0):
    return kvsynth.layer_kv(layer=0, tensor=0, n_heads=H, T=T, d=d, alpha=1.5,
                            data_seed=seed)[0].astype(np.float64)


def blobs_for(desc, params):
    return [torch.zeros(J.jolt_compressed_size(desc, p), dtype=torch.uint8, device="cuda") for p in params]


@pytest.mark.parametrize("bad", [np.nan, np.inf])
@pytest.mark.parametrize("method", ["exact", "flash"])
def test_nonfinite_cell_is_reported(bad, method):
    X = keys()
    xs, ex, desc = device_cells([X, keys(seed=1)], "bf16")
    bits = xs[1].view(torch.int16).clone()
    v = torch.tensor([bad], dtype=torch.bfloat16).view(torch.int16)
    bits[2, 100, 7] = v[0]
    xs[1] = bits.view(torch.bfloat16)
    o = None if method == "exact" else J.SpectrumOpts(J.JOLT_FLASH, 32, 0.0, 10, 1)
    ws = workspace(desc, 2, o)
    seeds = [1, 2]
    note("non-finite", method, bad)
    with pytest.raises(J.JoltError) as e:
        J.jolt_spectrum(ctx(), desc, xs, seeds, o, ws)
    assert e.value.code == J.JOLT_E_NONFINITE
    params = [J.Params(16, 16, 4, 64, J.JOLT_FACTOR_F16, 0, s) for s in seeds]
    with pytest.raises(J.JoltError) as e:
        J.jolt_compress(ctx(), desc, xs, params, o, ws, blobs_for(desc, params))
    assert e.value.code == J.JOLT_E_NONFINITE
    nt = J.jolt_truncated_spectra_workspace_size(desc, 2, 8, 2, o)
    wst = torch.empty(nt, dtype=torch.uint8, device="cuda")
    with pytest.raises(J.JoltError) as e:
        J.jolt_truncated_spectra(ctx(), desc, xs, 8, 2, seeds=seeds, opts=o, ws=wst)
    assert e.value.code == J.JOLT_E_NONFINITE
    # a failed call leaves no spectrum to reuse, and the context serves the next call
    reuse = J.SpectrumOpts(o.method if o else J.JOLT_EXACT, o.q if o else 0, 0.0, o.oversample if o else 0,
                           o.power_iters if o else 0, 1, 0)
    with pytest.raises(J.JoltError) as e:
        J.jolt_compress(ctx(), desc, xs, params, reuse, ws, blobs_for(desc, params))
    assert e.value.code == J.JOLT_E_STATE
    good, _, dgood = device_cells([X], "bf16")
    E, lamT, _ = J.jolt_spectrum(ctx(), dgood, good, [1], o, workspace(dgood, 1, o))
    assert np.isfinite(E).all() and np.isfinite(lamT).all()


@pytest.mark.parametrize("method", ["exact", "flash"])
def test_rank_deficient_and_zero_cells_are_not_solver_failures(method):
    """Rank 3 < r_T and an all-zero cell: the spectra equal the oracle's, compression at
    ranks above the cell's rank succeeds and reconstructs the low-rank cell exactly."""
    rng = np.random.default_rng(7)
    X = lowrank_cell(rng, 4, 300, 64, 3)
    Z = np.zeros_like(X)
    xs, ex, desc = device_cells([X, Z], "f32")
    o = None if method == "exact" else J.SpectrumOpts(J.JOLT_FLASH, 20, 0.0, 10, 1)
    ws = workspace(desc, 2, o)
    note("rank-deficient", method)
    E, lamT, lamd = J.jolt_spectrum(ctx(), desc, xs, [3, 4], o, ws)
    lam_exact, _ = otk.token_spectrum_exact(ex[0])
    n = 20 if method == "flash" else 300
    np.testing.assert_allclose(lamT[0, :n], lam_exact[:n], rtol=0, atol=1e-5 * lam_exact[0])
    assert E[1] == 0.0 and np.all(lamT[1] == 0.0) and np.all(lamd[1] == 0.0)
    params = [J.Params(8, 8, 0, 64, J.JOLT_FACTOR_F32, 0, s) for s in (3, 4)]
    blobs = blobs_for(desc, params)
    J.jolt_compress(ctx(), desc, xs, params, o, ws, blobs)
    torch.cuda.synchronize()
    Xh = decompress(blobs, desc, "f32")
    assert np.linalg.norm(Xh[0] - ex[0]) <= 1e-5 * np.linalg.norm(ex[0])
    assert np.all(Xh[1] == 0.0)


def test_inverse_iteration_limit_reports_noconv():
    X = keys()
    xs, ex, desc = device_cells([X], "bf16")
    ws = workspace(desc, 1)
    p = [J.Params(32, 32, 2, 64, J.JOLT_FACTOR_F16, 0, 1)]
    c2 = J.jolt_create(0)
    try:
        J.jolt_debug_set(c2, J.JOLT_DBG_INVIT_ITERS, 0)
        note("inverse iteration with zero sweeps")
        with pytest.raises(J.JoltError) as e:
            J.jolt_compress(c2, desc, xs, p, None, ws, blobs_for(desc, p))
        assert e.value.code == J.JOLT_E_NOCONV
        with pytest.raises(J.JoltError):
            J.jolt_debug_set(c2, J.JOLT_DBG_INVIT_ITERS, 9)
        J.jolt_debug_set(c2, J.JOLT_DBG_INVIT_ITERS, 2)
        blobs = blobs_for(desc, p)
        J.jolt_compress(c2, desc, xs, p, None, ws, blobs)
        torch.cuda.synchronize()
        assert np.isfinite(decompress(blobs, desc, "f32")[0]).all()
    finally:
        J.jolt_destroy(c2)


def test_tiny_core_takes_the_exponent_floor():
    """An fp32 cell of magnitude 2^-121 with fp16 factors: every core slice lies below
    2^-113, so its exponent is the floor -128 and the stored values stay below 2^15; the
    oracle's decode of the GPU's blob equals the GPU's decode."""
    X = keys(H=2) * 2.0 ** -121
    xs, ex, desc = device_cells([X], "f32")
    p = [J.Params(8, 8, 4, 64, J.JOLT_FACTOR_F16, 0, 3)]
    blobs = blobs_for(desc, p)
    note("tiny core")
    J.jolt_compress(ctx(), desc, xs, p, None, workspace(desc, 1), blobs)
    torch.cuda.synchronize()
    got = opl.read_blob(blob_bytes(blobs[0]))
    assert got["gexp"].min() >= -128 and (got["gexp"] == -128).any()
    assert np.abs(got["G_hat"]).max() < 2.0 ** 15
    Xh = decompress(blobs, desc, "f32")[0]
    want = opl.decode_blob(blob_bytes(blobs[0]))
    assert np.isfinite(Xh).all()
    assert np.linalg.norm(Xh - want) <= 1e-5 * np.linalg.norm(want)


def test_tridiagonalisation_lanes_do_not_change_results():
    """The exact spectrum of a batch of cells is the same bit for bit whether the blocked
    tridiagonalisation runs its matrices as one group on one stream or as several groups on
    up to four streams (JOLT_DBG_TRD_LANES; three cells, so 3 and 4 both give three groups);
    the setting rejects values outside 1..4."""
    cells = [keys(T=1024, H=8, seed=s) for s in range(3)]      # T above the one-workgroup size
    xs, ex, desc = device_cells(cells, "bf16")
    ws = workspace(desc, 3)
    out = []
    c2 = J.jolt_create(0)
    try:
        for lanes in (1, 2, 3, 4):
            J.jolt_debug_set(c2, J.JOLT_DBG_TRD_LANES, lanes)
            note("exact spectrum, tridiagonalisation lanes", lanes)
            E, lamT, lamd = J.jolt_spectrum(c2, desc, xs, None, None, ws)
            torch.cuda.synchronize()
            out.append((np.array(E), np.array(lamT), np.array(lamd)))
        for bad in (0, 5):
            with pytest.raises(J.JoltError):
                J.jolt_debug_set(c2, J.JOLT_DBG_TRD_LANES, bad)
    finally:
        J.jolt_destroy(c2)
    for other in out[1:]:
        for a, b in zip(out[0], other):
            assert np.array_equal(a, b)


def test_two_stage_and_one_stage_reductions_agree():
    """JOLT_DBG_TRD_TWO_STAGE: for T > 768 (here T = 1100, a ragged last panel) the exact
    token spectrum from the two-stage reduction (band of half-bandwidth 32 by panel QR and
    rank-64 updates, then bulge chasing) and from the one-stage blocked reduction agree within
    1e-5 of lambda_1 on fp32 cells, and the token factors at a gapped rank span the same
    subspace (projectors within 1e-4).  A compress that reuses a spectrum recorded by
    jolt_spectrum back-transforms with the reduction that made it, even after the setting
    has changed in between: its blobs equal those of a direct compress in that mode.
    Values outside -1..1 are rejected (-1, the default, chooses by batch size)."""
    cells = [keys(T=1100, H=8, seed=s) for s in range(3)]
    xs, ex, desc = device_cells(cells, "f32")
    ws = workspace(desc, 3)
    p = [J.Params(32, 32, 4, 64, J.JOLT_FACTOR_F32, 0, c) for c in range(3)]
    reuse = J.SpectrumOpts(J.JOLT_EXACT, 0, 0.0, 0, 0, 1, 0)
    lam, proj, direct = {}, {}, {}
    c2 = J.jolt_create(0)
    try:
        for mode in (1, 0):
            J.jolt_debug_set(c2, J.JOLT_DBG_TRD_TWO_STAGE, mode)
            note("exact spectrum, two-stage switch", mode)
            E, lamT, lamd = J.jolt_spectrum(c2, desc, xs, None, None, ws)
            lam[mode] = np.array(lamT)
            J.jolt_debug_set(c2, J.JOLT_DBG_TRD_TWO_STAGE, 1 - mode)
            blobs = blobs_for(desc, p)
            J.jolt_compress(c2, desc, xs, p, reuse, ws, blobs)
            torch.cuda.synchronize()
            U = torch.empty((1100, 32), device="cuda")
            J.jolt_debug_export(c2, 0, 0, U)
            U = U.cpu().numpy().astype(np.float64)
            proj[mode] = U @ U.T
            np.testing.assert_allclose(U.T @ U, np.eye(32), atol=1e-5)
            J.jolt_debug_set(c2, J.JOLT_DBG_TRD_TWO_STAGE, mode)
            ws2 = workspace(desc, 3)
            blobs2 = blobs_for(desc, p)
            J.jolt_compress(c2, desc, xs, p, None, ws2, blobs2)
            torch.cuda.synchronize()
            for a, b in zip(blobs, blobs2):
                assert blob_bytes(a) == blob_bytes(b)
        for bad in (-2, 2):
            with pytest.raises(J.JoltError):
                J.jolt_debug_set(c2, J.JOLT_DBG_TRD_TWO_STAGE, bad)
        J.jolt_debug_set(c2, J.JOLT_DBG_TRD_TWO_STAGE, -1)
    finally:
        J.jolt_destroy(c2)
    for c in range(3):
        sp = opl.spectrum(ex[c])
        for mode in (0, 1):
            np.testing.assert_allclose(lam[mode][c], sp["lam_T"], rtol=0, atol=1e-5 * sp["lam_T"][0])
    lam0 = opl.spectrum(ex[0])["lam_T"]
    assert (lam0[31] - lam0[32]) / lam0[31] > 0.02
    assert np.abs(proj[0] - proj[1]).max() < 1e-4


def test_large_batch_eigenvalues_by_bisection():
    """A call whose matrices times their order reach 32 * 4096 (here 120 token Grams of order
    T = 1100) resolves the tridiagonal eigenvalues by plain bisection instead of quarter-point
    multisection (and reduces by two stages): the token spectra of cells spread over the batch
    match the oracle within 1e-5 of lambda_1 on fp32 cells, and equal those of the same cells
    computed in a call of three (multisection, one stage) to the same bound.  The batch holds
    three synthetic cells, each copy scaled by its own factor (so that a mix-up between
    matrices would show)."""
    n = 120
    base = [keys(T=1100, H=8, seed=1000 + s) for s in range(3)]
    cells = [base[s % 3] * (1.0 + s / 64.0) for s in range(n)]
    xs, ex, desc = device_cells(cells, "f32")
    ws = workspace(desc, n)
    pick = [0, 57, 119]
    xs3, ex3, desc3 = device_cells([cells[c] for c in pick], "f32")
    ws3 = workspace(desc3, 3)
    c2 = J.jolt_create(0)
    try:
        note("exact spectrum of", n, "cells at T = 1100")
        E, lamT, lamd = J.jolt_spectrum(c2, desc, xs, None, None, ws)
        torch.cuda.synchronize()
        lam_big = [np.array(lamT[c]) for c in pick]
        note("exact spectrum of 3 of them")
        E3, lamT3, lamd3 = J.jolt_spectrum(c2, desc3, xs3, None, None, ws3)
        torch.cuda.synchronize()
        lam_small = [np.array(lamT3[i]) for i in range(3)]
    finally:
        J.jolt_destroy(c2)
    for i, c in enumerate(pick):
        sp = opl.spectrum(ex[c])
        tol = 1e-5 * sp["lam_T"][0]
        np.testing.assert_allclose(lam_big[i], sp["lam_T"], rtol=0, atol=tol)
        np.testing.assert_allclose(lam_big[i], lam_small[i], rtol=0, atol=tol)


def test_bulge_chase_that_gives_up_is_reported():
    """JOLT_DBG_BULGE_SPIN = 0 makes the first dependency wait of the two-stage reduction's
    bulge chase give up (forced from the host; the kernel still ends normally): the chase
    leaves NaN on the diagonal and jolt_spectrum reports JOLT_E_NOCONV.  With the default
    bound the same call on the same context succeeds again; values outside 0..2^24 are
    rejected."""
    cells = [keys(T=1024, H=4, seed=s) for s in range(2)]
    xs, ex, desc = device_cells(cells, "f32")
    ws = workspace(desc, 2)
    c2 = J.jolt_create(0)
    try:
        J.jolt_debug_set(c2, J.JOLT_DBG_TRD_TWO_STAGE, 1)
        J.jolt_debug_set(c2, J.JOLT_DBG_BULGE_SPIN, 0)
        note("exact spectrum, bulge chase forced to give up")
        with pytest.raises(J.JoltError) as e:
            J.jolt_spectrum(c2, desc, xs, None, None, ws)
        assert e.value.code == J.JOLT_E_NOCONV
        J.jolt_debug_set(c2, J.JOLT_DBG_BULGE_SPIN, 1 << 24)
        note("exact spectrum, default bound")
        E, lamT, lamd = J.jolt_spectrum(c2, desc, xs, None, None, ws)
        sp = opl.spectrum(ex[0])
        np.testing.assert_allclose(np.array(lamT)[0], sp["lam_T"], rtol=0, atol=1e-5 * sp["lam_T"][0])
        for bad in (-1, (1 << 24) + 1):
            with pytest.raises(J.JoltError):
                J.jolt_debug_set(c2, J.JOLT_DBG_BULGE_SPIN, bad)
    finally:
        J.jolt_destroy(c2)

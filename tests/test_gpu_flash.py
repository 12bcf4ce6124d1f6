"""GPU parity of the FlashJoLT token spectrum (section 5) against the fp64 oracle.

Both sides draw the same seeded Gaussian sketch (Philox4x32-10, Box-Muller,
rounded to bf16), so the randomized range finder is compared against the oracle
run with the same sketch.  The orthonormalisation differs (Householder QR in
the oracle, CholeskyQR2 on the GPU) but only through a rotation inside the
sketch range, which leaves the Ritz values, the captured subspace and every
reconstruction unchanged.  Tolerances as for the exact path: 1e-5 relative for
fp32 cells and 1e-3 for bf16 cells.
"""
import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from conftest import lowrank_cell
from gpu_util import blob_bytes, compress, ctx, decompress, device_cells, note, workspace
from oracle import pipeline as opl, tucker as otk
from oracle.philox import rotation_signs, sketch_matrix
from oracle.residual import quantize, rotate

pytestmark = pytest.mark.gpu


def kv_cell(T, H, d, seed=0, alpha=1.5, tensor=0):
    return kvsynth.layer_kv(layer=0, tensor=tensor, n_heads=H, T=T, d=d, alpha=alpha,
                            data_seed=seed)[0].astype(np.float64)


def flash_opts(q, p=10, iters=1):
    return J.SpectrumOpts(J.JOLT_FLASH, q, 0.0, p, iters)


def export(what, cell, shape, dtype=torch.float32):
    t = torch.empty(shape, dtype=dtype, device="cuda")
    J.jolt_debug_export(ctx(), what, cell, t)
    return t


def test_sketch_bits_match_oracle():
    """Omega (N x l, bf16) equals the oracle's sketch for the cell's seed, T ragged."""
    cells = [kv_cell(300, 4, 64), kv_cell(300, 4, 64, seed=1)]
    xs, ex, desc = device_cells(cells, "bf16")
    o = flash_opts(47)                                    # l = 57: not a multiple of 8
    params = [J.Params(8, 8, 0, 64, J.JOLT_FACTOR_F32, 0, s) for s in (17, 3)]
    compress(xs, desc, params, o)
    N, ell = 4 * 64, 57
    for c, seed in enumerate((17, 3)):
        got = export(3, c, (N, ell), torch.bfloat16).view(torch.int16).cpu().numpy().astype(np.int64)
        want = kvsynth.f32_to_bf16_bits(sketch_matrix(seed, N, ell).astype(np.float32))
        want = want.view(np.int16).astype(np.int64)
        diff = np.abs(got - want)
        # fp64 log/cos may differ in the last place from the host's; a bf16 rounding of such a
        # value can then move by one unit in the last place, never more
        assert np.mean(diff != 0) <= 1e-4 and diff.max() <= 1, (c, np.mean(diff != 0), diff.max())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("iters", [0, 1, 2])
def test_flash_spectrum_matches_oracle(dtype, iters):
    """q = 40, p = 10 on T = 700 (ragged), N = 256; captured Ritz values and the tail mass."""
    cells = [kv_cell(700, 4, 64), kv_cell(700, 4, 64, seed=2, alpha=0.7, tensor=1)]
    xs, ex, desc = device_cells(cells, dtype)
    o = flash_opts(40, 10, iters)
    ws = workspace(desc, 2, o)
    seeds = [5, 6]
    note("jolt_spectrum flash", dtype, "iters", iters)
    E, lamT, lamd = J.jolt_spectrum(ctx(), desc, xs, seeds, o, ws)
    assert lamT.shape == (2, 41)
    tol = 1e-5 if dtype == "f32" else 1e-3
    for c in range(2):
        lam, U, extra = otk.token_spectrum_flash(ex[c], q=40, p=10, power_iters=iters, seed=seeds[c])
        Er = otk.energy(ex[c])
        assert abs(E[c] / Er - 1) < 1e-10
        np.testing.assert_allclose(lamT[c, :40], lam[:40], rtol=0, atol=tol * lam[0])
        assert abs(lamT[c, 40] - lam[40]) <= tol * Er
        np.testing.assert_allclose(lamT[c].sum(), Er, rtol=1e-9)  # captured + tail = E


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_flash_wide_sketch_matches_oracle(dtype):
    """l = 200 spans four 64-wide Cholesky blocks (the last one ragged)."""
    cells = [kv_cell(700, 4, 64, seed=7), kv_cell(700, 4, 64, seed=8, alpha=0.7, tensor=1)]
    xs, ex, desc = device_cells(cells, dtype)
    o = flash_opts(190, 10, 1)
    ws = workspace(desc, 2, o)
    note("jolt_spectrum flash l=200", dtype)
    E, lamT, _ = J.jolt_spectrum(ctx(), desc, xs, [11, 12], o, ws)
    tol = 1e-5 if dtype == "f32" else 1e-3
    for c in range(2):
        lam, _, _ = otk.token_spectrum_flash(ex[c], q=190, p=10, power_iters=1, seed=11 + c)
        np.testing.assert_allclose(lamT[c, :190], lam[:190], rtol=0, atol=tol * lam[0])
        assert abs(lamT[c, 190] - lam[190]) <= tol * E[c]
    p = [J.Params(160, 48, 2, 64, J.JOLT_FACTOR_F32, 0, 11), J.Params(96, 64, 4, 64, J.JOLT_FACTOR_F32, 0, 12)]
    blobs, _ = compress(xs, desc, p, o, ws=ws)
    for c in range(2):
        U = export(0, c, (700, p[c].r_T)).cpu().numpy().astype(np.float64)
        np.testing.assert_allclose(U.T @ U, np.eye(p[c].r_T), atol=1e-5)
        ref = opl.compress_cell(ex[c], r_T=p[c].r_T, r_d=p[c].r_d, bits=p[c].bits, group=64,
                                seed=11 + c, factor_bytes=4, method="flash", q=190, p=10,
                                power_iters=1)
        Xt = export(2, c, (4, 700, 64)).cpu().numpy().astype(np.float64)
        eb_gpu, eb_ref = opl.rel_error(ex[c], Xt), opl.rel_error(ex[c], ref["Xtilde"])
        assert abs(eb_gpu / eb_ref - 1) < tol, (c, eb_gpu, eb_ref)


@pytest.mark.parametrize("dtype,fdt", [("f32", J.JOLT_FACTOR_F32), ("bf16", J.JOLT_FACTOR_F16)])
def test_flash_compress_matches_oracle(dtype, fdt):
    """Fixed ranks (24, 32), 4-bit residual, group 64, one power iteration."""
    X0 = kv_cell(700, 4, 64)
    xs, ex, desc = device_cells([X0, kv_cell(700, 4, 64, seed=4)], dtype)
    o = flash_opts(40, 10, 1)
    p = [J.Params(24, 32, 4, 64, fdt, 0, 9), J.Params(40, 64, 2, 64, fdt, 0, 10)]
    blobs, ws = compress(xs, desc, p, o)
    tol = 1e-5 if dtype == "f32" else 1e-3
    fb = 4 if fdt == J.JOLT_FACTOR_F32 else 2
    for c, (rT, rd, bits, seed) in enumerate(((24, 32, 4, 9), (40, 64, 2, 10))):
        ref = opl.compress_cell(ex[c], r_T=rT, r_d=rd, bits=bits, group=64, seed=seed,
                                factor_bytes=fb, method="flash", q=40, p=10, power_iters=1)
        got = opl.read_blob(blob_bytes(blobs[c]))
        assert (got["r_T"], got["r_d"], got["bits"]) == (rT, rd, bits)
        U = got["U_hat"]
        assert np.abs(U.T @ U - np.eye(rT)).max() < (1e-5 if fb == 4 else 2e-3)
        # the token subspace: projectors agree (Davis-Kahan with the Ritz gap at r_T)
        lam = ref["spec"]["lam_T"]
        gap = lam[rT - 1] - lam[rT] if rT < 40 else lam[rT - 1]
        ptol = min(0.05, max(tol, 1e-5 * lam[0] / gap))
        Ue = ref["U"]
        assert np.abs(U @ U.T - Ue @ Ue.T).max() < ptol + (0 if fb == 4 else 2e-3)
        Xt = export(2, c, (4, 700, 64)).cpu().numpy().astype(np.float64)
        eb_gpu, eb_ref = opl.rel_error(ex[c], Xt), opl.rel_error(ex[c], ref["Xtilde"])
        assert abs(eb_gpu / eb_ref - 1) < tol, (c, eb_gpu, eb_ref)
        codes_ref, _ = quantize(rotate(ex[c] - Xt, rotation_signs(seed, 64)), bits, 64)
        diff = np.abs(got["codes"].astype(int) - codes_ref.astype(int))
        assert np.mean(diff != 0) <= 1e-4 and diff.max() <= 1
    Xh = decompress(blobs, desc, "f32")
    for c, seed in enumerate((9, 10)):
        ref = opl.compress_cell(ex[c], r_T=p[c].r_T, r_d=p[c].r_d, bits=p[c].bits, group=64,
                                seed=seed, factor_bytes=fb, method="flash", q=40, p=10,
                                power_iters=1)
        e_gpu, e_ref = opl.rel_error(ex[c], Xh[c]), opl.rel_error(ex[c], ref["Xhat"])
        note(f"flash e2e {dtype} cell {c}: gpu {e_gpu:.9g} oracle {e_ref:.9g}")
        assert abs(e_gpu / e_ref - 1) < tol, (c, e_gpu, e_ref)


def test_flash_sketch_covering_all_tokens_is_exact():
    """l = T (T = 40 < q + p): the range is all of R^T, so the Ritz values are the exact
    token spectrum's top q and the tail is the exact remainder."""
    X = kv_cell(40, 4, 64)
    xs, ex, desc = device_cells([X], "f32")
    o = flash_opts(36, 10, 1)
    ws = workspace(desc, 1, o)
    note("jolt_spectrum flash l = T")
    E, lamT, _ = J.jolt_spectrum(ctx(), desc, xs, [1], o, ws)
    lam_exact, _ = otk.token_spectrum_exact(ex[0])
    np.testing.assert_allclose(lamT[0, :36], lam_exact[:36], rtol=0, atol=1e-5 * lam_exact[0])
    assert abs(lamT[0, 36] - lam_exact[36:].sum()) <= 1e-5 * E[0]


def test_flash_sketch_covering_all_features_is_exact():
    """l = N (m d = 64 < q + p): B = Q^T X_(2) keeps every direction of the row space."""
    X = kv_cell(300, 2, 32)
    xs, ex, desc = device_cells([X], "f32")
    o = flash_opts(60, 10, 0)
    ws = workspace(desc, 1, o)
    note("jolt_spectrum flash l = N")
    E, lamT, _ = J.jolt_spectrum(ctx(), desc, xs, [2], o, ws)
    lam_exact, _ = otk.token_spectrum_exact(ex[0])
    np.testing.assert_allclose(lamT[0, :60], lam_exact[:60], rtol=0, atol=1e-5 * lam_exact[0])


def test_flash_rank_deficient_cell_stays_finite():
    """Rank 6 < l = 30: the sketch Gram is singular; the captured spectrum and the rank-6
    reconstruction must still be right and every output finite."""
    rng = np.random.default_rng(3)
    X = lowrank_cell(rng, 4, 200, 64, 6)
    xs, ex, desc = device_cells([X], "f32")
    o = flash_opts(20, 10, 1)
    ws = workspace(desc, 1, o)
    note("jolt_spectrum flash rank-deficient")
    E, lamT, _ = J.jolt_spectrum(ctx(), desc, xs, [4], o, ws)
    assert np.all(np.isfinite(lamT))
    lam_exact, _ = otk.token_spectrum_exact(ex[0])
    np.testing.assert_allclose(lamT[0, :20], lam_exact[:20], rtol=0, atol=1e-5 * lam_exact[0])
    assert abs(lamT[0, 20]) <= 1e-5 * E[0]
    blobs, _ = compress(xs, desc, [J.Params(6, 6, 0, 64, J.JOLT_FACTOR_F32, 0, 4)], o, ws=ws)
    Xh = decompress(blobs, desc, "f32")[0]
    assert np.linalg.norm(Xh - ex[0]) <= 1e-5 * np.linalg.norm(ex[0])

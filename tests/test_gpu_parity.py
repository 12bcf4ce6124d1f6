"""GPU parity of the HIP path against the fp64 oracle, called through the C-ABI.

Tolerances (from the stated targets): reconstruction and relative Frobenius
errors within 1e-5 relative for fp32 cells and 1e-3 for bf16 cells;
quantiser codes equal except for at most 1e-4 of the entries, each off by at
most one level; eigenvalues within the same relative bound in units of the
largest.  Factors are compared through reconstructions and projectors, never
entry by entry (their signs and rotations inside degenerate eigenspaces are
not unique).
"""
import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from conftest import lowrank_cell
from gpu_util import blob_bytes, compress, ctx, decompress, device_cells, note, workspace
from oracle import alloc as oalloc, pipeline as opl

pytestmark = pytest.mark.gpu


def keys_cell(T=256, H=8, d=128, seed=0):
    return kvsynth.layer_kv(layer=0, tensor=0, n_heads=H, T=T, d=d, alpha=1.5, data_seed=seed)[0] \
        .astype(np.float64)


def code_mismatch(a, b):
    diff = np.abs(a.astype(int) - b.astype(int))
    return float(np.mean(diff != 0)), int(diff.max()) if diff.size else 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_spectrum_matches_oracle(dtype):
    xs, ex, desc = device_cells([keys_cell(), keys_cell(seed=1)], dtype)
    ws = workspace(desc, 2)
    note("jolt_spectrum exact", dtype, desc.T)
    E, lamT, lamd = J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    tol = 1e-5 if dtype == "f32" else 1e-3
    for c in range(2):
        sp = opl.spectrum(ex[c])
        assert abs(E[c] / sp["E"] - 1) < 1e-10
        np.testing.assert_allclose(lamT[c], sp["lam_T"], rtol=0, atol=tol * sp["lam_T"][0])
        np.testing.assert_allclose(lamd[c], sp["lam_d"], rtol=0, atol=tol * sp["lam_d"][0])


@pytest.mark.parametrize("dtype,fdt", [("f32", J.JOLT_FACTOR_F32), ("bf16", J.JOLT_FACTOR_F16)])
def test_fixed_rank_cell_matches_oracle(dtype, fdt):
    """keys, n_h = 8, T = 256, d = 128, ranks (64, 64), 2-bit residual, group 64, seed 0."""
    xs, ex, desc = device_cells([keys_cell()], dtype)
    p = J.Params(64, 64, 2, 64, fdt, 0, 0)
    blobs, ws = compress(xs, desc, [p])
    X = ex[0]
    ref = opl.compress_cell(X, r_T=64, r_d=64, bits=2, group=64, seed=0,
                            factor_bytes=4 if fdt == J.JOLT_FACTOR_F32 else 2)
    got = opl.read_blob(blob_bytes(blobs[0]))
    assert (got["m"], got["T"], got["d"], got["r_T"], got["r_d"], got["bits"], got["group"]) == \
        (8, 256, 128, 64, 64, 2, 64)
    tol = 1e-5 if dtype == "f32" else 1e-3
    # backbone: the cut at 64 lies in the noise bulk, so compare the backbone error
    Xt_gpu = torch.empty((8, 256, 128), device="cuda")
    J.jolt_debug_export(ctx(), 2, 0, Xt_gpu)
    Xt_gpu = Xt_gpu.cpu().numpy().astype(np.float64)
    eb_ref = opl.rel_error(X, ref["Xtilde"])
    eb_gpu = opl.rel_error(X, Xt_gpu)
    assert abs(eb_gpu / eb_ref - 1) < tol, (eb_gpu, eb_ref)
    # the GPU's X~ is the reconstruction of its own stored factors
    Xt_blob = opl.decode_parts_from_factors(got["U_hat"], got["Ud_hat"], got["G_hat"], got["gexp"],
                                            None, None, T=256, d=128, bits=0, group=64, seed=0)
    assert np.linalg.norm(Xt_gpu - Xt_blob) <= 1e-5 * np.linalg.norm(X)
    # factors are orthonormal up to their stored precision
    U = got["U_hat"]
    assert np.abs(U.T @ U - np.eye(64)).max() < (1e-5 if fdt == J.JOLT_FACTOR_F32 else 2e-3)
    # codes: the oracle's quantiser applied to the GPU's own X~ (stage-wise parity)
    from oracle.philox import rotation_signs
    from oracle.residual import quantize, rotate
    codes_ref, scales_ref = quantize(rotate(X - Xt_gpu, rotation_signs(0, 128)), 2, 64)
    frac, mx = code_mismatch(got["codes"], codes_ref)
    assert frac <= 1e-4 and mx <= 1, (frac, mx)
    np.testing.assert_allclose(got["scales"], scales_ref, rtol=2e-3)
    # decoding: the GPU's decompression of its own blob equals the oracle's decode of it
    Xh = decompress(blobs, desc, "f32")[0]
    Xh_orc = opl.decode_blob(blob_bytes(blobs[0]))
    assert np.linalg.norm(Xh - Xh_orc) <= 1e-5 * np.linalg.norm(X)
    # end to end: the relative error against the oracle's at the stated tolerance
    e_gpu, e_ref = opl.rel_error(X, Xh), opl.rel_error(X, ref["Xhat"])
    sp = ref["spec"]
    note(f"e2e {dtype}: gpu {e_gpu:.9g} oracle {e_ref:.9g} ratio-1 {e_gpu / e_ref - 1:.3g}; "
         f"token gap/lam1 {(sp['lam_T'][63] - sp['lam_T'][64]) / sp['lam_T'][0]:.3g}")
    assert abs(e_gpu / e_ref - 1) < tol, (e_gpu, e_ref)


@pytest.mark.parametrize("bits", [2, 4])
def test_gapped_fp32_cell_end_to_end(bits):
    """fp32 cell of token and feature rank 32 plus noise, cut at (32, 32) where both mode
    spectra have a wide gap: the backbone is determined to working accuracy, so the GPU's
    X~ matches the oracle's entry by entry and the end-to-end error to 1e-5."""
    rng = np.random.default_rng(40 + bits)
    X = lowrank_cell(rng, 8, 256, 128, 32, noise=0.02, decay=0.5)
    xs, ex, desc = device_cells([X], "f32")
    p = J.Params(32, 32, bits, 64, J.JOLT_FACTOR_F32, 0, 5)
    blobs, ws = compress(xs, desc, [p])
    ref = opl.compress_cell(ex[0], r_T=32, r_d=32, bits=bits, group=64, seed=5, factor_bytes=4)
    sp = ref["spec"]
    relgap_T = (sp["lam_T"][31] - sp["lam_T"][32]) / sp["lam_T"][31]
    relgap_d = (sp["lam_d"][31] - sp["lam_d"][32]) / sp["lam_d"][31]
    assert relgap_T > 0.5 and relgap_d > 0.5
    Xt = torch.empty((8, 256, 128), device="cuda")
    J.jolt_debug_export(ctx(), 2, 0, Xt)
    Xt = Xt.cpu().numpy().astype(np.float64)
    nX = np.linalg.norm(ex[0])
    assert np.linalg.norm(Xt - ref["Xtilde"]) <= 1e-5 * nX
    Xh = decompress(blobs, desc, "f32")[0]
    e_gpu, e_ref = opl.rel_error(ex[0], Xh), opl.rel_error(ex[0], ref["Xhat"])
    note(f"gapped b={bits}: e gpu {e_gpu:.9g} oracle {e_ref:.9g}")
    assert abs(e_gpu / e_ref - 1) < 1e-5, (e_gpu, e_ref)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_residual_only_codes_match_oracle(bits):
    """ranks (0, 0): X~ = 0, the residual is X itself; codes stage-wise exact."""
    rng = np.random.default_rng(bits)
    cells = [rng.standard_normal((4, 100, 128)) * np.exp(rng.uniform(-2, 2, (4, 100, 1))) for _ in range(3)]
    xs, ex, desc = device_cells(cells, "bf16")
    params = [J.Params(0, 0, bits, 64, J.JOLT_FACTOR_F16, 0, 11 + c) for c in range(3)]
    blobs, ws = compress(xs, desc, params)
    for c in range(3):
        ref = opl.compress_cell(ex[c], r_T=0, r_d=0, bits=bits, group=64, seed=11 + c)
        got = opl.read_blob(blob_bytes(blobs[c]))
        frac, mx = code_mismatch(got["codes"], ref["codes"])
        assert frac <= 1e-4 and mx <= 1, (c, frac, mx)
        np.testing.assert_allclose(got["scales"], ref["scales"], rtol=1e-3)


@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_decompress_of_oracle_blob(out_dtype):
    """The oracle writes a blob; the GPU decoder must reproduce the oracle's decode."""
    X = keys_cell(T=192, H=4)
    ref = opl.compress_cell(X, r_T=40, r_d=48, bits=4, group=32, seed=7, factor_bytes=2)
    blob = opl.write_blob(ref, in_dtype="bf16", n_heads=4)
    b = torch.from_numpy(np.frombuffer(blob, np.uint8).copy()).cuda()
    _, _, desc = device_cells([X], "bf16")
    Xh = decompress([b], desc, out_dtype)[0]
    want = opl.cast_output(ref["Xhat"], out_dtype)
    if out_dtype == "f32":
        assert np.linalg.norm(Xh - want) <= 1e-5 * np.linalg.norm(want)
    else:
        # bf16 outputs: equal except where fp32 rounding of the sum crosses a bf16 boundary
        diff = Xh != want
        assert diff.mean() < 1e-3
        assert np.all(np.abs(Xh - want) <= np.abs(want) * 2 ** -7 + 1e-30)


def test_eps2_matches_oracle():
    ws = torch.empty(J.jolt_eps2_workspace_size(128, 1 << 20), dtype=torch.uint8, device="cuda")
    note("jolt_eps2_calibrate")
    got = J.jolt_eps2_calibrate(ctx(), 64, 128, 0, 1 << 20, ws)
    ref = oalloc.calibrate_eps2(group=64, d=128, seed=0, n_samples=1 << 20)
    for b in (0, 2, 4, 8):
        assert abs(got[b] / ref[b] - 1) < 1e-4, (b, got[b], ref[b])


def test_compress_is_deterministic():
    xs, ex, desc = device_cells([keys_cell(T=128, H=4)], "bf16")
    p = [J.Params(32, 32, 4, 64, J.JOLT_FACTOR_F16, 0, 5)]
    b1, ws = compress(xs, desc, p)
    b2, _ = compress(xs, desc, p, ws=ws)
    assert blob_bytes(b1[0]) == blob_bytes(b2[0])
    p3 = [J.Params(32, 32, 4, 64, J.JOLT_FACTOR_F16, 0, 6)]
    b3, _ = compress(xs, desc, p3, ws=ws)
    assert blob_bytes(b3[0]) != blob_bytes(b1[0])


def test_spectrum_then_compress_reuses_and_matches_direct():
    xs, ex, desc = device_cells([keys_cell(T=128, H=4), keys_cell(T=128, H=4, seed=3)], "bf16")
    ws = workspace(desc, 2)
    E, lamT, lamd = J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    params = [J.Params(16, 24, 4, 64, J.JOLT_FACTOR_F16, 0, 1), J.Params(24, 16, 2, 64, J.JOLT_FACTOR_F16, 0, 2)]
    reuse = J.SpectrumOpts(J.JOLT_EXACT, 0, 0.0, 0, 0, 1, 0)
    b_reuse, _ = compress(xs, desc, params, reuse, ws=ws)
    b_again, _ = compress(xs, desc, params, reuse, ws=ws)     # compress keeps the spectrum
    ws2 = workspace(desc, 2)
    b_direct, _ = compress(xs, desc, params, ws=ws2)
    for a, b, c in zip(b_reuse, b_again, b_direct):
        assert blob_bytes(a) == blob_bytes(b) == blob_bytes(c)


@pytest.fixture(params=[0, 1], ids=["one_stage", "two_stage"])
def reduction(request):
    """Runs a test with the one-stage and with the two-stage reduction of the large token
    Grams (JOLT_DBG_TRD_TWO_STAGE on the shared context), restoring the automatic choice."""
    J.jolt_debug_set(ctx(), J.JOLT_DBG_TRD_TWO_STAGE, request.param)
    yield request.param
    J.jolt_debug_set(ctx(), J.JOLT_DBG_TRD_TWO_STAGE, -1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_blocked_tridiagonalisation_spectrum_and_subspace(dtype, reduction):
    """T = 1024 > 768 takes the blocked multi-workgroup tridiagonalisation (one or two
    stages)."""
    X = keys_cell(T=1024, H=4)
    xs, ex, desc = device_cells([X, keys_cell(T=1024, H=4, seed=5)], dtype)
    ws = workspace(desc, 2)
    note("jolt_spectrum exact T=1024", dtype)
    E, lamT, lamd = J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    tol = 1e-5 if dtype == "f32" else 1e-3
    for c in range(2):
        sp = opl.spectrum(ex[c])
        np.testing.assert_allclose(lamT[c], sp["lam_T"], rtol=0, atol=tol * sp["lam_T"][0])
    # r_T = 32: one layer's heads share a rank-32 token factor, so the cut has a clear gap;
    # Davis-Kahan bounds the subspace difference by ||dC|| / gap with ||dC|| ~ 1e-5 ||C||
    sp = opl.spectrum(ex[0])
    lam = sp["lam_T"]
    gap = lam[31] - lam[32]
    assert gap / lam[31] > 0.02
    ptol = min(0.05, 1e-5 * lam[0] / gap)
    fdt = J.JOLT_FACTOR_F32 if dtype == "f32" else J.JOLT_FACTOR_F16
    p = [J.Params(32, 32, 4, 64, fdt, 0, 0), J.Params(48, 40, 2, 64, fdt, 0, 1)]
    blobs, _ = compress(xs, desc, p, ws=ws)
    U = torch.empty((1024, 32), device="cuda")
    J.jolt_debug_export(ctx(), 0, 0, U)
    U = U.cpu().numpy().astype(np.float64)
    Ue = sp["U_T"][:, :32]
    assert np.abs(U @ U.T - Ue @ Ue.T).max() < ptol
    np.testing.assert_allclose(U.T @ U, np.eye(32), atol=1e-5)
    ref = opl.compress_cell(ex[0], r_T=32, r_d=32, bits=4, group=64, seed=0,
                            factor_bytes=4 if dtype == "f32" else 2, spec=sp)
    Xt = torch.empty((4, 1024, 128), device="cuda")
    J.jolt_debug_export(ctx(), 2, 0, Xt)
    Xt = Xt.cpu().numpy().astype(np.float64)
    # backbone error (first-order insensitive to the subspace) within the stated tolerance
    eb_gpu, eb_ref = opl.rel_error(ex[0], Xt), opl.rel_error(ex[0], ref["Xtilde"])
    assert abs(eb_gpu / eb_ref - 1) < tol, (eb_gpu, eb_ref)
    assert np.linalg.norm(Xt - ref["Xtilde"]) <= max(tol, ptol) * np.linalg.norm(ex[0])


@pytest.mark.parametrize("T,H", [(1001, 4), (900, 1)])
def test_blocked_tridiagonalisation_ragged_and_rank_deficient(T, H, reduction):
    """T = 1001: the last panel is ragged and rows are not 16-byte aligned; H = 1 with
    T = 900 > N = 128: the token Gram has rank 128, so the trailing columns of the
    reduction are numerically zero.  Spectrum within 1e-5 of lambda_1 (fp32 cell) and the
    backbone error at a gapped rank within 1e-5 relative."""
    X = keys_cell(T=T, H=H, seed=3)
    xs, ex, desc = device_cells([X], "f32")
    ws = workspace(desc, 1)
    note("jolt_spectrum exact blocked", T, H)
    E, lamT, lamd = J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    sp = opl.spectrum(ex[0])
    np.testing.assert_allclose(lamT[0], sp["lam_T"], rtol=0, atol=1e-5 * sp["lam_T"][0])
    assert np.all(np.isfinite(lamT))
    p = [J.Params(32, 32, 4, 64, J.JOLT_FACTOR_F32, 0, 0)]
    blobs, _ = compress(xs, desc, p, ws=ws)
    U = torch.empty((T, 32), device="cuda")
    J.jolt_debug_export(ctx(), 0, 0, U)
    U = U.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(U.T @ U, np.eye(32), atol=1e-5)
    ref = opl.compress_cell(ex[0], r_T=32, r_d=32, bits=4, group=64, seed=0, factor_bytes=4, spec=sp)
    Xt = torch.empty((H, T, 128), device="cuda")
    J.jolt_debug_export(ctx(), 2, 0, Xt)
    Xt = Xt.cpu().numpy().astype(np.float64)
    eb_gpu, eb_ref = opl.rel_error(ex[0], Xt), opl.rel_error(ex[0], ref["Xtilde"])
    assert abs(eb_gpu / eb_ref - 1) < 1e-5, (eb_gpu, eb_ref)


def test_workspace_overwrite_forgets_the_spectrum():
    """Reuse is explicit: after a decompress into the workspace that held the spectrum, a
    compress asking for reuse is refused, and one that recomputes equals a fresh one."""
    xs, ex, desc = device_cells([keys_cell(T=128, H=4, seed=9), keys_cell(T=128, H=4, seed=10)], "bf16")
    ws = workspace(desc, 2)
    params = [J.Params(16, 24, 4, 64, J.JOLT_FACTOR_F16, 0, 3), J.Params(24, 16, 2, 64, J.JOLT_FACTOR_F16, 0, 4)]
    reuse = J.SpectrumOpts(J.JOLT_EXACT, 0, 0.0, 0, 0, 1, 0)
    J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    blobs, _ = compress(xs, desc, params, ws=workspace(desc, 2))
    decompress(blobs, desc, "f32", ws=ws)          # overwrites ws
    with pytest.raises(J.JoltError) as ei:
        compress(xs, desc, params, reuse, ws=ws)
    assert ei.value.code == -7                    # JOLT_E_STATE
    b_after, _ = compress(xs, desc, params, ws=ws)
    for a, b in zip(blobs, b_after):
        assert blob_bytes(a) == blob_bytes(b)
    # two workspaces keep their own spectra
    ws2 = workspace(desc, 2)
    J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    J.jolt_spectrum(ctx(), desc, xs, None, None, ws2)
    b1, _ = compress(xs, desc, params, reuse, ws=ws)
    b2, _ = compress(xs, desc, params, reuse, ws=ws2)
    for a, b, c in zip(blobs, b1, b2):
        assert blob_bytes(a) == blob_bytes(b) == blob_bytes(c)


@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_decompress_reapplies_rope(out_dtype):
    """Appendix B: keys compressed before RoPE, rotation re-applied while decoding.  The
    decoder with RoPE equals the oracle's decode of the same blob followed by the oracle's
    rotation (base 1e6, positions 1000 + t)."""
    from oracle.rope import rope
    X = keys_cell(T=256, H=8, seed=2)
    xs, ex, desc = device_cells([X], "bf16")
    blobs, ws = compress(xs, desc, [J.Params(48, 64, 4, 64, J.JOLT_FACTOR_F16, 0, 5)])
    got_blob = opl.read_blob(blob_bytes(blobs[0]))
    dec = opl.decode_parts_from_factors(got_blob["U_hat"], got_blob["Ud_hat"], got_blob["G_hat"],
                                        got_blob["gexp"], got_blob["codes"], got_blob["scales"],
                                        T=256, d=128, bits=4, group=64, seed=5)
    want = rope(dec, 1e6, np.arange(256) + 1000.0)
    od = J.cell_desc(dtype=J.JOLT_BF16 if out_dtype == "bf16" else J.JOLT_F32, n_layers=1, n_heads=8,
                     T=256, d=128, stride_layer=8 * 256 * 128, stride_head=256 * 128, stride_token=128)
    out = torch.empty((8, 256, 128), dtype=torch.bfloat16 if out_dtype == "bf16" else torch.float32,
                      device="cuda")
    note("jolt_decompress_rope", out_dtype)
    J.jolt_decompress(ctx(), blobs, od, [out], ws, rope=(1e6, 1000))
    torch.cuda.synchronize()
    Xh = out.float().cpu().numpy().astype(np.float64)
    if out_dtype == "f32":
        assert np.linalg.norm(Xh - want) <= 1e-5 * np.linalg.norm(want)
    else:
        w16 = opl.cast_output(want, "bf16")
        diff = np.abs(Xh - w16)
        assert np.mean(diff != 0) < 1e-3
        assert (diff - np.abs(w16) * 2 ** -7).max() <= 1e-5 * float(np.sqrt(np.mean(X * X)))
    with pytest.raises(J.JoltError):
        J.jolt_decompress(ctx(), blobs, od, [out], ws, rope=(1.0, 0))


@pytest.mark.parametrize("dtype,d,r,bits,group", [("bf16", 32, 13, 8, 8), ("f32", 64, 21, 2, 16),
                                                  ("bf16", 128, 40, 4, 128), ("bf16", 128, 96, 8, 32)])
def test_fused_passes_shape_variants(dtype, d, r, bits, group):
    """The fused residual and decode passes (fp16 factors) over shapes their tiling treats
    apart: d = 32 / 64 / 128, T = 300 (two full 128-token tiles and a ragged one), r_T not a
    multiple of 8 (U_T rows read entry by entry) or up to three 32-row blocks of r_d,
    quantiser groups of 8 to 128 entries, 2 / 4 / 8-bit codes, bf16 and fp32 cells.
    Stage-wise against the oracle: X~ is the reconstruction of the blob's own factors, the
    codes and scales are the oracle quantiser's on X - X~, the decode is the oracle's decode
    of the blob."""
    rng = np.random.default_rng(1000 + d + r)
    X = lowrank_cell(rng, 4, 300, d, min(r, d), noise=0.02, decay=0.5)
    xs, ex, desc = device_cells([X], dtype)
    p = J.Params(r, min(r, d), bits, group, J.JOLT_FACTOR_F16, 0, 9)
    blobs, ws = compress(xs, desc, [p])
    got = opl.read_blob(blob_bytes(blobs[0]))
    nX = np.linalg.norm(ex[0])
    Xt_gpu = torch.empty((4, 300, d), device="cuda")
    J.jolt_debug_export(ctx(), 2, 0, Xt_gpu)
    Xt_gpu = Xt_gpu.cpu().numpy().astype(np.float64)
    Xt_blob = opl.decode_parts_from_factors(got["U_hat"], got["Ud_hat"], got["G_hat"], got["gexp"],
                                            None, None, T=300, d=d, bits=0, group=group, seed=9)
    assert np.linalg.norm(Xt_gpu - Xt_blob) <= 1e-5 * nX
    from oracle.philox import rotation_signs
    from oracle.residual import quantize, rotate
    codes_ref, scales_ref = quantize(rotate(ex[0] - Xt_gpu, rotation_signs(9, d)), bits, group)
    frac, mx = code_mismatch(got["codes"], codes_ref)
    assert frac <= 1e-4 and mx <= 1, (frac, mx)
    np.testing.assert_allclose(got["scales"], scales_ref, rtol=2e-3)
    Xh = decompress(blobs, desc, "f32")[0]
    Xh_orc = opl.decode_blob(blob_bytes(blobs[0]))
    assert np.linalg.norm(Xh - Xh_orc) <= 1e-5 * nX

"""GPU parity of the three-mode spectral diagnostics (section 3, appendix A) against the
fp64 oracle, through the C-ABI.

The slice-mode spectrum comes from jolt_slice_spectrum, the token- and feature-mode
spectra from jolt_spectrum (exact method); each is summarised by jolt_mode_summary
(pinned against the oracle on the host).  Tolerances: eigenvalues within 1e-5 of the
largest for the slice and feature modes (their Grams are accumulated in fp32 per token and
fp64 across tokens), the stated 1e-5 (fp32) / 1e-3 (bf16) for the token mode; effective
ranks equal to the oracle's unless the oracle's truncation error sits within the
eigenvalue tolerance of the threshold.
"""
import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from gpu_util import ctx, note, workspace
from oracle import diagnostics as dg

pytestmark = pytest.mark.gpu


def _upload(x, dtype):
    """fp64 array -> (device tensor of the cache dtype, exact fp64 copy)."""
    if dtype == "bf16":
        bits = kvsynth.f32_to_bf16_bits(x.astype(np.float32))
        t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return t, kvsynth.bf16_bits_to_f32(bits).astype(np.float64)
    x32 = x.astype(np.float32)
    return torch.from_numpy(x32.copy()).cuda(), x32.astype(np.float64)


def _slice_spectrum(t, desc, n_cells=1, cells=None):
    ws = torch.empty(J.jolt_slice_spectrum_workspace_size(desc, n_cells), dtype=torch.uint8, device="cuda")
    note("jolt_slice_spectrum", desc.n_layers, "x", desc.n_heads, "slices, T", desc.T, "d", desc.d)
    lam = J.jolt_slice_spectrum(ctx(), desc, cells if cells is not None else [t], ws)
    torch.cuda.synchronize()
    return lam


def _rank_ok(lam_oracle, r_gpu, err, tol_err=1e-3):
    """The GPU's effective rank equals the oracle's, or is its neighbour where the oracle's
    truncation error at the lower of the two ranks is within tol_err of the threshold."""
    r_want = dg.rank_for_error(lam_oracle, err)
    if r_gpu == r_want:
        return True
    if abs(r_gpu - r_want) != 1:
        return False
    return abs(dg.truncation_error(lam_oracle, min(r_gpu, r_want)) - err) <= tol_err or \
        abs(dg.truncation_error(lam_oracle, max(r_gpu, r_want)) - err) <= tol_err


@pytest.mark.parametrize("dtype,L,H,B,T,d", [
    ("bf16", 1, 8, 1, 1024, 128),     # one Mistral-shaped layer at the appendix's T
    ("f32", 1, 40, 1, 300, 64),       # m not a multiple of 16, ragged token chunks
    ("bf16", 5, 40, 2, 256, 128),     # a LLaMA-shaped group (m = 200) inside a batch-2 cache
    ("f32", 1, 1, 1, 100, 32),        # a single slice
])
def test_slice_spectrum_matches_oracle(dtype, L, H, B, T, d):
    rng = np.random.default_rng(7)
    # slices of unequal energy with shared token structure
    cache = rng.standard_normal((L, B, H, T, d)) * rng.uniform(0.2, 2.0, (L, 1, H, 1, 1))
    cache += 0.5 * rng.standard_normal((1, 1, 1, T, d))
    t, exact = _upload(cache, dtype)
    desc = J.cell_desc(dtype=J.JOLT_BF16 if dtype == "bf16" else J.JOLT_F32, n_layers=L, n_heads=H,
                       T=T, d=d, stride_layer=B * H * T * d, stride_head=T * d, stride_token=d)
    # the cell of batch item B - 1 (slice s = layer * H + head)
    cell_ptr = t[0, B - 1]
    lam = _slice_spectrum(None, desc, 1, [cell_ptr])[0]
    X = exact[:, B - 1].reshape(L * H, T, d)
    want = dg.mode_spectrum(X, 0)
    assert lam.shape == want.shape
    np.testing.assert_allclose(lam, want, rtol=0, atol=1e-5 * want[0])


@pytest.mark.parametrize("tensor", [0, 1])
def test_three_mode_table_matches_oracle(tensor):
    """Appendix A's table for one layer of the Mistral-shaped synthetic cache (T = 1024)."""
    H, T, d = 8, 1024, 128
    x = kvsynth.layer_kv(layer=15, tensor=tensor, n_heads=H, T=T, d=d, alpha=(1.5, 0.7)[tensor],
                         n_out=2, out_scale=10.0, data_seed=0)[0].astype(np.float64)
    t, X = _upload(x, "bf16")
    desc = J.cell_desc(dtype=J.JOLT_BF16, n_layers=1, n_heads=H, T=T, d=d,
                       stride_layer=H * T * d, stride_head=T * d, stride_token=d)
    lam_s = _slice_spectrum(t, desc)[0]
    ws = workspace(desc, 1)
    note("jolt_spectrum exact", T)
    E, lam_t, lam_f = J.jolt_spectrum(ctx(), desc, [t], None, None, ws)
    torch.cuda.synchronize()
    got = {"slices": lam_s, "tokens": lam_t[0], "features": lam_f[0]}
    for k, mode in enumerate(dg.MODES):
        want = dg.mode_spectrum(X, k)
        tol = 1e-3 if mode == "tokens" else 1e-5
        np.testing.assert_allclose(got[mode], want, rtol=0, atol=tol * want[0])
        rng_, ra, rb = J.jolt_mode_summary(got[mode], 0.10, 0.20)
        for r, e in ((ra, 0.10), (rb, 0.20)):
            assert _rank_ok(want, r, e), (mode, r, e, dg.rank_for_error(want, e))
        if mode != "tokens":
            assert rng_ == pytest.approx(dg.sigma_range(want), rel=1e-3)
        else:
            # sigma_min of the token unfolding sits near the bottom of the spectrum: the
            # range is checked against the bracket the eigenvalue tolerance allows
            lo = np.sqrt(want[0] / (want[-1] + tol * want[0]))
            assert rng_ >= lo * (1 - 1e-6)

"""GPU parity of the truncated feature spectra (the exact ST-HOSVD tau of section 4's
eq. (2)) against the fp64 oracle, through the C-ABI.

jolt_truncated_spectra returns, for every cell and every grid token rank r, the
eigenvalues mu(r) of the feature Gram of the cell truncated to r token directions.  The
oracle computes the same rows from its own token factor (exact eigenvectors, or its own
FlashJoLT run with the same Philox sketch).

Inputs are exactly low rank (before the cache dtype's rounding) with distinct singular
values, so every grid projector is either well determined (below the rank, where the
spectral gaps are large) or irrelevant (at and above the rank, where F_Y(r) = F; only the
rounding noise of the cache dtype lives there).  Tolerance: |d mu| <= 2e-5 E per entry --
the fp32 products, fp32 block Grams with fp64 running sums and the fp32 tridiagonalisation
of a d x d matrix each add O(d u_32) of ||F|| <= E, and the rounding noise holds far less
than that of E.

At the full Mistral-shaped size (16 cells, T = 4096, exact) the oracle cannot form every
row, so the test checks what holds at any size: trace(F_Y(r)) equals the captured token
mass sum_{i < r} lambda_T,i, the last row (r = T) is the feature spectrum, the rows grow
with r (Weyl) and never exceed the feature spectrum, and the resulting tau lies between
the two mode-tail bounds.
"""
import os

import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from conftest import lowrank_cell
from gpu_util import compress, ctx, decompress, device_cells, note
from oracle import alloc as oalloc, pipeline as opl, tucker as otk

pytestmark = pytest.mark.gpu

FLASH = dict(method=J.JOLT_FLASH, q=24, ratio=2.0, oversample=8, power_iters=1)


def _trunc(xs, desc, step, n_r, opts=None, seeds=None):
    nb = J.jolt_truncated_spectra_workspace_size(desc, len(xs), step, n_r, opts)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    note("jolt_truncated_spectra", len(xs), "cells T", desc.T, "d", desc.d, "step", step, "n_r", n_r)
    mu = J.jolt_truncated_spectra(ctx(), desc, xs, step, n_r, seeds=seeds, opts=opts, ws=ws)
    torch.cuda.synchronize()
    return mu, ws


def _cells(rng, n, m, T, d, rank):
    out = []
    for i in range(n):
        x = lowrank_cell(rng, m, T, d, rank, decay=0.7 + 0.3 * i)
        out.append(x / np.sqrt(np.mean(x * x)))
    return out


@pytest.mark.parametrize("dtype,m,T,d,step", [
    ("f32", 4, 200, 64, 8),      # ragged: the last grid point (200) is not a tile multiple
    ("bf16", 8, 256, 128, 16),
    ("bf16", 3, 96, 32, 4),
])
def test_exact_truncated_spectra_match_oracle(dtype, m, T, d, step):
    rng = np.random.default_rng(11)
    xs, exact, desc = device_cells(_cells(rng, 2, m, T, d, 10), dtype)
    n_r = T // step
    mu, _ = _trunc(xs, desc, step, n_r)
    rs = [step * (k + 1) for k in range(n_r)]
    for c, X in enumerate(exact):
        _, U_T = otk.token_spectrum_exact(X)
        want = otk.truncated_feature_spectra(X, U_T, rs)
        E = otk.energy(X)
        np.testing.assert_allclose(mu[c], want, rtol=0, atol=2e-5 * E)


def test_flash_truncated_spectra_match_oracle():
    rng = np.random.default_rng(12)
    xs, exact, desc = device_cells(_cells(rng, 2, 4, 160, 64, 8), "bf16")
    seeds = [5, 9]
    step = 4
    n_r = 24 // step
    mu, _ = _trunc(xs, desc, step, n_r, opts=FLASH, seeds=seeds)
    for c, X in enumerate(exact):
        sp = opl.spectrum(X, method="flash", q=24, p=8, power_iters=1, seed=seeds[c])
        want = otk.truncated_feature_spectra(X, sp["U_T"], [step * (k + 1) for k in range(n_r)])
        np.testing.assert_allclose(mu[c], want, rtol=0, atol=2e-5 * otk.energy(X))


def test_reused_spectrum_gives_the_same_rows():
    """opts.reuse = 1 takes the token spectrum jolt_spectrum left in the same workspace:
    the rows are bit-identical to those of a call that computes it."""
    rng = np.random.default_rng(13)
    xs, exact, desc = device_cells(_cells(rng, 3, 4, 128, 64, 6), "bf16")
    mu0, ws = _trunc(xs, desc, 8, 16)
    J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    mu1 = J.jolt_truncated_spectra(ctx(), desc, xs, 8, 16, opts=dict(method=J.JOLT_EXACT, reuse=1), ws=ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(mu0, mu1)
    # a capped grid (n_r < rT_max / step) returns the leading rows
    mu2, _ = _trunc(xs, desc, 8, 5)
    np.testing.assert_allclose(mu2, mu0[:, :5], rtol=0, atol=1e-6 * mu0.max())


def test_allocation_on_gpu_rows_lands_on_its_model_error():
    """Joint allocation from the GPU's exact tau with residual bits off: the compressed
    cells' measured relative errors equal their modelled tau (up to the fp16 rounding of
    the stored factors), and the oracle allocator fed the same rows agrees bit for bit."""
    rng = np.random.default_rng(14)
    cells = [x + 0.02 * rng.standard_normal(x.shape) for x in _cells(rng, 4, 8, 256, 64, 12)]
    xs, exact, desc = device_cells(cells, "bf16")
    step = 8
    n_r = 256 // step
    mu, ws = _trunc(xs, desc, step, n_r)
    E, LT, LD = J.jolt_spectrum(ctx(), desc, xs, None, None, ws)
    torch.cuda.synchronize()
    specs = [dict(m=8, T=256, d=64, c=2, g=64, E=float(E[i]), lam_T=LT[i], lam_d=LD[i], rT_max=256,
                  mu=mu[i]) for i in range(4)]
    eps2 = {0: 1.0, 2: 0.26, 4: 0.0101, 8: 3.5e-5}
    budget = sum(x.size for x in cells) * 2 / 4.0
    got = J.jolt_allocate(specs, budget, eps2, bits=(0,), step=step)
    ocells = [oalloc.CellSpectrum(m=8, T=256, d=64, c=2, g=64, E=s["E"], lam_T=s["lam_T"], lam_d=s["lam_d"],
                                  rT_max=256, mu=s["mu"]) for s in specs]
    ref = oalloc.allocate(ocells, budget, eps2, bits=(0,), step=step)
    assert got["alloc"] == [tuple(a) for a in ref["alloc"]]
    params = [J.Params(rT, rd, 0, 64, J.JOLT_FACTOR_F16, 0, i) for i, (rT, rd, _) in enumerate(got["alloc"])]
    blobs, _ = compress(xs, desc, params)
    outs = decompress(blobs, desc)
    for i, (rT, rd, _) in enumerate(got["alloc"]):
        tab = oalloc.st_tau_table(float(E[i]), mu[i])
        model = 1.0 if rT == 0 else tab[rT // step - 1][rd]
        meas = float(np.sum((exact[i] - outs[i]) ** 2)) / float(E[i])
        assert meas == pytest.approx(model, abs=2e-3), (i, rT, rd)


def test_mistral_shaped_full_cache_properties():
    """16 cells of the Mistral-shaped T = 4096 cache (exact method), r_T every 64 tokens."""
    cfg = dict(kvsynth.CONFIGS["mistral7b_gqa_T4096"])
    gl = cfg.pop("group_layers")
    note("generate mistral7b_gqa_T4096")
    K, V = kvsynth.make_cache(**cfg, workers=min(16, os.cpu_count() or 1))
    L, B, H, T, d = K.shape
    Kd = torch.from_numpy(K.view(np.int16)).view(torch.bfloat16).cuda()
    Vd = torch.from_numpy(V.view(np.int16)).view(torch.bfloat16).cuda()
    desc = J.cell_desc(dtype=J.JOLT_BF16, n_layers=gl, n_heads=H, T=T, d=d, stride_layer=B * H * T * d,
                       stride_head=T * d, stride_token=d)
    ptrs = []
    for X in (Kd, Vd):
        for g in range(L // gl):
            ptrs.append(X.data_ptr() + (g * gl * B * H) * T * d * 2)
    step, n_r = 64, T // 64
    ws = torch.empty(J.jolt_truncated_spectra_workspace_size(desc, len(ptrs), step, n_r), dtype=torch.uint8,
                     device="cuda")
    note("jolt_spectrum", len(ptrs), "cells")
    E, LT, LD = J.jolt_spectrum(ctx(), desc, ptrs, None, None, ws)
    note("jolt_truncated_spectra (reused spectrum)", step, n_r)
    mu = J.jolt_truncated_spectra(ctx(), desc, ptrs, step, n_r, opts=dict(method=J.JOLT_EXACT, reuse=1), ws=ws)
    torch.cuda.synchronize()
    for c in range(len(ptrs)):
        e = float(E[c])
        head = np.cumsum(LT[c])
        for k in range(n_r):
            r = step * (k + 1)
            assert abs(mu[c, k].sum() - head[r - 1]) <= 2e-4 * e, (c, r)
        np.testing.assert_allclose(mu[c, -1], LD[c], rtol=0, atol=2e-5 * e)
        assert (np.diff(mu[c], axis=0) >= -2e-5 * e).all()
        assert (mu[c] <= LD[c][None, :] + 2e-5 * e).all()
        tab = oalloc.st_tau_table(e, mu[c])
        tauT = otk.tail_fractions(LT[c], e)
        taud = otk.tail_fractions(LD[c], e)
        for k in range(n_r):
            r = step * (k + 1)
            for rd in range(8, d + 1, 8):
                assert tab[k][rd] >= max(tauT[r], taud[rd]) - 3e-4
                assert tab[k][rd] <= min(1.0, tauT[r] + taud[rd]) + 3e-4

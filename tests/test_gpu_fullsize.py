"""GPU parity at the workloads' full per-cell sizes, through the whole-cache runtime.

Every test runs ``CacheCodec`` -- the launch configuration bench.py times: one
library call per chunk of up to 16 cells, spectrum -> host allocation ->
compress -> decompress -- on a seeded synthetic cache, then checks what the fp64
oracle can compute at that size one cell (or one token row) at a time, and
properties that hold at any size:

* spectra of a sampled cell (energy, token and feature eigenvalues; FlashJoLT
  Ritz values and tail from the oracle run with the GPU's own sketch) within
  1e-3 of the largest eigenvalue (bf16 caches);
* the oracle's allocator fed the GPU spectra returns the same allocation;
* quantiser codes stage-wise (the oracle's rotation and quantiser applied to
  the GPU's exported X~) equal except <= 1e-4 of entries, each off by <= 1;
* X~ equals the oracle's reconstruction from the blob's stored factors;
* the decoder reproduces the oracle's decode of the same blob;
* backbone and end-to-end relative errors within 1e-3 relative of the
  oracle's at the same ranks and bits;
* blobs within the byte budget; per-layer errors finite.

Workloads (synthetic stand-ins for the paper's Mistral-7B and LLaMA-2-13B caches):
the Mistral-shaped T = 4096 cache in full (16 cells, exact, 2x); the T = 32768 cache
restricted to its first layer group (2 of its 16 cells, each at full size; FlashJoLT,
2x); the T = 131072 long-context group in full (2 cells, FlashJoLT, 3x; its Ritz values
and tail against the oracle run with the GPU's sketch over the whole cell, the codec
checks on sampled token rows); the LLaMA-shaped MHA cache restricted to its first layer
group and two batch items (4 of its 64 cells, m = 200, each at full size; exact and
FlashJoLT, each at 2x and 3x).
"""
import gc
import os

import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from gpu_util import note
from oracle import alloc as oalloc, pipeline as opl, tucker as otk
from oracle.philox import rotation_signs
from oracle.residual import quantize, rotate

pytestmark = pytest.mark.gpu

TOL = 1e-3            # bf16 caches
WORKERS = min(16, os.cpu_count() or 1)
_CACHES = {}          # the last generated host cache (read only)


class Run:
    """A synthetic cache pushed through CacheCodec; host copies for the oracle."""

    def __init__(self, name, *, n_layers=None, batch=None, method, ratio):
        from paper_2607_12550_amd.cache import CacheCodec
        cfg = dict(kvsynth.CONFIGS[name])
        self.gl = cfg.pop("group_layers")
        if n_layers is not None:
            cfg["n_layers"] = n_layers
        if batch is not None:
            cfg["batch"] = batch
        self.cfg = cfg
        note("generate", name, {k: cfg[k] for k in ("n_layers", "n_heads", "T", "batch")})
        key = (name, cfg["n_layers"], cfg["batch"])
        if key not in _CACHES:             # the same cells serve several budgets / methods
            _CACHES.clear()
            _CACHES[key] = kvsynth.make_cache(**cfg, workers=WORKERS)
        self.K_np, self.V_np = _CACHES[key]
        to_dev = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        self.K, self.V = to_dev(self.K_np), to_dev(self.V_np)
        note("codec", name, method, ratio)
        self.codec = c = CacheCodec(self.K, self.V, group_layers=self.gl, method=method, ratio=ratio)
        self.eps2 = c.calibrate()
        c.spectrum()
        self.alloc = c.allocate()
        c.compress()
        self.Kout, self.Vout = torch.empty_like(self.K), torch.empty_like(self.V)
        c.decompress(self.Kout, self.Vout)
        torch.cuda.synchronize()
        self.H, self.T, self.d = cfg["n_heads"], cfg["T"], cfg["d"]
        self.m = self.gl * self.H

    def close(self):
        self.codec.close()
        del self.K, self.V, self.Kout, self.Vout, self.codec
        gc.collect()
        torch.cuda.empty_cache()

    # ---- per-cell views
    def index(self, tensor, group, batch=0):
        for i, c in enumerate(self.codec.cells):
            if (c.tensor, c.group, c.batch) == (tensor, group, batch):
                return i
        raise KeyError((tensor, group, batch))

    def cell_x(self, i):
        c = self.codec.cells[i]
        src = (self.K_np, self.V_np)[c.tensor][c.group * self.gl:(c.group + 1) * self.gl, c.batch]
        return kvsynth.bf16_bits_to_f32(src).reshape(self.m, self.T, self.d).astype(np.float64)

    def cell_out(self, i):
        c = self.codec.cells[i]
        out = (self.Kout, self.Vout)[c.tensor][c.group * self.gl:(c.group + 1) * self.gl, c.batch]
        return out.float().cpu().numpy().reshape(self.m, self.T, self.d).astype(np.float64)

    def blob(self, i):
        c = self.codec
        off = c.blob_ptrs[i] - c.arena.data_ptr()
        return c.arena[off:off + c.blob_sizes[i]].cpu().numpy().tobytes()

    def export(self, what, i, shape, dtype=torch.float32):
        """Intermediate of the last compress call (the last chunk of cells)."""
        c = self.codec
        last0 = (len(c.cells) - 1) // c.chunk * c.chunk
        assert i >= last0, "only the last chunk's intermediates are exported"
        t = torch.empty(shape, dtype=dtype, device="cuda")
        J.jolt_debug_export(c.ctx, what, i - last0, t)
        torch.cuda.synchronize()
        return t

    def decode_f32(self, i):
        """The GPU decoder on blob i alone, fp32 output (no bf16 output rounding)."""
        c = self.codec
        od = J.cell_desc(dtype=J.JOLT_F32, n_layers=self.gl, n_heads=self.H, T=self.T, d=self.d,
                         stride_layer=self.H * self.T * self.d, stride_head=self.T * self.d,
                         stride_token=self.d)
        out = torch.empty((self.m, self.T, self.d), dtype=torch.float32, device="cuda")
        J.jolt_decompress(c.ctx, [c.blob_ptrs[i]], od, [out], c.dec_ws, blob_bytes=[c.blob_sizes[i]],
                          ws_bytes=c.dec_ws.numel())
        torch.cuda.synchronize()
        return out.cpu().numpy().astype(np.float64)


def code_mismatch(a, b):
    diff = np.abs(a.astype(np.int16) - b.astype(np.int16))
    return float(np.mean(diff != 0)), int(diff.max()) if diff.size else 0


def check_bf16_decode(Xh, want, X):
    """bf16 decoder output vs the oracle's decode of the same blob rounded to bf16: equal
    except where the fp32 sum X~ + r^ lands on the other side of a bf16 rounding boundary
    (one bf16 unit, 2^-7 relative at most) or, where X~ and r^ cancel, within the fp32
    error of the two terms (absolute, 1e-5 of the cell's RMS)."""
    diff = np.abs(Xh - want)
    assert np.mean(diff != 0) < 1e-3
    slack = diff - np.abs(want) * 2 ** -7
    rms = float(np.sqrt(np.mean(X * X)))
    assert slack.max() <= 1e-5 * rms, (float(slack.max()), rms)


def check_allocation(run):
    """P-alloc: the oracle allocator on the GPU spectra gives the same allocation."""
    E, LT, LD = run.codec.spectra
    fb = run.codec.fbytes
    cells = [oalloc.CellSpectrum(m=run.m, T=run.T, d=run.d, c=fb, g=run.codec.group, E=float(E[i]),
                                 lam_T=LT[i], lam_d=LD[i], rT_max=run.codec.rT_max)
             for i in range(len(run.codec.cells))]
    budget = run.codec.cache_bytes / run.codec.ratio
    ref = oalloc.allocate(cells, budget, run.eps2, bits=run.codec.bits)
    got = [(p.r_T, p.r_d, p.bits) for p in run.codec.params]
    assert got == [tuple(a) for a in ref["alloc"]]
    assert ref["total_bytes"] <= budget
    # blobs: eq. (1) payload plus one header and section alignment per blob
    slack = len(got) * (opl.HEADER_BYTES + 6 * opl.ALIGN)
    assert run.codec.compressed_bytes() <= budget + slack
    return got


def check_cell_codec(run, i, *, method, q=0, spec=None):
    """Stage-wise codes, closed-loop X~, decode of the blob, errors vs the oracle, one cell."""
    X = run.cell_x(i)
    p = run.codec.params[i]
    seed = run.codec.seeds[i]
    got = opl.read_blob(run.blob(i))
    assert (got["m"], got["T"], got["d"], got["r_T"], got["r_d"], got["bits"]) == \
        (run.m, run.T, run.d, p.r_T, p.r_d, p.bits)
    Xt = run.export(2, i, (run.m, run.T, run.d)).cpu().numpy().astype(np.float64)
    nX = np.linalg.norm(X)
    # closed loop: the GPU's X~ is the reconstruction of its own stored factors
    Xt_blob = opl.decode_parts_from_factors(got["U_hat"], got["Ud_hat"], got["G_hat"], got["gexp"],
                                            None, None, T=run.T, d=run.d, bits=0, group=p.group,
                                            seed=seed)
    assert np.linalg.norm(Xt - Xt_blob) <= 1e-5 * nX
    if p.bits:
        codes_ref, scales_ref = quantize(rotate(X - Xt, rotation_signs(seed, run.d)), p.bits, p.group)
        frac, mx = code_mismatch(got["codes"], codes_ref)
        assert frac <= 1e-4 and mx <= 1, (i, frac, mx)
        np.testing.assert_allclose(got["scales"], scales_ref, rtol=2e-3)
        del codes_ref, scales_ref
    # decoder: the cache output equals the oracle's decode of the same blob, cast to bf16
    want = opl.cast_output(opl.decode_parts_from_factors(
        got["U_hat"], got["Ud_hat"], got["G_hat"], got["gexp"], got.get("codes"), got.get("scales"),
        T=run.T, d=run.d, bits=p.bits, group=p.group, seed=seed), "bf16")
    Xh = run.cell_out(i)
    check_bf16_decode(Xh, want, X)
    del want, Xh, Xt_blob
    # errors against the oracle compressing the same cell at the same ranks and bits
    ref = opl.compress_cell(X, r_T=p.r_T, r_d=p.r_d, bits=p.bits, group=p.group, seed=seed,
                            factor_bytes=run.codec.fbytes, spec=spec, method=method, q=q)
    eb_gpu, eb_ref = opl.rel_error(X, Xt), opl.rel_error(X, ref["Xtilde"])
    assert abs(eb_gpu / eb_ref - 1) < TOL, (i, eb_gpu, eb_ref)
    e_gpu, e_ref = opl.rel_error(X, run.decode_f32(i)), opl.rel_error(X, ref["Xhat"])
    assert abs(e_gpu / e_ref - 1) < TOL, (i, e_gpu, e_ref)
    note(f"cell {i}: ranks ({p.r_T}, {p.r_d}) b={p.bits}  backbone {eb_gpu:.6f} / {eb_ref:.6f}  "
         f"end-to-end {e_gpu:.6f} / {e_ref:.6f}")


def check_layer_errors(run, bound=0.05):
    from paper_2607_12550_amd.cache import layer_errors
    eK, eV = layer_errors(run.K, run.Kout), layer_errors(run.V, run.Vout)
    assert np.all(np.isfinite(eK)) and np.all(np.isfinite(eV))
    assert eK.max() < bound and eV.max() < bound, (eK.max(), eV.max())


# ------------------------------------------------------------------------------- workloads
def test_mistral7b_gqa_T4096_exact_full_cache():
    """32 L x 8 KV heads x T 4096 x 128, bf16: 16 cells (m = 32), exact spectrum, 2x."""
    run = Run("mistral7b_gqa_T4096", method="exact", ratio=2.0)
    try:
        check_allocation(run)
        check_layer_errors(run)
        E, LT, LD = run.codec.spectra
        i = run.index(1, 0)                                 # values of layer group 0
        X = run.cell_x(i)
        note("oracle exact spectrum, cell", i)
        sp = opl.spectrum(X)
        assert abs(E[i] / sp["E"] - 1) < 1e-10
        np.testing.assert_allclose(LT[i], sp["lam_T"], rtol=0, atol=TOL * sp["lam_T"][0])
        np.testing.assert_allclose(LD[i], sp["lam_d"], rtol=0, atol=TOL * sp["lam_d"][0])
        check_cell_codec(run, i, method="exact", spec=sp)
    finally:
        run.close()


def _flash_spectrum_parity(run, i, q):
    """Ritz values and tail of cell i vs the oracle run with the GPU's exported sketch."""
    E, LT, _ = run.codec.spectra
    X = run.cell_x(i)
    N, ell = run.m * run.d, run.codec.ell
    om = run.export(3, i, (N, ell), torch.bfloat16).float().cpu().numpy().astype(np.float64)
    note("oracle flash spectrum, cell", i, "l", ell)
    lam, U, extra = otk.token_spectrum_flash(X, q=q, p=10, power_iters=1, seed=run.codec.seeds[i],
                                             omega=om)
    assert abs(E[i] / otk.energy(X) - 1) < 1e-10
    np.testing.assert_allclose(LT[i, :q], lam[:q], rtol=0, atol=TOL * lam[0])
    assert abs(LT[i, q] - lam[q]) <= TOL * E[i]
    spec = dict(E=otk.energy(X), lam_T=lam, lam_d=otk.feature_spectrum(X)[0], U_T=U,
                rT_max=extra["q_eff"], extra=extra)
    return X, spec


def test_mistral7b_gqa_T32768_flash_full_cells():
    """Layer group 0 of the T = 32768 cache: 2 full cells (m = 32, N = 4096), q = 512,
    l = 522, one power iteration, 2x."""
    run = Run("mistral7b_gqa_T32768", n_layers=4, method="flash", ratio=2.0)
    try:
        assert run.codec.ell == 522
        check_allocation(run)
        check_layer_errors(run)
        i = run.index(1, 0)
        X, spec = _flash_spectrum_parity(run, i, 512)
        np.testing.assert_allclose(run.codec.spectra[2][i], spec["lam_d"], rtol=0,
                                   atol=TOL * spec["lam_d"][0])
        del X
        check_cell_codec(run, i, method="flash", q=512, spec=spec)
    finally:
        run.close()


@pytest.mark.parametrize("ratio", [2.0, 3.0])
def test_llama2_13b_mha_T4096_exact(ratio):
    """Layer group 0 (5 layers x 40 heads, m = 200, N = 25600) of two batch items, exact, at
    the workload's 2x and 3x budgets."""
    run = Run("llama2_13b_mha_T4096_b4", n_layers=5, batch=2, method="exact", ratio=ratio)
    try:
        assert len(run.codec.cells) == 4
        check_allocation(run)
        check_layer_errors(run)
        E, LT, LD = run.codec.spectra
        i = run.index(0, 0, 1)                              # keys of batch item 1: strided cell
        X = run.cell_x(i)
        note("oracle exact spectrum, cell", i)
        sp = opl.spectrum(X)
        assert abs(E[i] / sp["E"] - 1) < 1e-10
        np.testing.assert_allclose(LT[i], sp["lam_T"], rtol=0, atol=TOL * sp["lam_T"][0])
        np.testing.assert_allclose(LD[i], sp["lam_d"], rtol=0, atol=TOL * sp["lam_d"][0])
        check_cell_codec(run, i, method="exact", spec=sp)
    finally:
        run.close()


@pytest.mark.parametrize("ratio", [2.0, 3.0])
def test_llama2_13b_mha_T4096_flash(ratio):
    """Same cells, FlashJoLT (q = 128, l = 138), at 2x and 3x."""
    run = Run("llama2_13b_mha_T4096_b4", n_layers=5, batch=2, method="flash", ratio=ratio)
    try:
        assert run.codec.ell == 138
        check_allocation(run)
        check_layer_errors(run)
        i = run.index(1, 0, 1)
        X, spec = _flash_spectrum_parity(run, i, 128)
        del X
        check_cell_codec(run, i, method="flash", q=128, spec=spec)
    finally:
        run.close()


def test_longctx_T131072_flash_3x_sampled():
    """4 L x 8 heads x T 131072 (2 cells, m = 32), FlashJoLT q = 512, 3x: checks one token
    row or one direction at a time (the cells are too large for the whole-cell oracle)."""
    run = Run("longctx_4L8h_T131072", method="flash", ratio=3.0)
    try:
        check_allocation(run)
        check_layer_errors(run)
        E, LT, LD = run.codec.spectra
        q = run.codec.rT_max
        assert q == 512 and np.isclose(LT[:, :q + 1].sum(axis=1), E, rtol=1e-9).all()
        i = run.index(1, 0)
        # Ritz values and tail of the whole cell against the oracle run with the GPU's sketch
        X, _ = _flash_spectrum_parity(run, i, q)
        assert abs(E[i] / otk.energy(X) - 1) < 1e-10
        mu, _ = otk.feature_spectrum(X)
        np.testing.assert_allclose(LD[i], mu, rtol=0, atol=TOL * mu[0])
        p = run.codec.params[i]
        assert p.r_T > 0
        # each kept direction u_k of the stored U_T is a Ritz vector: ||X_(2)^T u_k||^2 = lam_k
        U = run.export(0, i, (run.T, p.r_T)).cpu().numpy().astype(np.float64)
        for k in sorted({0, 1, p.r_T // 2, p.r_T - 1}):
            rq = sum(float(np.sum((X[s].T @ U[:, k]) ** 2)) for s in range(run.m))
            assert abs(rq - LT[i, k]) <= TOL * LT[i, 0], (k, rq, LT[i, k])
        # ST-HOSVD bound by discarded mode energy (Ritz spectrum incl. the tail, feature spectrum)
        tau_T = otk.tail_fractions(LT[i], E[i])[p.r_T]
        tau_d = otk.tail_fractions(LD[i], E[i])[p.r_d]
        Xt = run.export(2, i, (run.m, run.T, run.d)).cpu().numpy()
        err2 = sum(float(np.sum((X[s] - Xt[s]) ** 2)) for s in range(run.m))
        assert err2 <= (tau_T + tau_d + 1e-5) * E[i], (err2 / E[i], tau_T, tau_d)
        # sampled token rows: X~ from the stored factors, codes, decode
        got = opl.read_blob(run.blob(i))
        rows = np.sort(np.random.default_rng(0).choice(run.T, 256, replace=False))
        Xs, Xts = X[:, rows], Xt[:, rows].astype(np.float64)
        del X, Xt
        Xt_blob = opl.decode_parts_from_factors(got["U_hat"][rows], got["Ud_hat"], got["G_hat"],
                                                got["gexp"], None, None, T=len(rows), d=run.d,
                                                bits=0, group=p.group, seed=run.codec.seeds[i])
        assert np.linalg.norm(Xts - Xt_blob) <= 1e-5 * np.linalg.norm(Xs)
        codes = got["codes"][:, rows] if p.bits else None
        scales = got["scales"][:, rows] if p.bits else None
        if p.bits:
            cref, sref = quantize(rotate(Xs - Xts, rotation_signs(run.codec.seeds[i], run.d)), p.bits, p.group)
            frac, mx = code_mismatch(codes, cref)
            assert frac <= 1e-4 and mx <= 1, (frac, mx)
            np.testing.assert_allclose(scales, sref, rtol=2e-3)
        want = opl.cast_output(opl.decode_parts_from_factors(
            got["U_hat"][rows], got["Ud_hat"], got["G_hat"], got["gexp"], codes, scales,
            T=len(rows), d=run.d, bits=p.bits, group=p.group, seed=run.codec.seeds[i]), "bf16")
        check_bf16_decode(run.cell_out(i)[:, rows], want, Xs)
    finally:
        run.close()

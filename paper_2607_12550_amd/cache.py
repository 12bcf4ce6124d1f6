"""Whole-cache runtime over the C-ABI: cell planning, buffers and the budgeted pipeline.

A KV cache is two tensors ``[L][B][H][T][d]`` (keys, values) resident on the GPU.
Section 4 of the paper cuts the L layers into contiguous groups and compresses
keys and values of every group separately; here every (group, K/V, batch item)
is one cell, read in place through a strided descriptor.  This module only
marshals pointers, sizes buffers and sequences the library calls:
``jolt_spectrum`` for every cell (and ``jolt_truncated_spectra`` when eq. (2)'s tau is
taken exactly), ``jolt_allocate`` under the global byte budget
B = cache bytes / R (eq. (3)), ``jolt_compress`` into one blob arena, and
``jolt_decompress`` back into caller-provided tensors.  The compression method
itself runs entirely inside libjolt.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from . import (JOLT_BF16, JOLT_EXACT, JOLT_F32, JOLT_FACTOR_F16, JOLT_FACTOR_F32, JOLT_FLASH,
               HEADER_BYTES, Params, SpectrumOpts, cell_desc, jolt_allocate, jolt_compress,
               jolt_compressed_size, jolt_create, jolt_decompress, jolt_destroy,
               jolt_decompress_workspace_size, jolt_eps2_calibrate, jolt_eps2_workspace_size, jolt_q_cap,
               jolt_spectrum, jolt_spectrum_len, jolt_truncated_spectra,
               jolt_truncated_spectra_workspace_size, jolt_workspace_size)


@dataclass
class CellRef:
    tensor: int        # 0 = keys, 1 = values
    group: int
    batch: int
    ptr: int           # device address of element (layer0 of group, batch, head 0, t 0, f 0)


@dataclass
class Plan:
    cells: list
    desc: object
    n_heads: int
    group_layers: int
    cache_bytes: int
    params: list = field(default_factory=list)
    offsets: list = field(default_factory=list)
    sizes: list = field(default_factory=list)


class CacheCodec:
    """Budgeted compression of a KV cache held as two [L][B][H][T][d] tensors."""

    def __init__(self, K: torch.Tensor, V: torch.Tensor, *, group_layers: int,
                 method: str = "exact", ratio: float = 2.0, q: int = 0, oversample: int = 10,
                 power_iters: int = 1, group: int = 64, bits=(0, 2, 4, 8), step: int = 8,
                 count_scale_bytes: bool = True, seed: int = 0, max_cells_per_call: int = 16, r_max: int = 0,
                 workspace_cap_bytes: int = 0, device: int = 0, tau: str = "bound",
                 tau_rT_cap: int | None = None):
        assert K.shape == V.shape and K.dtype == V.dtype and K.is_cuda and K.is_contiguous()
        L, B, H, T, d = K.shape
        if L % group_layers:
            raise ValueError("the number of layers must be a multiple of group_layers")
        self.K, self.V = K, V
        self.shape = (L, B, H, T, d)
        self.dtype = JOLT_BF16 if K.dtype == torch.bfloat16 else JOLT_F32
        esz = K.element_size()
        self.group_layers, self.ratio, self.group, self.bits, self.step = group_layers, ratio, group, bits, step
        self.count_scale_bytes = count_scale_bytes
        self.method = JOLT_FLASH if method == "flash" else JOLT_EXACT
        self.opts = SpectrumOpts(self.method, q, float(ratio), oversample, power_iters, 0, r_max)
        # compress takes each chunk's spectrum from the workspace its spectrum call filled
        self.reuse_opts = SpectrumOpts(self.method, q, float(ratio), oversample, power_iters, 1, r_max)
        self.factor_dtype = JOLT_FACTOR_F16 if self.dtype == JOLT_BF16 else JOLT_FACTOR_F32
        self.fbytes = 2 if self.factor_dtype == JOLT_FACTOR_F16 else 4
        self.desc = cell_desc(dtype=self.dtype, n_layers=group_layers, n_heads=H, T=T, d=d,
                              stride_layer=B * H * T * d, stride_head=T * d, stride_token=d)
        self.cells = []
        for t, X in enumerate((K, V)):
            for g in range(L // group_layers):
                for b in range(B):
                    off = ((g * group_layers * B + b) * H) * T * d
                    self.cells.append(CellRef(t, g, b, X.data_ptr() + off * esz))
        self.seeds = [seed + i for i in range(len(self.cells))]
        self.cache_bytes = 2 * K.numel() * esz
        self.chunk = max(1, min(max_cells_per_call, len(self.cells)))
        self.ctx = jolt_create(device)
        self.n_lam, self.rT_max = jolt_spectrum_len(self.desc, self.opts)
        # one workspace per chunk of cells when they fit under the cap, so that compress
        # reuses every chunk's spectrum; otherwise one shared workspace (spectra recomputed)
        n_chunks = (len(self.cells) + self.chunk - 1) // self.chunk
        # eq. (2)'s tau: the additive mode-tail bound, or the exact ST-HOSVD value from the
        # truncated feature spectra on the r_T grid up to a cap: tau_rT_cap tokens, or (None)
        # one chosen per allocation -- 4x the largest r_T the bound's allocation takes (at
        # least 256), doubled while the exact allocation reaches it
        if tau not in ("bound", "exact"):
            raise ValueError("tau must be 'bound' or 'exact'")
        self.tau = tau
        self.tau_auto = tau == "exact" and tau_rT_cap is None
        nr_max = self.rT_max // step
        self.tau_nr = (nr_max if self.tau_auto else min(self.rT_max, tau_rT_cap) // step) if tau == "exact" else 0
        if tau == "exact" and self.tau_nr < 1:
            raise ValueError("the r_T grid holds no point below the cap")
        self.mu = None
        self.tau_cap_used = 0
        ws_bytes = jolt_workspace_size(self.desc, self.chunk, self.opts) if tau == "bound" else \
            jolt_truncated_spectra_workspace_size(self.desc, self.chunk, step, self.tau_nr, self.opts)
        if not workspace_cap_bytes:      # default: half of the device's memory
            workspace_cap_bytes = torch.cuda.get_device_properties(K.device).total_memory // 2
        n_ws = n_chunks if n_chunks * ws_bytes <= workspace_cap_bytes else 1
        self.ws_list = [torch.empty(ws_bytes, dtype=torch.uint8, device=K.device) for _ in range(n_ws)]
        self.ws = self.ws_list[0]
        # decode workspace: sized for the largest r_T of each allocation (set_params)
        self.dec_ws = torch.empty(jolt_decompress_workspace_size(self.desc, self.chunk, 0),
                                  dtype=torch.uint8, device=K.device)
        # FlashJoLT sketch width l = min(q + p, T, m d) (section 5); 0 for the exact path
        qq = q or (jolt_q_cap(T, ratio) if self.method == JOLT_FLASH else 0)
        self.ell = min(qq + oversample, T, group_layers * H * d) if self.method == JOLT_FLASH else 0
        self.eps2 = None
        # blob arena: at most the whole budget plus per-blob headers and alignment
        arena = int(self.cache_bytes / ratio) + len(self.cells) * (HEADER_BYTES + 8 * 256) + (1 << 20)
        self.arena = torch.zeros(arena, dtype=torch.uint8, device=K.device)
        self.params = None
        self.spectra_fresh = False
        self.blob_ptrs = None
        self.blob_sizes = None
        self.hdr = None
        self.spectra = None

    def close(self):
        if self.ctx:
            jolt_destroy(self.ctx)
            self.ctx = None

    def _chunks(self):
        for i in range(0, len(self.cells), self.chunk):
            yield i, self.cells[i:i + self.chunk]

    def _ws(self, i):
        return self.ws_list[(i // self.chunk) % len(self.ws_list)]

    def calibrate(self, n_samples: int = 1 << 20, seed: int = 0):
        d = self.shape[4]
        ws = torch.empty(jolt_eps2_workspace_size(d, n_samples), dtype=torch.uint8, device=self.K.device)
        self.eps2 = jolt_eps2_calibrate(self.ctx, self.group, d, seed, n_samples, ws)
        return self.eps2

    def spectrum(self, stream=None):
        E, LT, LD = [], [], []
        for i, cs in self._chunks():
            e, lt, ld = jolt_spectrum(self.ctx, self.desc, [c.ptr for c in cs], self.seeds[i:i + len(cs)],
                                      self.opts, self._ws(i), stream=stream)
            E.append(e); LT.append(lt); LD.append(ld)
        self.spectra = (np.concatenate(E), np.concatenate(LT), np.concatenate(LD))
        self.mu = None
        if self.tau == "exact" and not self.tau_auto:
            self.truncated_spectra(self.tau_nr, stream)
        self.spectra_fresh = True
        return self.spectra

    def truncated_spectra(self, n_r: int, stream=None):
        """mu of every cell on the r_T grid step .. n_r step; each chunk's token spectrum is
        taken from its workspace when every chunk has its own (recomputed otherwise)."""
        own = len(self.ws_list) * self.chunk >= len(self.cells) and self.spectra_fresh
        MU = []
        for i, cs in self._chunks():
            MU.append(jolt_truncated_spectra(self.ctx, self.desc, [c.ptr for c in cs], self.step, n_r,
                                             seeds=self.seeds[i:i + len(cs)],
                                             opts=self.reuse_opts if own else self.opts, ws=self._ws(i),
                                             stream=stream))
        self.mu = np.concatenate(MU)
        self.tau_cap_used = n_r * self.step
        return self.mu

    def allocate(self, budget_bytes=None, strategy: str = "joint"):
        """Ranks and bits of every cell under the byte budget: the joint Lagrangian dual, or
        one of the ablation allocators ("greedy", "rank_only", "uniform"; the greedy one
        spends the keys' and the values' shares separately)."""
        E, LT, LD = self.spectra
        L, B, H, T, d = self.shape
        m = self.group_layers * H
        cells = [dict(m=m, T=T, d=d, c=self.fbytes, g=self.group, E=float(E[i]), lam_T=LT[i],
                      lam_d=LD[i], rT_max=self.rT_max, pool=self.cells[i].tensor)
                 for i in range(len(self.cells))]
        if self.mu is not None:
            for i, c in enumerate(cells):
                c["mu"] = self.mu[i]
        budget = self.cache_bytes / self.ratio if budget_bytes is None else budget_bytes

        def run(cs):
            return jolt_allocate(cs, budget, self.eps2, bits=self.bits, step=self.step,
                                 count_scale_bytes=self.count_scale_bytes, strategy=strategy)

        if self.tau_auto:
            top = max(r for r, _, _ in run([{k: v for k, v in c.items() if k != "mu"} for c in cells])["alloc"])
            n_r = min(self.tau_nr, max(256, 4 * top) // self.step)
            while True:
                self.truncated_spectra(n_r)
                for i, c in enumerate(cells):
                    c["mu"] = self.mu[i]
                res = run(cells)
                if n_r >= self.tau_nr or max(r for r, _, _ in res["alloc"]) < n_r * self.step:
                    break
                n_r = min(self.tau_nr, 2 * n_r)
        else:
            res = run(cells)
        self.set_params([Params(rT, rd, b, self.group, self.factor_dtype, 0, s)
                         for (rT, rd, b), s in zip(res["alloc"], self.seeds)])
        return res

    def set_params(self, params):
        self.params = params
        need = jolt_decompress_workspace_size(self.desc, self.chunk, max(p.r_T for p in params))
        if need > self.dec_ws.numel():
            self.dec_ws = None
            self.dec_ws = torch.empty(need, dtype=torch.uint8, device=self.K.device)
        sizes = [jolt_compressed_size(self.desc, p) for p in params]
        offs, pos = [], 0
        for s in sizes:
            offs.append(pos)
            pos += (s + 255) // 256 * 256
        if pos > self.arena.numel():
            self.arena = torch.zeros(pos, dtype=torch.uint8, device=self.K.device)
        base = self.arena.data_ptr()
        self.blob_ptrs = [base + o for o in offs]
        self.blob_sizes = sizes

    def compress(self, stream=None):
        for i, cs in self._chunks():
            n = len(cs)
            ws = self._ws(i)
            reuse = len(self.ws_list) * self.chunk >= len(self.cells) and self.spectra_fresh
            jolt_compress(self.ctx, self.desc, [c.ptr for c in cs], self.params[i:i + n],
                          self.reuse_opts if reuse else self.opts,
                          ws, self.blob_ptrs[i:i + n], ws_bytes=ws.numel(),
                          blob_bytes=self.blob_sizes[i:i + n], stream=stream)

    def headers(self):
        """Host copy of every blob header (lets decompress skip the device->host read)."""
        out = np.zeros((len(self.cells), HEADER_BYTES), np.uint8)
        for i, p in enumerate(self.blob_ptrs):
            t = torch.empty(HEADER_BYTES, dtype=torch.uint8)
            src = self.arena[p - self.arena.data_ptr():p - self.arena.data_ptr() + HEADER_BYTES]
            t.copy_(src)
            out[i] = t.numpy()
        self.hdr = out
        return out

    def decompress(self, Kout: torch.Tensor, Vout: torch.Tensor, stream=None):
        L, B, H, T, d = self.shape
        out_dtype = JOLT_BF16 if Kout.dtype == torch.bfloat16 else JOLT_F32
        od = cell_desc(dtype=out_dtype, n_layers=self.group_layers, n_heads=H, T=T, d=d,
                       stride_layer=B * H * T * d, stride_head=T * d, stride_token=d)
        esz = Kout.element_size()
        outs = []
        for c in self.cells:
            off = ((c.group * self.group_layers * B + c.batch) * H) * T * d
            outs.append((Kout, Vout)[c.tensor].data_ptr() + off * esz)
        for i, cs in self._chunks():
            n = len(cs)
            hdr = self.hdr[i:i + n] if self.hdr is not None else None
            jolt_decompress(self.ctx, self.blob_ptrs[i:i + n], od, outs[i:i + n], self.dec_ws, hdr_host=hdr,
                            blob_bytes=self.blob_sizes[i:i + n], ws_bytes=self.dec_ws.numel(), stream=stream)

    def compressed_bytes(self) -> int:
        return int(sum(self.blob_sizes))

    def payload_bytes(self, with_scales: bool = True) -> int:
        """Eq. (1) bytes of the chosen allocation (factors + codes [+ scales])."""
        L, B, H, T, d = self.shape
        m = self.group_layers * H
        tot = 0
        for p in self.params:
            s = (m * p.r_T * p.r_d + T * p.r_T + d * p.r_d) * self.fbytes
            if p.bits:
                s += p.bits * m * T * d // 8 + (2 * (m * T * d // p.group) if with_scales else 0)
            tot += s
        return tot


def layer_errors(X: torch.Tensor, Xh: torch.Tensor) -> np.ndarray:
    """Relative Frobenius error per layer of a [L][B][H][T][d] cache."""
    L = X.shape[0]
    out = np.zeros(L)
    for l in range(L):
        a = X[l].float()
        b = Xh[l].float()
        out[l] = float(torch.linalg.vector_norm(a - b) / torch.linalg.vector_norm(a))
    return out

"""Seeded synthetic KV-cache generator.

This module produces the *inputs* that both the GPU library and the fp64
oracle consume.  It contains none of the compression method's arithmetic:
only the data recipe below (a low-rank-plus-noise model of a KV cache with
outlier feature channels) and an fp32 -> bf16 cast for the stored tensor.

Recipe for one (batch item b, layer l, tensor t in {K, V}):

* token factor ``A`` (T x r): AR(1) rows, ``a_0 ~ N(0, I)``,
  ``a_t = rho * a_{t-1} + sqrt(1 - rho^2) * eps_t``; shared by every head of
  the layer;
* core ``C_h`` (r x r): iid N(0, 1), one per head;
* feature factor ``F`` (d x r): orthonormal columns of QR(N(0,1)^{d x r})
  scaled by ``i^-alpha`` (i = 1..r); shared across heads and batch items;
* ``X_h = A C_h F^T + N(0, noise^2)``;
* ``n_out`` feature channels (drawn per layer and tensor, shared across heads
  and batch) are then multiplied by ``out_scale``;
* stored as bf16 (round to nearest even) or kept as fp32.

Every draw comes from its own ``numpy.random.Generator(PCG64)`` keyed by a
``SeedSequence`` over (data_seed, role, b, l, t[, h]) so any layer can be
regenerated alone.
"""
from __future__ import annotations

import numpy as np

__all__ = ["layer_kv", "make_cache", "f32_to_bf16_bits", "bf16_bits_to_f32",
           "apply_rope", "CONFIGS"]

_ROLE_A, _ROLE_C, _ROLE_F, _ROLE_N, _ROLE_O, _ROLE_ALPHA = 1, 2, 3, 4, 5, 6
_THREAD_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    u = x32.view(np.uint32)
    # u + 0x7FFF + lsb stays below 2^32 for every non-NaN pattern; NaNs are replaced below
    with np.errstate(over="ignore"):
        r = (u >> 16) & np.uint32(1)
        r += np.uint32(0x7FFF)
        r += u
        r >>= 16
    out = r.astype(np.uint16)
    nan = np.isnan(x32)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _ar1(rng: np.random.Generator, T: int, r: int, rho: float) -> np.ndarray:
    from scipy.signal import lfilter
    eps = rng.standard_normal((T, r))
    x = eps.copy()
    x[1:] *= np.sqrt(1.0 - rho * rho)
    return lfilter([1.0], [1.0, -rho], x, axis=0)


def layer_kv(*, layer: int, tensor: int, n_heads: int, T: int, d: int,
             batch: int = 1, alpha: float, n_out: int = 2, out_scale: float = 10.0,
             noise: float = 0.05, rho: float = 0.9, rank: int = 32,
             data_seed: int = 0) -> np.ndarray:
    """One layer's K (tensor=0) or V (tensor=1) cache, fp32, shape [batch][n_heads][T][d]."""
    if rank > d:
        raise ValueError("rank must not exceed d")
    rf = _rng(data_seed, _ROLE_F, layer, tensor)
    q, _ = np.linalg.qr(rf.standard_normal((d, rank)))
    F = q * (np.arange(1, rank + 1, dtype=np.float64) ** (-alpha))[None, :]
    ro = _rng(data_seed, _ROLE_O, layer, tensor)
    chans = ro.choice(d, size=n_out, replace=False) if n_out > 0 else np.zeros(0, int)
    out = np.empty((batch, n_heads, T, d), dtype=np.float32)
    for b in range(batch):
        A = _ar1(_rng(data_seed, _ROLE_A, b, layer, tensor), T, rank, rho)
        for h in range(n_heads):
            C = _rng(data_seed, _ROLE_C, b, layer, tensor, h).standard_normal((rank, rank))
            x = (A @ C) @ F.T
            x += noise * _rng(data_seed, _ROLE_N, b, layer, tensor, h).standard_normal((T, d))
            if n_out:
                x[:, chans] *= out_scale
            out[b, h] = x
    return out


def layer_alpha(layer: int, tensor: int, lo: float, hi: float, data_seed: int = 0) -> float:
    """Per-layer spectral decay drawn uniformly from [lo, hi]."""
    return float(_rng(data_seed, _ROLE_ALPHA, layer, tensor).uniform(lo, hi))


def make_cache(*, n_layers: int, n_heads: int, T: int, d: int, batch: int = 1,
               alpha_K=1.5, alpha_V=0.7, n_out: int = 2, out_scale: float = 10.0,
               noise: float = 0.05, dtype: str = "bf16", data_seed: int = 0,
               layers=None, workers: int = 1):
    """Whole cache as two arrays [L][batch][n_heads][T][d].

    ``alpha_K`` / ``alpha_V`` are floats or (lo, hi) ranges for a per-layer
    draw.  ``dtype='bf16'`` returns uint16 bf16 bit patterns, ``'f32'`` returns
    float32.  ``layers`` restricts generation to a subset of layer indices.
    ``workers > 1`` generates the (layer, K/V) slabs in that many processes; the
    values do not depend on it.
    """
    layers = list(range(n_layers)) if layers is None else list(layers)
    shape = (len(layers), batch, n_heads, T, d)
    np_dt = np.uint16 if dtype == "bf16" else np.float32
    K = np.empty(shape, dtype=np_dt)
    V = np.empty(shape, dtype=np_dt)
    jobs = []
    for i, l in enumerate(layers):
        for t, a in enumerate((alpha_K, alpha_V)):
            alpha = layer_alpha(l, t, *a, data_seed=data_seed) if isinstance(a, tuple) else a
            jobs.append((i, t, dict(layer=l, tensor=t, n_heads=n_heads, T=T, d=d, batch=batch,
                                    alpha=alpha, n_out=n_out, out_scale=out_scale, noise=noise,
                                    data_seed=data_seed, bf16=dtype == "bf16")))
    if workers > 1 and len(jobs) > 1:
        import concurrent.futures as cf
        import multiprocessing as mp
        import os
        # one BLAS thread per worker process: the workers already occupy the cores, and
        # nested BLAS threads only oversubscribe them (the values do not depend on it)
        saved = {k: os.environ.get(k) for k in _THREAD_VARS}
        os.environ.update({k: "1" for k in _THREAD_VARS})
        try:
            with cf.ProcessPoolExecutor(max_workers=min(workers, len(jobs)),
                                        mp_context=mp.get_context("spawn")) as ex:
                results = ex.map(_layer_job, [j[2] for j in jobs])
                for (i, t, _), x in zip(jobs, results):
                    (K, V)[t][i] = x
        finally:
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
    else:
        for i, t, kw in jobs:
            (K, V)[t][i] = _layer_job(kw)
    return K, V


def _layer_job(kw):
    kw = dict(kw)
    bf16 = kw.pop("bf16")
    x = layer_kv(**kw)
    return f32_to_bf16_bits(x) if bf16 else x


def apply_rope(x: np.ndarray, base: float) -> np.ndarray:
    """Post-RoPE variant of a key tensor [..., T, d] (fp32): the rotary position
    embedding of the Mistral / LLaMA checkpoints (feature pairs (j, j + d/2) of token t
    turned by t * base^(-2 j / d)), computed in fp64 and returned as fp32.  Used to build
    the post-RoPE inputs of appendix B's comparison; it is part of the model, not of the
    compression method."""
    T, d = x.shape[-2], x.shape[-1]
    h = d // 2
    w = base ** (-2.0 * np.arange(h) / d)
    ang = np.arange(T, dtype=np.float64)[:, None] * w[None, :]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty(x.shape, dtype=np.float32)
    flat_in = x.reshape(-1, T, d)
    flat_out = out.reshape(-1, T, d)
    for i in range(flat_in.shape[0]):
        a = flat_in[i].astype(np.float64)
        x1, x2 = a[:, :h], a[:, h:]
        flat_out[i, :, :h] = x1 * c - x2 * s
        flat_out[i, :, h:] = x2 * c + x1 * s
    return out


# Workload shapes (synthetic stand-ins for the paper's Mistral-7B / LLaMA-2-13B caches).
CONFIGS = {
    "keys_fp32_8h_T256": dict(n_layers=1, n_heads=8, T=256, d=128, batch=1,
                              alpha_K=1.5, alpha_V=1.5, n_out=2, out_scale=10.0,
                              dtype="f32", group_layers=1),
    "mistral7b_gqa_T4096": dict(n_layers=32, n_heads=8, T=4096, d=128, batch=1,
                                alpha_K=1.5, alpha_V=0.7, n_out=2, out_scale=10.0,
                                dtype="bf16", group_layers=4),
    "mistral7b_gqa_T32768": dict(n_layers=32, n_heads=8, T=32768, d=128, batch=1,
                                 alpha_K=1.5, alpha_V=0.7, n_out=2, out_scale=10.0,
                                 dtype="bf16", group_layers=4),
    "llama2_13b_mha_T4096_b4": dict(n_layers=40, n_heads=40, T=4096, d=128, batch=4,
                                    alpha_K=(1.0, 1.8), alpha_V=(0.5, 0.9), n_out=2,
                                    out_scale=10.0, dtype="bf16", group_layers=5),
    "longctx_4L8h_T131072": dict(n_layers=4, n_heads=8, T=131072, d=128, batch=1,
                                 alpha_K=0.7, alpha_V=0.7, n_out=4, out_scale=20.0,
                                 dtype="bf16", group_layers=4),
}

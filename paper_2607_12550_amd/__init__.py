"""Python binding of ``libjolt`` (MI355X / gfx950 JoLT-FlashJoLT compression path).

Argument marshalling only: every step of the method runs in the library's HIP
kernels.  Functions keep the C-ABI names (``jolt_spectrum``, ``jolt_compress``,
``jolt_decompress``, ``jolt_allocate`` ...).  Device buffers are passed as torch
CUDA tensors (or raw integer device addresses); streams as ``torch.cuda.Stream``
or raw ``hipStream_t`` integers.  If the compiled library is missing, importing
this package raises: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os
import re

import numpy as np

__all__ = ["JoltError", "lib", "CellDesc", "SpectrumOpts", "Params", "CellSpectrum", "AllocOpts",
           "JOLT_F32", "JOLT_BF16", "JOLT_EXACT", "JOLT_FLASH", "JOLT_FACTOR_F32",
           "JOLT_FACTOR_F16", "Rope", "jolt_last_error", "jolt_create", "jolt_destroy", "jolt_q_cap",
           "jolt_spectrum_len", "jolt_workspace_size", "jolt_decompress_workspace_size", "jolt_spectrum", "jolt_compressed_size",
           "jolt_compress", "jolt_decompress", "jolt_allocate", "jolt_eps2_workspace_size",
           "jolt_eps2_calibrate", "jolt_slice_spectrum_workspace_size", "jolt_slice_spectrum",
           "jolt_mode_summary", "jolt_truncated_spectra_workspace_size", "jolt_truncated_spectra",
           "jolt_attend_workspace_size", "jolt_attend", "jolt_attend_noalloc", "JOLT_ATTEND_SCRATCH_BYTES", "jolt_debug_export", "jolt_debug_set",
           "jolt_profile_enable", "jolt_profile_reset", "JOLT_E_NONFINITE", "JOLT_E_NOCONV",
           "JOLT_DBG_INVIT_ITERS", "JOLT_DBG_TRD_LANES", "JOLT_DBG_TRD_TWO_STAGE", "JOLT_DBG_BULGE_SPIN",
           "jolt_profile_read", "STAGES", "cell_desc", "LIB_PATH", "HEADER_PATH"]

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libjolt.so")
HEADER_PATH = os.path.join(os.path.dirname(HERE), "include", "jolt.h")

JOLT_OK, JOLT_F32, JOLT_BF16 = 0, 0, 1
JOLT_E_INVAL, JOLT_E_UNSUPPORTED, JOLT_E_WORKSPACE, JOLT_E_BLOB = -1, -2, -3, -4
JOLT_E_HIP, JOLT_E_NONFINITE, JOLT_E_STATE, JOLT_E_NOCONV = -5, -6, -7, -8
JOLT_DBG_INVIT_ITERS = 0
JOLT_DBG_TRD_LANES = 1
JOLT_DBG_TRD_TWO_STAGE = 2
JOLT_DBG_BULGE_SPIN = 3
JOLT_ATTEND_SCRATCH_BYTES = 64 << 20
JOLT_EXACT, JOLT_FLASH = 0, 1
JOLT_FACTOR_F32, JOLT_FACTOR_F16 = 0, 1
HEADER_BYTES = 128


class JoltError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libjolt error {code}: {msg}")
        self.code = code


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2607_12550_amd/build.py` "
                      "(or __graft_entry__.build())")
# torch ships its own HIP runtime; loading it first makes the library bind to that same
# runtime instance (loaded the other way round, the library's first HIP call can find no
# device in a process where torch already uses the GPU)
import torch  # noqa: E402,F401

lib = C.CDLL(LIB_PATH)


class CellDesc(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("n_layers", C.c_int32), ("n_heads", C.c_int32),
                ("T", C.c_int32), ("d", C.c_int32), ("reserved", C.c_int32),
                ("stride_layer", C.c_int64), ("stride_head", C.c_int64),
                ("stride_token", C.c_int64)]


class SpectrumOpts(C.Structure):
    _fields_ = [("method", C.c_int32), ("q", C.c_int32), ("ratio", C.c_double),
                ("oversample", C.c_int32), ("power_iters", C.c_int32), ("reuse", C.c_int32),
                ("r_max", C.c_int32)]


class Params(C.Structure):
    _fields_ = [("r_T", C.c_int32), ("r_d", C.c_int32), ("bits", C.c_int32), ("group", C.c_int32),
                ("factor_dtype", C.c_int32), ("reserved", C.c_int32), ("seed", C.c_uint64)]


class CellSpectrum(C.Structure):
    _fields_ = [("m", C.c_int32), ("T", C.c_int32), ("d", C.c_int32), ("c", C.c_int32),
                ("g", C.c_int32), ("n_lam_T", C.c_int32), ("rT_max", C.c_int32),
                ("pool", C.c_int32), ("E", C.c_double),
                ("lam_T", C.POINTER(C.c_double)), ("lam_d", C.POINTER(C.c_double)),
                ("n_mu", C.c_int32), ("reserved", C.c_int32), ("mu", C.POINTER(C.c_double))]


class Rope(C.Structure):
    _fields_ = [("base", C.c_double), ("position_offset", C.c_int32), ("reserved", C.c_int32)]


class AllocOpts(C.Structure):
    _fields_ = [("budget_bytes", C.c_double), ("eps2", C.c_double * 4), ("bit_mask", C.c_int32),
                ("step", C.c_int32), ("floor_rT", C.c_int32), ("floor_rd", C.c_int32),
                ("floor_bits", C.c_int32), ("count_scale_bytes", C.c_int32), ("strategy", C.c_int32)]


_vp, _sz, _i32, _dbl = C.c_void_p, C.c_size_t, C.c_int32, C.c_double
_P = C.POINTER
_SIGS = {
    "jolt_last_error": (C.c_char_p, []),
    "jolt_create": (C.c_int, [_P(_vp), C.c_int]),
    "jolt_destroy": (C.c_int, [_vp]),
    "jolt_q_cap": (C.c_int, [C.c_int, _dbl]),
    "jolt_spectrum_len": (C.c_int, [_P(CellDesc), _P(SpectrumOpts), _P(_i32), _P(_i32)]),
    "jolt_workspace_size": (C.c_int, [_P(CellDesc), C.c_int, _P(SpectrumOpts), _P(_sz)]),
    "jolt_decompress_workspace_size": (C.c_int, [_P(CellDesc), C.c_int, C.c_int, _P(_sz)]),
    "jolt_spectrum": (C.c_int, [_vp, _P(CellDesc), C.c_int, _P(_vp), _P(C.c_uint64),
                                _P(SpectrumOpts), _vp, _sz, _P(_dbl), _P(_dbl), _P(_dbl), _vp]),
    "jolt_compressed_size": (C.c_int, [_P(CellDesc), _P(Params), _P(_sz)]),
    "jolt_compress": (C.c_int, [_vp, _P(CellDesc), C.c_int, _P(_vp), _P(Params),
                                _P(SpectrumOpts), _vp, _sz, _P(_vp), _P(_sz), _vp]),
    "jolt_decompress": (C.c_int, [_vp, C.c_int, _P(_vp), _P(_sz), _vp, _P(CellDesc), _P(_vp),
                                  _vp, _sz, _vp]),
    "jolt_decompress_rope": (C.c_int, [_vp, C.c_int, _P(_vp), _P(_sz), _vp, _P(CellDesc), _P(_vp),
                                       _P(Rope), _vp, _sz, _vp]),
    "jolt_allocate": (C.c_int, [_P(CellSpectrum), C.c_int, _P(AllocOpts), _P(_i32), _P(_i32),
                                _P(_i32), _P(_dbl), _P(_dbl), _P(_dbl), _P(_i32)]),
    "jolt_eps2_workspace_size": (C.c_int, [C.c_int, C.c_int, _P(_sz)]),
    "jolt_eps2_calibrate": (C.c_int, [_vp, C.c_int, C.c_int, C.c_uint64, C.c_int, _P(_dbl),
                                      _vp, _sz, _vp]),
    "jolt_slice_spectrum_workspace_size": (C.c_int, [_P(CellDesc), C.c_int, _P(_sz)]),
    "jolt_slice_spectrum": (C.c_int, [_vp, _P(CellDesc), C.c_int, _P(_vp), _vp, _sz, _P(_dbl), _vp]),
    "jolt_mode_summary": (C.c_int, [_P(_dbl), C.c_int, _dbl, _dbl, _P(_dbl), _P(_i32), _P(_i32)]),
    "jolt_attend_workspace_size": (C.c_int, [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, _P(_sz)]),
    "jolt_attend": (C.c_int, [_vp, C.c_int, _P(_vp), _P(_sz), _P(_vp), _P(_sz), _vp, _vp, _P(_i32),
                              C.c_int, _vp, C.c_float, _vp, _vp, _sz, _vp]),
    "jolt_truncated_spectra_workspace_size": (C.c_int, [_P(CellDesc), C.c_int, _P(SpectrumOpts),
                                                         C.c_int, C.c_int, _P(_sz)]),
    "jolt_truncated_spectra": (C.c_int, [_vp, _P(CellDesc), C.c_int, _P(_vp), _P(C.c_uint64),
                                         _P(SpectrumOpts), C.c_int, C.c_int, _vp, _sz, _P(_dbl), _vp]),
    "jolt_debug_export": (C.c_int, [_vp, C.c_int, C.c_int, _vp, _sz, _vp]),
    "jolt_debug_set": (C.c_int, [_vp, C.c_int, C.c_int64]),
    "jolt_attend_noalloc": (C.c_int, [_vp, C.c_int, _P(_vp), _P(_sz), _P(_vp), _P(_sz), _vp, _vp, _P(_i32),
                                      C.c_int, _vp, C.c_float, _vp, _vp]),
    "jolt_profile_enable": (C.c_int, [_vp, C.c_int]),
    "jolt_profile_reset": (C.c_int, [_vp]),
    "jolt_profile_read": (C.c_int, [_vp, C.c_int, _P(_dbl), _P(C.c_int64)]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype, _f.argtypes = _res, _args


def header_functions() -> list:
    """Names of the functions declared in include/jolt.h."""
    with open(HEADER_PATH) as f:
        src = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(jolt_\w+)\s*\(", src, re.M)))


def jolt_last_error() -> str:
    return lib.jolt_last_error().decode()


def _check(rc):
    if rc < 0:
        raise JoltError(rc, jolt_last_error())
    return rc


def _addr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s) -> int:
    if s is None:
        return 0
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _ptrs(xs):
    return (_vp * len(xs))(*[_addr(x) for x in xs])


def cell_desc(*, dtype, n_layers, n_heads, T, d, stride_layer, stride_head, stride_token) -> CellDesc:
    return CellDesc(dtype, n_layers, n_heads, T, d, 0, stride_layer, stride_head, stride_token)


def _opts(opts):
    if opts is None:
        return None
    if isinstance(opts, SpectrumOpts):
        return C.byref(opts)
    return C.byref(SpectrumOpts(**opts))


# ----------------------------------------------------------------------------- entry points
def jolt_create(device: int = 0) -> int:
    h = _vp()
    _check(lib.jolt_create(C.byref(h), device))
    return h.value


def jolt_destroy(ctx: int) -> None:
    _check(lib.jolt_destroy(ctx))


def jolt_q_cap(T: int, ratio: float) -> int:
    return _check(lib.jolt_q_cap(T, ratio))


def jolt_spectrum_len(desc: CellDesc, opts=None):
    n, r = _i32(), _i32()
    _check(lib.jolt_spectrum_len(C.byref(desc), _opts(opts), C.byref(n), C.byref(r)))
    return n.value, r.value


def jolt_workspace_size(desc: CellDesc, n_cells: int, opts=None) -> int:
    b = _sz()
    _check(lib.jolt_workspace_size(C.byref(desc), n_cells, _opts(opts), C.byref(b)))
    return b.value


def jolt_decompress_workspace_size(out_desc: CellDesc, n_cells: int, max_rT: int) -> int:
    b = _sz()
    _check(lib.jolt_decompress_workspace_size(C.byref(out_desc), n_cells, max_rT, C.byref(b)))
    return b.value


def jolt_spectrum(ctx, desc: CellDesc, X, seeds=None, opts=None, ws=None, ws_bytes=None,
                  stream=None):
    """Returns (E[n], lam_T[n, n_lam_T], lam_d[n, d]) as numpy float64 arrays."""
    n = len(X)
    n_lam, _ = jolt_spectrum_len(desc, opts)
    E = np.zeros(n)
    lam_T = np.zeros((n, n_lam))
    lam_d = np.zeros((n, desc.d))
    sd = (C.c_uint64 * n)(*seeds) if seeds is not None else None
    wsb = ws_bytes if ws_bytes is not None else (ws.numel() * ws.element_size())
    _check(lib.jolt_spectrum(ctx, C.byref(desc), n, _ptrs(X), sd, _opts(opts), _addr(ws), wsb,
                             E.ctypes.data_as(_P(_dbl)), lam_T.ctypes.data_as(_P(_dbl)),
                             lam_d.ctypes.data_as(_P(_dbl)), _stream(stream)))
    return E, lam_T, lam_d


def jolt_truncated_spectra_workspace_size(desc: CellDesc, n_cells: int, step: int, n_r: int,
                                          opts=None) -> int:
    b = _sz()
    _check(lib.jolt_truncated_spectra_workspace_size(C.byref(desc), n_cells, _opts(opts), step, n_r,
                                                     C.byref(b)))
    return b.value


def jolt_truncated_spectra(ctx, desc: CellDesc, X, step: int, n_r: int, seeds=None, opts=None,
                           ws=None, ws_bytes=None, stream=None) -> np.ndarray:
    """mu[n_cells, n_r, d] (float64): eigenvalues of the feature Gram of the cell truncated
    to r_T = (k + 1) step in the token mode, row k, descending."""
    n = len(X)
    mu = np.zeros((n, n_r, desc.d))
    sd = (C.c_uint64 * n)(*seeds) if seeds is not None else None
    wsb = ws_bytes if ws_bytes is not None else (ws.numel() * ws.element_size())
    _check(lib.jolt_truncated_spectra(ctx, C.byref(desc), n, _ptrs(X), sd, _opts(opts), step, n_r,
                                      _addr(ws), wsb, mu.ctypes.data_as(_P(_dbl)), _stream(stream)))
    return mu


def jolt_compressed_size(desc: CellDesc, params: Params) -> int:
    b = _sz()
    _check(lib.jolt_compressed_size(C.byref(desc), C.byref(params), C.byref(b)))
    return b.value


def jolt_compress(ctx, desc: CellDesc, X, params, opts=None, ws=None, blobs=None, ws_bytes=None,
                  blob_bytes=None, stream=None) -> None:
    n = len(X)
    parr = (Params * n)(*params)
    bb = blob_bytes if blob_bytes is not None else [b.numel() * b.element_size() for b in blobs]
    wsb = ws_bytes if ws_bytes is not None else (ws.numel() * ws.element_size())
    _check(lib.jolt_compress(ctx, C.byref(desc), n, _ptrs(X), parr, _opts(opts), _addr(ws), wsb,
                             _ptrs(blobs), (_sz * n)(*bb), _stream(stream)))


def jolt_decompress(ctx, blobs, out_desc: CellDesc, Xhat, ws=None, hdr_host=None,
                    blob_bytes=None, ws_bytes=None, stream=None, rope=None) -> None:
    """rope: None, or (base, position_offset) to re-apply the rotary embedding while decoding."""
    n = len(blobs)
    bb = blob_bytes if blob_bytes is not None else [b.numel() * b.element_size() for b in blobs]
    wsb = ws_bytes if ws_bytes is not None else (ws.numel() * ws.element_size())
    hdr = None
    if hdr_host is not None:
        hdr_host = np.ascontiguousarray(hdr_host, dtype=np.uint8)
        hdr = hdr_host.ctypes.data
    if rope is None:
        _check(lib.jolt_decompress(ctx, n, _ptrs(blobs), (_sz * n)(*bb), hdr, C.byref(out_desc),
                                   _ptrs(Xhat), _addr(ws), wsb, _stream(stream)))
    else:
        r = Rope(float(rope[0]), int(rope[1]), 0)
        _check(lib.jolt_decompress_rope(ctx, n, _ptrs(blobs), (_sz * n)(*bb), hdr, C.byref(out_desc),
                                        _ptrs(Xhat), C.byref(r), _addr(ws), wsb, _stream(stream)))


ALLOC_STRATEGIES = {"joint": 0, "greedy": 1, "rank_only": 2, "uniform": 3}


def jolt_allocate(cells, budget_bytes: float, eps2, *, bits=(0, 2, 4, 8), step: int = 8,
                  floors=(0, 0, 0), count_scale_bytes: bool = True, strategy: str = "joint") -> dict:
    """cells: dicts with m, T, d, c, g, E, lam_T, lam_d, rT_max (numpy arrays for lam_*),
    optionally pool (budget pool of the greedy allocator, default 0) and mu (n_mu x d
    truncated feature spectra at r_T = step, 2 step, ...: exact ST-HOSVD tau)."""
    n = len(cells)
    keep = []
    arr = (CellSpectrum * n)()
    for i, c in enumerate(cells):
        lt = np.ascontiguousarray(c["lam_T"], dtype=np.float64)
        ld = np.ascontiguousarray(c["lam_d"], dtype=np.float64)
        keep += [lt, ld]
        mu = c.get("mu")
        n_mu, mu_p = 0, None
        if mu is not None:
            mu = np.ascontiguousarray(mu, dtype=np.float64)
            if mu.ndim != 2 or mu.shape[1] != c["d"]:
                raise ValueError("mu must be n_mu x d")
            keep.append(mu)
            n_mu, mu_p = mu.shape[0], mu.ctypes.data_as(_P(_dbl))
        arr[i] = CellSpectrum(c["m"], c["T"], c["d"], c["c"], c["g"], len(lt), c["rT_max"],
                              int(c.get("pool", 0)), c["E"], lt.ctypes.data_as(_P(_dbl)),
                              ld.ctypes.data_as(_P(_dbl)), n_mu, 0, mu_p)
    mask = sum(1 << i for i, b in enumerate((0, 2, 4, 8)) if b in bits)
    e4 = (C.c_double * 4)(*[float(eps2[b]) for b in (0, 2, 4, 8)])
    o = AllocOpts(budget_bytes, e4, mask, step, floors[0], floors[1], floors[2],
                  1 if count_scale_bytes else 0, ALLOC_STRATEGIES[strategy])
    rT, rd, bb = (_i32 * n)(), (_i32 * n)(), (_i32 * n)()
    lam, tot, err, inf = _dbl(), _dbl(), _dbl(), _i32()
    _check(lib.jolt_allocate(arr, n, C.byref(o), rT, rd, bb, C.byref(lam), C.byref(tot),
                             C.byref(err), C.byref(inf)))
    return dict(alloc=[(rT[i], rd[i], bb[i]) for i in range(n)], lam=lam.value,
                total_bytes=tot.value, model_error=err.value, infeasible=bool(inf.value))


def jolt_eps2_workspace_size(d: int, n_samples: int) -> int:
    b = _sz()
    _check(lib.jolt_eps2_workspace_size(d, n_samples, C.byref(b)))
    return b.value


def jolt_eps2_calibrate(ctx, group: int, d: int, seed: int, n_samples: int, ws,
                        stream=None) -> dict:
    out = (C.c_double * 4)()
    _check(lib.jolt_eps2_calibrate(ctx, group, d, seed, n_samples, out, _addr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)))
    return {0: out[0], 2: out[1], 4: out[2], 8: out[3]}


STAGES = ["feature_gram", "token_gram", "tridiag_large", "reserved3", "reserved4", "tridiag_small", "eigvals",
          "eigvecs", "backtransform", "project", "core", "serialize", "reconstruct", "residual",
          "decode", "sketch", "orth", "slice_gram", "attend", "trunc_gram"]


def jolt_profile_enable(ctx, on: bool = True) -> None:
    _check(lib.jolt_profile_enable(ctx, 1 if on else 0))


def jolt_profile_reset(ctx) -> None:
    _check(lib.jolt_profile_reset(ctx))


def jolt_profile_read(ctx) -> dict:
    """{stage name: (total ms, launches)} accumulated since the last reset."""
    out = {}
    for i, name in enumerate(STAGES):
        ms, n = _dbl(), C.c_int64()
        _check(lib.jolt_profile_read(ctx, i, C.byref(ms), C.byref(n)))
        out[name] = (ms.value, n.value)
    return out


def jolt_slice_spectrum_workspace_size(desc: CellDesc, n_cells: int) -> int:
    n = _sz(0)
    _check(lib.jolt_slice_spectrum_workspace_size(C.byref(desc), n_cells, C.byref(n)))
    return n.value


def jolt_slice_spectrum(ctx, desc: CellDesc, X, ws, ws_bytes=None, stream=None) -> np.ndarray:
    """Slice-mode eigenvalues [n_cells, m] (descending) of each cell, as float64."""
    n = len(X)
    m = desc.n_layers * desc.n_heads
    lam = np.zeros((n, m))
    wsb = ws_bytes if ws_bytes is not None else (ws.numel() * ws.element_size())
    _check(lib.jolt_slice_spectrum(ctx, C.byref(desc), n, _ptrs(X), _addr(ws), wsb,
                                   lam.ctypes.data_as(_P(_dbl)), _stream(stream)))
    return lam


def jolt_mode_summary(lam, err_a: float = 0.10, err_b: float = 0.20):
    """(sigma_1 / sigma_min, rank at err_a, rank at err_b) of one mode spectrum."""
    lam = np.ascontiguousarray(lam, dtype=np.float64)
    rng, ra, rb = _dbl(0), _i32(0), _i32(0)
    _check(lib.jolt_mode_summary(lam.ctypes.data_as(_P(_dbl)), len(lam), err_a, err_b,
                                 C.byref(rng), C.byref(ra), C.byref(rb)))
    return rng.value, ra.value, rb.value


def jolt_attend_workspace_size(n_items: int, n_q: int, T: int, d: int, max_rT_k: int, max_rT_v: int) -> int:
    n = _sz(0)
    _check(lib.jolt_attend_workspace_size(n_items, n_q, T, d, max_rT_k, max_rT_v, C.byref(n)))
    return n.value


def jolt_attend(ctx, k_blobs, v_blobs, k_hdr, v_hdr, layers, Q, O, scale: float, ws, ws_bytes=None,
                stream=None, k_bytes=None, v_bytes=None) -> None:
    """Attention of Q [n_items, n_q, d] (device fp32) over the compressed cells; writes O.

    k_hdr / v_hdr: host uint8 arrays [n_items, 128] of the blob headers."""
    n = len(k_blobs)
    kb = k_bytes if k_bytes is not None else [b.numel() for b in k_blobs]
    vb = v_bytes if v_bytes is not None else [b.numel() for b in v_blobs]
    kh = np.ascontiguousarray(k_hdr, dtype=np.uint8)
    vh = np.ascontiguousarray(v_hdr, dtype=np.uint8)
    lay = (_i32 * n)(*layers)
    wsb = ws_bytes if ws_bytes is not None else (ws.numel() * ws.element_size())
    _check(lib.jolt_attend(ctx, n, _ptrs(k_blobs), (_sz * n)(*kb), _ptrs(v_blobs), (_sz * n)(*vb),
                           kh.ctypes.data, vh.ctypes.data, lay, Q.shape[1], _addr(Q), float(scale),
                           _addr(O), _addr(ws), wsb, _stream(stream)))


def jolt_attend_noalloc(ctx, k_blobs, v_blobs, k_hdr, v_hdr, layers, Q, O, scale: float, stream=None,
                        k_bytes=None, v_bytes=None) -> None:
    """jolt_attend on the library's fixed device scratch (no workspace argument)."""
    n = len(k_blobs)
    kb = k_bytes if k_bytes is not None else [b.numel() for b in k_blobs]
    vb = v_bytes if v_bytes is not None else [b.numel() for b in v_blobs]
    kh = np.ascontiguousarray(k_hdr, dtype=np.uint8)
    vh = np.ascontiguousarray(v_hdr, dtype=np.uint8)
    lay = (_i32 * n)(*layers)
    _check(lib.jolt_attend_noalloc(ctx, n, _ptrs(k_blobs), (_sz * n)(*kb), _ptrs(v_blobs), (_sz * n)(*vb),
                                   kh.ctypes.data, vh.ctypes.data, lay, Q.shape[1], _addr(Q), float(scale),
                                   _addr(O), _stream(stream)))


def jolt_debug_export(ctx, what: int, cell: int, dst, stream=None) -> None:
    _check(lib.jolt_debug_export(ctx, what, cell, _addr(dst), dst.numel() * dst.element_size(),
                                 _stream(stream)))


def jolt_debug_set(ctx, what: int, value: int) -> None:
    _check(lib.jolt_debug_set(ctx, what, value))

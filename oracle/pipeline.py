"""One cell end to end, the blob byte format, and budgeted cache compression (fp64 oracle).

Steps for one cell X (m x T x d), following sections 4 and 5 of the paper:

1. spectrum: energy E, token-mode spectrum (exact or FlashJoLT), feature-mode
   spectrum;
2. ST-HOSVD truncation at (r_T, r_d) and serialisation of the factors;
3. reconstruction X~ from the stored factors;
4. residual R = X - X~ (against the decoder's X~: the "closed loop" reading),
   rotated, quantised at b bits and packed;
5. decode: X^ = X~ + unrotate(dequantise(codes)).

Budgeted mode (eq. (3)): the spectra of every (layer group, K/V[, batch item])
cell feed one Lagrangian allocation under a global byte budget, then each cell
is compressed at its allocated (r_T, r_d, b).

Blob byte format (little-endian; shared by definition with the GPU library,
written here independently):

* 128-byte header: b"JOLT", u32 version = 1, u32 in_dtype (0 fp32, 1 bf16),
  u32 factor_dtype (0 fp32, 1 fp16), u32 m, T, d, r_T, r_d, bits, group,
  method (0 exact, 1 flash), u64 seed, u64 offsets of U_T, U_d, G, exponents,
  scales, codes, u64 total bytes, u32 n_heads, zero padding;
* sections, each starting on a 256-byte boundary: U_T (T x r_T row-major),
  U_d (d x r_d row-major), G (m x r_T x r_d, slice s scaled by 2^-e_s), one
  int8 exponent e_s per slice, fp16 scales (one per quantiser group, order
  (slice, token, group)), packed codes (order (slice, token, feature)).
"""
from __future__ import annotations

import struct

import numpy as np

from . import tucker as tk
from .alloc import CellSpectrum, allocate, q_cap
from .philox import rotation_signs
from .residual import dequantize, pack, quantize, rotate, unpack, unrotate
from .rounding import bf16_bits, fp16_bits, to_bf16

HEADER_BYTES = 128
ALIGN = 256
MAGIC = b"JOLT"
METHOD_EXACT, METHOD_FLASH = 0, 1


def _align(x: int) -> int:
    return (x + ALIGN - 1) // ALIGN * ALIGN


def blob_layout(m, T, d, r_T, r_d, bits, group, factor_bytes):
    """Section offsets and total size of a blob."""
    off = {}
    pos = _align(HEADER_BYTES)
    for name, size in (("UT", T * r_T * factor_bytes), ("Ud", d * r_d * factor_bytes),
                       ("G", m * r_T * r_d * factor_bytes), ("gexp", m),
                       ("scales", 2 * (m * T * d // group) if bits else 0),
                       ("codes", (m * T * d * bits) // 8)):
        off[name] = pos
        pos = _align(pos + size) if name != "codes" else pos + size
    off["total"] = pos
    return off


def spectrum(X: np.ndarray, *, method: str = "exact", R: float = 2.0, q: int = 0,
             p: int = 10, power_iters: int = 1, seed: int = 0) -> dict:
    """Energy and mode spectra of one cell (section 4; section 5 for 'flash')."""
    m, T, d = X.shape
    E = tk.energy(X)
    lam_d, _ = tk.feature_spectrum(X)
    if method == "exact":
        lam_T, U_T = tk.token_spectrum_exact(X)
        rT_max = min(T, m * d)
        extra = {}
    elif method == "flash":
        qq = q if q > 0 else q_cap(T, R)
        lam_T, U_T, extra = tk.token_spectrum_flash(X, q=qq, p=p, power_iters=power_iters,
                                                    seed=seed)
        rT_max = extra["q_eff"]
    else:
        raise ValueError(method)
    return dict(E=E, lam_T=lam_T, lam_d=lam_d, U_T=U_T, rT_max=rT_max, extra=extra)


def compress_cell(X: np.ndarray, *, r_T: int, r_d: int, bits: int, group: int = 64,
                  seed: int = 0, factor_bytes: int = 2, spec: dict | None = None,
                  method: str = "exact", R: float = 2.0, q: int = 0, p: int = 10,
                  power_iters: int = 1) -> dict:
    """Compress one cell at fixed (r_T, r_d, b); returns every intermediate."""
    m, T, d = X.shape
    if spec is None:
        spec = spectrum(X, method=method, R=R, q=q, p=p, power_iters=power_iters, seed=seed)
    if r_T > spec["rT_max"] or r_d > d:
        raise ValueError("rank exceeds the admissible maximum")
    U, U_d, G, mu_Y = tk.st_hosvd(X, spec["U_T"], r_T, r_d)
    U_hat, Ud_hat, G_hat, gexp = tk.serialize(U, U_d, G, factor_bytes)
    Xt = tk.reconstruct(U_hat, Ud_hat, G_hat, gexp, T, d)
    signs = rotation_signs(seed, d)
    out = dict(spec=spec, U=U, U_d=U_d, G=G, mu_Y=mu_Y, U_hat=U_hat, Ud_hat=Ud_hat,
               G_hat=G_hat, gexp=gexp, Xtilde=Xt, signs=signs, r_T=r_T, r_d=r_d,
               bits=bits, group=group, seed=seed, factor_bytes=factor_bytes,
               method=method)
    if bits:
        Rp = rotate(X - Xt, signs)
        codes, scales = quantize(Rp, bits, group)
        out.update(Rrot=Rp, codes=codes, scales=scales)
    out["Xhat"] = decode(out)
    return out


def decode(parts: dict) -> np.ndarray:
    """X^ = X~ + s * H_d(dequantised codes) / sqrt(d) (section 4: decoding inverts the rotation)."""
    Xt = parts["Xtilde"]
    if not parts["bits"]:
        return Xt.copy()
    rp = dequantize(parts["codes"], parts["scales"], parts["bits"], parts["group"])
    return Xt + unrotate(rp, parts["signs"])


def decode_parts_from_factors(U_hat, Ud_hat, G_hat, gexp, codes, scales, *, T, d, bits,
                              group, seed):
    Xt = tk.reconstruct(U_hat, Ud_hat, G_hat, gexp, T, d)
    parts = dict(Xtilde=Xt, bits=bits, group=group, codes=codes, scales=scales,
                 signs=rotation_signs(seed, d))
    return decode(parts)


# ----------------------------------------------------------------------------- blob I/O
def write_blob(parts: dict, *, in_dtype: str, n_heads: int) -> bytes:
    Xt = parts["Xtilde"]
    m, T, d = Xt.shape
    r_T, r_d, bits, group = parts["r_T"], parts["r_d"], parts["bits"], parts["group"]
    fb = parts["factor_bytes"]
    lay = blob_layout(m, T, d, r_T, r_d, bits, group, fb)
    buf = bytearray(lay["total"])
    hdr = struct.pack("<4s11I Q 7Q I", MAGIC, 1, 1 if in_dtype == "bf16" else 0,
                      1 if fb == 2 else 0, m, T, d, r_T, r_d, bits, group,
                      METHOD_FLASH if parts["method"] == "flash" else METHOD_EXACT,
                      parts["seed"], lay["UT"], lay["Ud"], lay["G"], lay["gexp"],
                      lay["scales"], lay["codes"], lay["total"], n_heads)
    buf[:len(hdr)] = hdr

    def put(name, arr):
        b = arr.tobytes()
        buf[lay[name]:lay[name] + len(b)] = b

    if fb == 2:
        put("UT", fp16_bits(parts["U_hat"]))
        put("Ud", fp16_bits(parts["Ud_hat"]))
        put("G", fp16_bits(parts["G_hat"]))
    else:
        put("UT", parts["U_hat"].astype(np.float32))
        put("Ud", parts["Ud_hat"].astype(np.float32))
        put("G", parts["G_hat"].astype(np.float32))
    put("gexp", parts["gexp"].astype(np.int8))
    if bits:
        put("scales", fp16_bits(parts["scales"]))
        put("codes", pack(parts["codes"], bits))
    return bytes(buf)


def read_blob(blob: bytes) -> dict:
    f = struct.unpack_from("<4s11I Q 7Q I", blob, 0)
    if f[0] != MAGIC or f[1] != 1:
        raise ValueError("not a version-1 blob")
    (_, _, in_dt, fdt, m, T, d, r_T, r_d, bits, group, method, seed,
     oUT, oUd, oG, oE, oS, oC, total, n_heads) = f
    fb = 2 if fdt == 1 else 4

    def get(off, n, dt):
        return np.frombuffer(blob, dtype=dt, count=n, offset=off)

    if fb == 2:
        def fac(off, n):
            return get(off, n, np.float16).astype(np.float64)
    else:
        def fac(off, n):
            return get(off, n, np.float32).astype(np.float64)
    U_hat = fac(oUT, T * r_T).reshape(T, r_T)
    Ud_hat = fac(oUd, d * r_d).reshape(d, r_d)
    G_hat = fac(oG, m * r_T * r_d).reshape(m, r_T, r_d)
    gexp = get(oE, m, np.int8).astype(np.int64)
    out = dict(in_dtype="bf16" if in_dt == 1 else "f32", factor_bytes=fb, m=m, T=T, d=d,
               r_T=r_T, r_d=r_d, bits=bits, group=group, seed=seed, n_heads=n_heads,
               method="flash" if method == METHOD_FLASH else "exact", total=total,
               U_hat=U_hat, Ud_hat=Ud_hat, G_hat=G_hat, gexp=gexp)
    if bits:
        n = m * T * d
        out["scales"] = get(oS, n // group, np.float16).astype(np.float64).reshape(
            m, T, d // group)
        out["codes"] = unpack(get(oC, n * bits // 8, np.uint8), bits, n).reshape(m, T, d)
    return out


def decode_blob(blob: bytes) -> np.ndarray:
    b = read_blob(blob)
    return decode_parts_from_factors(b["U_hat"], b["Ud_hat"], b["G_hat"], b["gexp"],
                                     b.get("codes"), b.get("scales"), T=b["T"], d=b["d"],
                                     bits=b["bits"], group=b["group"], seed=b["seed"])


# ----------------------------------------------------------------------------- metrics
def rel_error(X: np.ndarray, Xhat: np.ndarray) -> float:
    den = float(np.sqrt(np.sum(X * X)))
    return float(np.sqrt(np.sum((X - Xhat) ** 2))) / den if den > 0 else 0.0


def per_layer_rel_error(X: np.ndarray, Xhat: np.ndarray, n_heads: int) -> list:
    m = X.shape[0]
    return [rel_error(X[l * n_heads:(l + 1) * n_heads], Xhat[l * n_heads:(l + 1) * n_heads])
            for l in range(m // n_heads)]


def cast_output(Xhat: np.ndarray, out_dtype: str) -> np.ndarray:
    return to_bf16(Xhat) if out_dtype == "bf16" else Xhat.astype(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------- budget mode
def compress_cells(cells, *, ratio: float, eps2: dict, method: str = "exact",
                   in_bytes: int = 2, group: int = 64, seeds=None, bits=(0, 2, 4, 8),
                   q: int = 0, p: int = 10, power_iters: int = 1, step: int = 8,
                   count_scales: bool = True, factor_bytes: int | None = None,
                   tau: str = "bound"):
    """Budgeted compression of a list of cells X (each m x T x d) at ``ratio``.

    Budget B = (cache bytes) / ratio with cache bytes = sum of m T d * in_bytes.
    tau = "bound" models the truncation error by the additive mode-tail bound,
    "exact" by the truncated feature spectra at every grid r_T (exact ST-HOSVD).
    Returns dict(specs, allocation, parts per cell).
    """
    fb = factor_bytes if factor_bytes is not None else (2 if in_bytes == 2 else 4)
    seeds = list(range(len(cells))) if seeds is None else list(seeds)
    specs, cs = [], []
    for X, sd in zip(cells, seeds):
        sp = spectrum(X, method=method, R=ratio, q=q, p=p, power_iters=power_iters, seed=sd)
        specs.append(sp)
        m, T, d = X.shape
        mu = None
        if tau == "exact":
            mu = tk.truncated_feature_spectra(X, sp["U_T"], list(range(step, sp["rT_max"] + 1, step)))
        elif tau != "bound":
            raise ValueError(tau)
        cs.append(CellSpectrum(m=m, T=T, d=d, c=fb, g=group, E=sp["E"], lam_T=sp["lam_T"],
                               lam_d=sp["lam_d"], rT_max=sp["rT_max"], mu=mu))
    total_in = float(sum(X.size for X in cells) * in_bytes)
    res = allocate(cs, total_in / ratio, eps2, bits=bits, step=step,
                   count_scales=count_scales)
    parts = []
    for X, sp, sd, (rT, rd, b) in zip(cells, specs, seeds, res["alloc"]):
        parts.append(compress_cell(X, r_T=rT, r_d=rd, bits=b, group=group, seed=sd,
                                   factor_bytes=fb, spec=sp, method=method))
    return dict(specs=specs, cells=cs, allocation=res, parts=parts, budget=total_in / ratio)

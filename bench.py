#!/usr/bin/env python3
"""Benchmark: KV-cache compression + decompression throughput on one MI355X.

Workload (default): a LLaMA-2-13B-shaped MHA cache, bf16 keys and values, 40 layers x
40 heads x T 4096 x d 128, batch 4 (13.4 GB), cut into layer groups of 5 -> 64 cells
(8 groups x K/V x 4 batch items, m = 200 slices each), all cells in one library call.
Exact token-mode spectrum, ranks and residual bits chosen by the Lagrangian dual at a
2x byte budget, 2/4/8-bit residual grid, group 64.  Synthetic data (seeded low-rank
AR(1) token factors, Gaussian cores, per-layer feature-spectrum decays, 2 outlier
channels x10, N(0, 0.05^2) noise); no model weights are involved.

One step = the whole path over the cache: spectrum of every cell, allocation,
compression into blobs, decompression back to a bf16 cache.  value = cache bytes x
steps / wall time of the timed steps (GB/s, 1 GB = 1e9 B), inputs resident in HBM.

Also reported: compress-only and decompress-only rates, mean relative Frobenius error
over layers for K and V, achieved ratio, per-stage device times from the library's
event instrumentation (one extra step), per-pass and whole-path roofline fractions on
the algorithmic bytes and flops of the design, FlashJoLT on the same cache and budget
(exact / FlashJoLT compression-time ratio), and the fp64 oracle timed on a bounded
sample of cells on the host CPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_GBS = 8000.0          # MI355X HBM3E peak, GB/s
# method and byte budget each synthetic workload is run at (section 6 set-ups)
WORKLOAD_RUN = {
    "keys_fp32_8h_T256": ("exact", 2.0),
    "mistral7b_gqa_T4096": ("exact", 2.0),
    "mistral7b_gqa_T32768": ("flash", 2.0),
    "llama2_13b_mha_T4096_b4": ("exact", 2.0),
    "longctx_4L8h_T131072": ("flash", 3.0),
}
MFMA_TF = {"fp32": 157.3, "bf16": 2500.0, "fp16": 2500.0, "fp64": 78.6}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llama2_13b_mha_T4096_b4")
    ap.add_argument("--cells-per-call", type=int, default=64,
                    help="cells batched into one library call (each call has its own workspace)")
    ap.add_argument("--compare-steps", type=int, default=3,
                    help="timed compress passes of FlashJoLT on the same cache after an exact run "
                         "(0 = skip the comparison)")
    ap.add_argument("--ratio", type=float, default=0.0, help="0 = the workload's budget")
    ap.add_argument("--method", default="", choices=["", "exact", "flash"],
                    help="empty = the workload's method")
    ap.add_argument("--allocator", default="joint", choices=["joint", "greedy", "rank_only", "uniform"],
                    help="allocation strategy (the joint dual, or an ablation allocator)")
    ap.add_argument("--tau", default="bound", choices=["bound", "exact"],
                    help="eq. (2)'s truncation error: the additive mode-tail bound, or the exact "
                         "ST-HOSVD value from the truncated feature spectra (one extra pass per step)")
    ap.add_argument("--rope-post", type=float, default=0.0,
                    help="> 1: compress post-RoPE keys (rotary base given) instead of pre-RoPE "
                         "ones, for the appendix-B comparison")
    ap.add_argument("--power-iters", type=int, default=1)
    ap.add_argument("--oversample", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gen-workers", type=int, default=16,
                    help="processes generating the synthetic cache (1 = in this process, e.g. under a "
                         "hardware-counter profiler; the values do not depend on it)")
    ap.add_argument("--cpu-sample-T", type=int, default=0,
                    help="tokens of the oracle sample cell (0 = the workload's T)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before the run, one streaming pass (out = -in, fp32) that reads and "
                         "writes this many MiB: the reference dispatch for scaling HBM "
                         "traffic counters")
    ap.add_argument("--trd-lanes", type=int, default=0,
                    help="streams of the exact path's tridiagonalisation (library default 4); "
                         "1 keeps every launch on one stream, for counter collection")
    ap.add_argument("--trd-stages", type=int, default=-1, choices=[-1, 1, 2],
                    help="reduction of the exact path's token Grams to tridiagonal form: 2 "
                         "two-stage (band, then bulge chasing), 1 one-stage; -1 the library's "
                         "choice (two stages once a call's matrices times T reach 32 * 4096)")
    ap.add_argument("--no-stage-profile", action="store_true",
                    help="skip the event-instrumented step; the stage and roofline fields are "
                         "then omitted")
    ap.add_argument("--attend", action="store_true",
                    help="instead of the benchmark step: decode-time attention of one new token "
                         "(4 query heads per key-value head for GQA caches, 1 for MHA) over every "
                         "layer of the compressed --workload cache, on the factors vs the "
                         "materialising path (decompress, then attention)")
    ap.add_argument("--diagnostics", action="store_true",
                    help="instead of the benchmark step: the appendix-A three-mode table of one "
                         "synthetic Mistral-shaped layer (layer 15, T = 1024, K and V), and the "
                         "slice-mode spectrum timed over every cell of --workload")
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def pass_model(codec):
    """Algorithmic bytes and flops of the roofline passes of one step (the section-4/5 path
    over every cell, then its decompression), as the design counts them: bytes are the
    minimum each pass must move (an fp32 X~ round trip is not algorithmic), flops the
    useful ones.  Eigensolvers, QR and the allocator are timed but on neither roofline.
    Returns {pass: dict(bytes, flops, peak_tf, stages, direction)}; `stages` are the
    instrumented library stages whose time the pass takes."""
    L, B, H, T, d = codec.shape
    m = codec.group_layers * H
    N = m * d
    nc = len(codec.cells)
    esz = 2 if codec.dtype == 1 else 4
    elt = float(m) * T * d                        # entries per cell
    flash = codec.method == 1
    mfma = 2500.0 if esz == 2 else 157.3          # products reading the cache: bf16 cores
    rT = [p.r_T for p in codec.params]
    bits = [p.bits for p in codec.params]
    g = codec.group
    out = {}
    fg_peak = 2500.0 if (esz == 2 and d == 128) else 157.3
    out["feature_gram"] = dict(bytes=nc * elt * esz, flops=nc * elt * 2.0 * d, peak_tf=fg_peak,
                               stages=["feature_gram"], direction="compress")
    if flash:
        reads = 2 + 2 * codec.opts.power_iters      # X Omega, (X^T Q, X Q') per iteration, Q^T X
        out["sketch"] = dict(bytes=nc * elt * esz * reads, flops=nc * elt * 2.0 * codec.ell * reads,
                             peak_tf=mfma, stages=["sketch"], direction="compress")
    else:
        out["token_gram"] = dict(bytes=nc * elt * esz, flops=nc * elt * float(T + 1), peak_tf=mfma,
                                 stages=["token_gram"], direction="compress")
        out["project"] = dict(bytes=nc * elt * esz, flops=sum(elt * 2.0 * r for r in rT), peak_tf=mfma,
                              stages=["project"], direction="compress")
    code_b = sum(elt * (b / 8.0 + (2.0 / g if b else 0.0)) for b in bits)
    recon_f = sum(elt * 2.0 * r for r in rT)
    out["residual"] = dict(bytes=nc * elt * esz + code_b, flops=recon_f, peak_tf=2500.0,
                           stages=["reconstruct", "residual"], direction="compress")
    out["decode"] = dict(bytes=code_b + nc * elt * esz, flops=recon_f, peak_tf=2500.0,
                         stages=["reconstruct", "decode"], direction="decompress")
    return out


def roofline_report(model, prof_c, prof_d, step_ms):
    """Per-pass fractions and the whole-path fraction t_roof / t from the instrumented
    compress (prof_c) and decompress (prof_d) stage times of one step."""
    passes = {}
    t_roof = 0.0
    for name, p in model.items():
        prof = prof_c if p["direction"] == "compress" else prof_d
        ms = sum(prof.get(s, (0.0, 0))[0] for s in p["stages"])
        launches = sum(prof.get(s, (0.0, 0))[1] for s in p["stages"])
        t_b = p["bytes"] / (HBM_GBS * 1e9) * 1e3           # ms at the HBM peak
        t_f = p["flops"] / (p["peak_tf"] * 1e12) * 1e3      # ms at the matrix-core peak
        t_roof += max(t_b, t_f)
        if ms <= 0:
            continue
        passes[name] = {"ms": round(ms, 3), "launches": launches,
                        "bound": "hbm" if t_b >= t_f else "mfma",
                        "GBps": round(p["bytes"] / ms / 1e6, 1), "hbm_frac": round(t_b / ms, 4),
                        "TFLOPs": round(p["flops"] / ms / 1e9, 2), "mfma_peak_TFLOPs": p["peak_tf"],
                        "mfma_frac": round(t_f / ms, 4), "frac": round(max(t_b, t_f) / ms, 4),
                        "alg_bytes": p["bytes"], "alg_flops": p["flops"]}
    whole = {"t_roof_ms": round(t_roof, 3), "t_ms": round(step_ms, 3),
             "frac": round(t_roof / step_ms, 5) if step_ms > 0 else None}
    return passes, whole


# kernel source of each pass whose HBM traffic was taken with hardware counters
PASS_SOURCE = {"token_gram": "paper_2607_12550_amd/csrc/k_gemm16.hip",
               "residual": "paper_2607_12550_amd/csrc/k_fused.hip",
               "decode": "paper_2607_12550_amd/csrc/k_fused.hip"}


def measured_traffic(name, workload):
    """HBM bytes per launch of a pass from the committed counter summary
    profiles/traffic_<pass>_<workload>.md (lines 'traffic_bytes_per_launch: X' and
    'source_sha256: H'); None when there is none or the kernel source changed since."""
    import hashlib
    src = PASS_SOURCE.get(name)
    path = os.path.join(ROOT, "profiles", f"traffic_{name}_{workload}.md")
    if not src or not os.path.exists(path):
        return None
    with open(os.path.join(ROOT, src), "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.split(":", 1)[0].strip() in ("traffic_bytes_per_launch", "source_sha256"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip().strip("`")
    if fields.get("source_sha256") != sha or "traffic_bytes_per_launch" not in fields:
        return None
    return float(fields["traffic_bytes_per_launch"])


def cpu_baseline(K_np, V_np, cfg, params, group, T_sample, method, q, p, iters, n_cells,
                 min_seconds=10.0, max_cells=16):
    """fp64 oracle on whole cells (keys, then values, of layer groups 0, 1, ... of batch item
    0) timed on the host cores until at least min_seconds of work (at most max_cells cells);
    the whole cache's oracle time is that sample's time scaled by n_cells / k."""
    import numpy as np
    import kvsynth
    from oracle import pipeline as opl
    gl, H, d = cfg["group_layers"], cfg["n_heads"], cfg["d"]
    n_groups = cfg["n_layers"] // gl
    cores = len(os.sched_getaffinity(0))
    done, nbytes, t_all = [], 0, 0.0
    for i in range(max_cells):
        g, tensor = i // 2, i % 2
        if g >= n_groups:
            break
        src = (K_np, V_np)[tensor]
        x = kvsynth.bf16_bits_to_f32(src[g * gl:(g + 1) * gl, 0, :, :T_sample, :]).astype(np.float64)
        X = x.reshape(gl * H, T_sample, d)
        pc = params[(tensor * n_groups + g) * cfg["batch"]]   # codec cell order: tensor, group, batch
        t0 = time.perf_counter()
        sp = opl.spectrum(X, method=method, q=q, p=p, power_iters=iters, seed=0)
        rT = min(pc.r_T, sp["rT_max"])
        rd = pc.r_d if rT else 0
        opl.compress_cell(X, r_T=rT, r_d=rd, bits=pc.bits, group=group, seed=0,
                          factor_bytes=2, spec=sp)
        t_all += time.perf_counter() - t0
        nbytes += X.size * 2
        done.append(f"{'KV'[tensor]}{g}:({rT},{rd},{pc.bits})")
        if t_all >= min_seconds:
            break
    k = len(done)
    return {"value": round(nbytes / t_all / 1e9, 5), "unit": "GB/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{k} of {n_cells} cells, whole ({gl} layers x {H} heads, T={T_sample}, d={d}, "
                      f"bf16, {nbytes / 1e6:.1f} MB) {' '.join(done)}: {method} spectrum + compress at "
                      f"the allocated ranks/bits + decode, fp64 numpy/LAPACK, {t_all:.1f} s; the whole "
                      f"cache extrapolated x{n_cells / k:.0f}",
            "seconds": round(t_all, 2),
            "extrapolated_full_cache_s": round(t_all * n_cells / k, 1)}


def diagnostics(args):
    """Appendix A's table (sigma_1 / sigma_min and ranks at 10% / 20% relative Frobenius
    error per mode) for one synthetic layer, from the library's three mode spectra; then
    the slice-mode Gram of every cell of the workload, timed with the stage events."""
    import numpy as np
    import torch

    import kvsynth
    import paper_2607_12550_amd as J
    from paper_2607_12550_amd.cache import CacheCodec

    ctx = J.jolt_create(0)
    H, T, d = 8, 1024, 128
    desc = J.cell_desc(dtype=J.JOLT_BF16, n_layers=1, n_heads=H, T=T, d=d,
                       stride_layer=H * T * d, stride_head=T * d, stride_token=d)
    ws_s = torch.empty(J.jolt_slice_spectrum_workspace_size(desc, 1), dtype=torch.uint8, device="cuda")
    ws = torch.empty(J.jolt_workspace_size(desc, 1, None), dtype=torch.uint8, device="cuda")
    rows = []
    for tensor, name in ((0, "K"), (1, "V")):
        x = kvsynth.layer_kv(layer=15, tensor=tensor, n_heads=H, T=T, d=d, alpha=(1.5, 0.7)[tensor],
                             n_out=2, out_scale=10.0, data_seed=0)[0]
        t = torch.from_numpy(kvsynth.f32_to_bf16_bits(x).view(np.int16)).view(torch.bfloat16).cuda()
        lam_s = J.jolt_slice_spectrum(ctx, desc, [t], ws_s)[0]
        _, lam_t, lam_f = J.jolt_spectrum(ctx, desc, [t], None, None, ws)
        for mode, lam, n in (("heads", lam_s, H), ("tokens", lam_t[0], T), ("features", lam_f[0], d)):
            rng, r10, r20 = J.jolt_mode_summary(lam, 0.10, 0.20)
            # an infinite range: the smallest eigenvalue is below the fp32 Gram's resolution
            rows.append({"tensor": name, "mode": f"{mode} ({n})",
                         "sigma_range": round(rng, 2) if np.isfinite(rng) else "inf",
                         "r_10pct": f"{r10}/{n}", "r_20pct": f"{r20}/{n}"})
            log(f"{name} {mode:9s} ({n:5d})  sigma1/sigmamin {rng:12.2f}  r10 {r10:5d}/{n}  r20 {r20:5d}/{n}")
    # slice-mode Gram over every cell of the workload
    cfg = dict(kvsynth.CONFIGS[args.workload])
    gl = cfg.pop("group_layers")
    # generation runs in worker processes (the values do not depend on their number)
    Knp, Vnp = kvsynth.make_cache(**cfg, workers=min(16, os.cpu_count() or 1))
    to_dev = (lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()) \
        if cfg["dtype"] == "bf16" else (lambda a: torch.from_numpy(a).cuda())
    K, V = to_dev(Knp), to_dev(Vnp)
    codec = CacheCodec(K, V, group_layers=gl, method="exact", ratio=2.0)
    cd, ptrs = codec.desc, [c.ptr for c in codec.cells]
    wsc = torch.empty(J.jolt_slice_spectrum_workspace_size(cd, len(ptrs)), dtype=torch.uint8, device="cuda")
    J.jolt_slice_spectrum(ctx, cd, ptrs, wsc)                       # warm-up
    J.jolt_profile_enable(ctx, True)
    J.jolt_profile_reset(ctx)
    reps = 5
    for _ in range(reps):
        J.jolt_slice_spectrum(ctx, cd, ptrs, wsc)
    prof = J.jolt_profile_read(ctx)
    J.jolt_profile_enable(ctx, False)
    ms = prof["slice_gram"][0] / reps
    m = cd.n_layers * cd.n_heads
    elems = float(m) * cd.T * cd.d * len(ptrs)
    flops = float(m) * (m + 16) * cd.T * cd.d * len(ptrs)       # the tile pairs I >= J
    esz = 2 if cfg["dtype"] == "bf16" else 4
    out = {"diagnostics": "appendix A, synthetic Mistral-shaped layer 15, T = 1024", "rows": rows,
           "slice_gram": {"workload": args.workload, "cells": len(ptrs), "m": m, "ms": round(ms, 4),
                          "GBps_cache_read": round(elems * esz / ms / 1e6, 1),
                          "TFLOPs_fp32": round(flops / ms / 1e9, 2), "peak_fp32_TFLOPs": 157.3,
                          "eig_ms": round((prof["tridiag_small"][0] + prof["eigvals"][0]) / reps, 4)}}
    print(json.dumps(out))
    codec.close()
    J.jolt_destroy(ctx)


def attend_bench(args):
    """Decode-time attention on the compressed cache.  The cache is compressed once (the
    workload's method and budget); then one query token per sequence attends over every
    layer: with the fused kernels reading only the blobs, and, for reference, with the
    materialising path (jolt_decompress of every cell to bf16, then fp32 attention in torch).
    Algorithmic bytes of the fused path: per item (layer) the key and value token factors
    U_T (T r_T c), the codes of the layer's H slices (H T d b / 8) and their scales
    (2 H T d / g); the core and feature factors are negligible."""
    import numpy as np
    import torch

    import kvsynth
    import paper_2607_12550_amd as J
    from paper_2607_12550_amd.cache import CacheCodec

    cfg = dict(kvsynth.CONFIGS[args.workload])
    gl = cfg.pop("group_layers")
    method, ratio = WORKLOAD_RUN.get(args.workload, ("exact", 2.0))
    method, ratio = args.method or method, args.ratio or ratio
    log("generating", args.workload)
    # generation runs in worker processes (the values do not depend on their number)
    Knp, Vnp = kvsynth.make_cache(**cfg, workers=min(16, os.cpu_count() or 1))
    dev = torch.device("cuda", 0)
    to_dev = (lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)) \
        if cfg["dtype"] == "bf16" else (lambda a: torch.from_numpy(a).to(dev))
    K, V = to_dev(Knp), to_dev(Vnp)
    del Knp, Vnp
    codec = CacheCodec(K, V, group_layers=gl, method=method, ratio=ratio)
    codec.calibrate()
    codec.spectrum()
    codec.allocate()
    codec.compress()
    hdr = codec.headers()
    L, B, H, T, d = codec.shape
    rep = 4 if H == 8 else 1
    n_q = rep * H
    # items: every (group, batch item, layer of the group)
    pair = {}
    for i, c in enumerate(codec.cells):
        pair.setdefault((c.group, c.batch), [None, None])[c.tensor] = i
    items = [(pair[(g, b)][0], pair[(g, b)][1], li, g * gl + li, b)
             for (g, b) in sorted(pair) for li in range(gl)]
    kb = [codec.blob_ptrs[k] for k, _, _, _, _ in items]
    vb = [codec.blob_ptrs[v] for _, v, _, _, _ in items]
    ks = [codec.blob_sizes[k] for k, _, _, _, _ in items]
    vs = [codec.blob_sizes[v] for _, v, _, _, _ in items]
    kh = np.stack([hdr[k] for k, _, _, _, _ in items])
    vh = np.stack([hdr[v] for _, v, _, _, _ in items])
    layers = [li for _, _, li, _, _ in items]
    params = codec.params
    rk = max(params[k].r_T for k, _, _, _, _ in items)
    rv = max(params[v].r_T for _, v, _, _, _ in items)
    n = len(items)
    ws = torch.empty(J.jolt_attend_workspace_size(n, n_q, T, d, rk, rv), dtype=torch.uint8, device=dev)
    g = torch.Generator(device="cpu").manual_seed(0)
    Q = torch.randn((n, n_q, d), generator=g).to(dev)
    O = torch.empty_like(Q)
    scale = 1.0 / float(np.sqrt(d))
    call = lambda: J.jolt_attend(codec.ctx, kb, vb, kh, vh, layers, Q, O, scale, ws, k_bytes=ks, v_bytes=vs)
    call()
    torch.cuda.synchronize()
    reps = 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    fused_ms = e0.elapsed_time(e1) / reps
    # materialising path: decompress every cell to bf16, then attention of the same queries
    Kout, Vout = torch.empty_like(K), torch.empty_like(V)

    def materialise():
        codec.decompress(Kout, Vout)
        Kl = torch.stack([Kout[l, b] for _, _, _, l, b in items]).float()        # [n, H, T, d]
        Vl = torch.stack([Vout[l, b] for _, _, _, l, b in items]).float()
        q = Q.view(n, H, rep, d)
        p_ = torch.softmax(scale * torch.matmul(q, Kl.transpose(-1, -2).contiguous()), dim=-1)
        return torch.matmul(p_, Vl).view(n, n_q, d)

    ref = materialise()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        materialise()
    e1.record()
    torch.cuda.synchronize()
    mat_ms = e0.elapsed_time(e1) / reps
    rel = float(torch.linalg.norm(O - ref) / torch.linalg.norm(ref))
    c = 2 if params[0].factor_dtype == J.JOLT_FACTOR_F16 else 4
    nbytes = 0
    for k, v, _, _, _ in items:
        for p_ in (params[k], params[v]):
            nbytes += T * p_.r_T * c + H * T * d * p_.bits // 8 + (2 * H * T * d // p_.group if p_.bits else 0)
    cache_layer_bytes = n * 2 * H * T * d * (2 if cfg["dtype"] == "bf16" else 4)
    out = {"attend": {"workload": args.workload, "method": method, "ratio": ratio, "items": n, "n_q": n_q,
                      "kv_heads": H, "T": T, "d": d, "fused_ms": round(fused_ms, 4),
                      "materialise_ms": round(mat_ms, 4), "speedup": round(mat_ms / fused_ms, 2),
                      "bytes_read": nbytes, "uncompressed_kv_bytes": cache_layer_bytes,
                      "GBps": round(nbytes / fused_ms / 1e6, 1), "frac_hbm": round(nbytes / fused_ms / 1e6 / HBM_GBS, 4),
                      "rel_diff_vs_materialising": rel}}
    print(json.dumps(out))
    codec.close()


def _profiled_step(J, codec, Kout, Vout, allocator):
    """One extra step with the library's stage events on: stage times of the compress part
    (spectrum, allocation, compress) and of the decompression, separately."""
    import torch
    J.jolt_profile_enable(codec.ctx, True)
    J.jolt_profile_reset(codec.ctx)
    codec.spectrum()
    codec.allocate(strategy=allocator)
    codec.compress()
    torch.cuda.synchronize()
    prof_c = J.jolt_profile_read(codec.ctx)
    J.jolt_profile_reset(codec.ctx)
    codec.decompress(Kout, Vout)
    torch.cuda.synchronize()
    prof_d = J.jolt_profile_read(codec.ctx)
    J.jolt_profile_enable(codec.ctx, False)
    return prof_c, prof_d


def method_comparison(K, V, gl, ratio, args, exact_compress_ms):
    """FlashJoLT against the exact path on the same cache and budget (section 5 reports
    5.25-13.57x on real caches at T = 1024): the compress part of a step (spectrum,
    allocation, compress) timed for the randomized method, with its error."""
    import numpy as np
    import torch
    from paper_2607_12550_amd.cache import CacheCodec, layer_errors
    codec = CacheCodec(K, V, group_layers=gl, method="flash", ratio=ratio,
                       oversample=args.oversample, power_iters=args.power_iters, max_cells_per_call=64)
    codec.calibrate()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    for s in range(1 + args.compare_steps):
        e0.record()
        codec.spectrum()
        codec.allocate()
        codec.compress()
        e1.record()
        torch.cuda.synchronize()
        if s:
            times.append(e0.elapsed_time(e1))
    Kout, Vout = torch.empty_like(K), torch.empty_like(V)
    codec.decompress(Kout, Vout)
    torch.cuda.synchronize()
    eK, eV = layer_errors(K, Kout), layer_errors(V, Vout)
    flash_ms = float(np.median(times))
    out = {"flash_compress_ms": round(flash_ms, 2), "exact_compress_ms": round(exact_compress_ms, 2),
           "exact_over_flash": round(exact_compress_ms / flash_ms, 2), "flash_q": codec.opts.q or codec.rT_max,
           "flash_ell": codec.ell, "flash_rel_frobenius_error": {"K": round(float(eK.mean()), 6),
                                                                  "V": round(float(eV.mean()), 6)},
           "paper_context": "5.25-13.57x FlashJoLT over exact compression time (Mistral-7B-v0.3, "
                            "T = 1024, real caches, one A100-40GB; section 5, appendix C)"}
    codec.close()
    del codec, Kout, Vout
    torch.cuda.empty_cache()
    return out


def trd_stages_used(args, cells_per_call, T):
    """Reduction of the exact token Grams to tridiagonal form in this run: the forced one, or
    the library's automatic choice (two stages once a call's matrices times T reach
    32 * 4096; T up to 768 is reduced in one workgroup per matrix)."""
    if T <= 768:
        return "one-workgroup"
    if args.trd_stages in (1, 2):
        return "two-stage" if args.trd_stages == 2 else "one-stage"
    return "two-stage" if cells_per_call * T >= 32 * 4096 else "one-stage"


def main():
    args = parse()
    if args.attend:
        attend_bench(args)
        return
    if args.diagnostics:
        diagnostics(args)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: there is no multi-GPU path (cells would shard "
              "across GPUs, with an all-gather of the spectra before the allocation).", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import kvsynth
    import paper_2607_12550_amd as J
    from paper_2607_12550_amd.cache import CacheCodec, layer_errors

    cfg = dict(kvsynth.CONFIGS[args.workload])
    gl = cfg.pop("group_layers")
    method, ratio = WORKLOAD_RUN.get(args.workload, ("exact", 2.0))
    method = args.method or method
    ratio = args.ratio or ratio
    log("generating", args.workload)
    t0 = time.perf_counter()
    # generation runs in worker processes (the values do not depend on their number)
    Knp, Vnp = kvsynth.make_cache(**cfg, workers=max(1, min(args.gen_workers, os.cpu_count() or 1)))
    if args.rope_post > 1.0:
        for l in range(Knp.shape[0]):
            xr = kvsynth.apply_rope(kvsynth.bf16_bits_to_f32(Knp[l]) if cfg["dtype"] == "bf16" else Knp[l],
                                    args.rope_post)
            Knp[l] = kvsynth.f32_to_bf16_bits(xr) if cfg["dtype"] == "bf16" else xr
        log(f"keys rotated (RoPE base {args.rope_post:g}) before compression")
    log(f"generated in {time.perf_counter() - t0:.1f} s")
    dev = torch.device("cuda", 0)
    to_dev = (lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)) \
        if cfg["dtype"] == "bf16" else (lambda a: torch.from_numpy(a).to(dev))
    K, V = to_dev(Knp), to_dev(Vnp)
    if args.calib_copy_mib:
        src = torch.ones((args.calib_copy_mib << 20) // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        log(f"calibration pass: {args.calib_copy_mib} MiB read + written")
        del src, dst
    codec = CacheCodec(K, V, group_layers=gl, method=method, ratio=ratio,
                       oversample=args.oversample, power_iters=args.power_iters, tau=args.tau,
                       max_cells_per_call=args.cells_per_call)
    if args.trd_lanes:
        J.jolt_debug_set(codec.ctx, J.JOLT_DBG_TRD_LANES, args.trd_lanes)
    if args.trd_stages > 0:
        J.jolt_debug_set(codec.ctx, J.JOLT_DBG_TRD_TWO_STAGE, 1 if args.trd_stages == 2 else 0)
    eps2 = codec.calibrate()
    log("eps2", eps2, "cells", len(codec.cells), "per call", codec.chunk)
    Kout, Vout = torch.empty_like(K), torch.empty_like(V)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    t_comp, t_dec = [], []

    alloc_res = {}

    def step():
        ev[0].record(stream)
        codec.spectrum(stream)
        alloc_res.update(codec.allocate(strategy=args.allocator))
        codec.compress(stream)
        ev[1].record(stream)
        codec.decompress(Kout, Vout, stream)
        ev[2].record(stream)

    for w in range(args.warmup):
        log("warmup step", w)
        step()
    torch.cuda.synchronize()
    # timed steps: the production path (no instrumentation)
    t0 = time.perf_counter()
    for s in range(args.steps):
        step()
        torch.cuda.synchronize()
        t_comp.append(ev[0].elapsed_time(ev[1]))
        t_dec.append(ev[1].elapsed_time(ev[2]))
        log(f"step {s}: compress {t_comp[-1]:.1f} ms, decompress {t_dec[-1]:.1f} ms")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = elapsed / args.steps * 1e3
    # one extra instrumented step: HIP events around every stage, compress and decompress apart
    prof_c, prof_d = ({}, {}) if args.no_stage_profile else _profiled_step(J, codec, Kout, Vout, args.allocator)

    cache_bytes = codec.cache_bytes
    value = cache_bytes * args.steps / elapsed / 1e9
    eK = layer_errors(K, Kout)
    eV = layer_errors(V, Vout)
    comp_bytes = codec.compressed_bytes()
    alloc = [(p.r_T, p.r_d, p.bits) for p in codec.params]
    roof, passes, whole = None, {}, None
    if prof_c:
        passes, whole = roofline_report(pass_model(codec), prof_c, prof_d, step_ms)
        dom = max(passes, key=lambda k: passes[k]["ms"])
        P = passes[dom]
        if P["bound"] == "hbm":
            roof = {"kernel": dom, "bound": "hbm", "achieved": P["GBps"], "peak": HBM_GBS, "unit": "GB/s",
                    "frac": P["hbm_frac"]}
        else:
            roof = {"kernel": dom, "bound": "mfma", "achieved": P["TFLOPs"], "peak": P["mfma_peak_TFLOPs"],
                    "unit": "TFLOP/s", "frac": P["mfma_frac"]}
        roof["traffic"] = measured_traffic(dom, args.workload)
        roof["launches"] = P["launches"]
        roof["avg_launch_us"] = round(P["ms"] * 1e3 / max(1, P["launches"]), 2)
        roof["whole_path"] = whole
    stages = {}
    for tag, prof in (("compress", prof_c), ("decompress", prof_d)):
        for s_, v in prof.items():
            if v[1]:
                stages[f"{tag}:{s_}"] = {"ms_per_step": round(v[0], 3), "launches_per_step": v[1]}
    out = {
        "metric": "KV GB/s compressed+decompressed per GPU; rel. Frobenius error K/V at 2x",
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": args.workload, "layers": cfg["n_layers"], "kv_heads": cfg["n_heads"],
                   "T": cfg["T"], "head_dim": cfg["d"], "batch": cfg["batch"], "group_layers": gl,
                   "cells": len(codec.cells), "cells_per_call": codec.chunk, "method": method,
                   "ratio": ratio, "allocator": args.allocator, "tau": args.tau,
                   **({"tau_rT_cap": codec.tau_cap_used} if args.tau == "exact" else {}),
                   "keys": "post-rope" if args.rope_post > 1.0 else "pre-rope",
                   **({"tridiagonalisation": trd_stages_used(args, codec.chunk, cfg["T"])}
                      if method == "exact" else {}),
                   "cache_bytes": cache_bytes},
        "compress_GBps": round(cache_bytes / (np.median(t_comp) * 1e-3) / 1e9, 3),
        "decompress_GBps": round(cache_bytes / (np.median(t_dec) * 1e-3) / 1e9, 3),
        "rel_frobenius_error": {"K": round(float(eK.mean()), 6), "V": round(float(eV.mean()), 6)},
        "achieved_ratio": round(cache_bytes / comp_bytes, 4),
        "achieved_ratio_eq1_payload": round(cache_bytes / codec.payload_bytes(), 4),
        "allocation_rT_max": max(a[0] for a in alloc),
        "allocation_model_error": alloc_res.get("model_error"),
        "stage_ms_per_step": stages,
        "passes": passes,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        Ts = args.cpu_sample_T or cfg["T"]
        out["cpu_baseline"] = cpu_baseline(Knp, Vnp, dict(cfg, group_layers=gl), codec.params,
                                           codec.group, Ts, method, codec.opts.q or codec.rT_max,
                                           args.oversample, args.power_iters, len(codec.cells))
    exact_compress_ms = float(np.median(t_comp))
    codec.close()
    del codec, Kout, Vout
    torch.cuda.empty_cache()
    if method == "exact" and args.compare_steps > 0:
        log("FlashJoLT on the same cache ...")
        out["method_comparison"] = method_comparison(K, V, gl, ratio, args, exact_compress_ms)
    print(json.dumps(out))


if __name__ == "__main__":
    main()

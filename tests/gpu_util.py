"""Helpers for the GPU parity tests: device buffers, contexts, calls through the C-ABI."""
import sys

import numpy as np
import torch

import kvsynth
import paper_2607_12550_amd as J

_CTX = None


def note(*a):
    print("[gpu-step]", *a, file=sys.stderr, flush=True)


def ctx():
    global _CTX
    if _CTX is None:
        assert torch.cuda.is_available(), "GPU tests need a GPU"
        _CTX = J.jolt_create(0)
    return _CTX


def device_cells(cells_f64, dtype):
    """List of (m, T, d) fp64 arrays -> (torch device tensors, exact fp64 copies, desc)."""
    xs, exact = [], []
    for x in cells_f64:
        if dtype == "bf16":
            bits = kvsynth.f32_to_bf16_bits(x.astype(np.float32))
            t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).cuda()
            exact.append(kvsynth.bf16_bits_to_f32(bits).astype(np.float64))
        else:
            x32 = x.astype(np.float32)
            t = torch.from_numpy(x32.copy()).cuda()
            exact.append(x32.astype(np.float64))
        xs.append(t)
    m, T, d = cells_f64[0].shape
    desc = J.cell_desc(dtype=J.JOLT_BF16 if dtype == "bf16" else J.JOLT_F32, n_layers=1, n_heads=m,
                       T=T, d=d, stride_layer=m * T * d, stride_head=T * d, stride_token=d)
    return xs, exact, desc


def workspace(desc, n, opts=None):
    nb = J.jolt_workspace_size(desc, n, opts)
    return torch.empty(nb, dtype=torch.uint8, device="cuda")


def compress(xs, desc, params, opts=None, ws=None):
    n = len(xs)
    ws = workspace(desc, n, opts) if ws is None else ws
    blobs = [torch.zeros(J.jolt_compressed_size(desc, p), dtype=torch.uint8, device="cuda")
             for p in params]
    note("jolt_compress", n, "cells", [(p.r_T, p.r_d, p.bits) for p in params])
    J.jolt_compress(ctx(), desc, xs, params, opts, ws, blobs)
    torch.cuda.synchronize()
    return blobs, ws


def decompress(blobs, desc, out_dtype="f32", ws=None):
    m, T, d = desc.n_layers * desc.n_heads, desc.T, desc.d
    od = J.cell_desc(dtype=J.JOLT_BF16 if out_dtype == "bf16" else J.JOLT_F32, n_layers=desc.n_layers,
                     n_heads=desc.n_heads, T=T, d=d, stride_layer=desc.stride_layer,
                     stride_head=desc.stride_head, stride_token=desc.stride_token)
    outs = [torch.empty((m, T, d), dtype=torch.bfloat16 if out_dtype == "bf16" else torch.float32,
                        device="cuda") for _ in blobs]
    ws = workspace(desc, len(blobs)) if ws is None else ws
    note("jolt_decompress", len(blobs), "blobs")
    J.jolt_decompress(ctx(), blobs, od, outs, ws)
    torch.cuda.synchronize()
    return [o.float().cpu().numpy().astype(np.float64) for o in outs]


def blob_bytes(b):
    return b.cpu().numpy().tobytes()

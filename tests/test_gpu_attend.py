"""GPU parity of decode-time attention evaluated on the compressed factors (section 8)
against the oracle's softmax attention over the oracle's decode of the same blobs.

Blobs come from the oracle's writer (any ranks and bits, including a residual-only key
cell, a backbone-only value cell and fp32 factors) and from the GPU compressor.  The
tolerance is fp32 arithmetic over at most a few hundred terms per sum: every output
entry of a query head is within 1e-4 of the norm of that head's output.  The fused path is also checked against
the materialising path (jolt_decompress to fp32, then attention on the CPU).
"""
import numpy as np
import pytest
import torch

import kvsynth
import paper_2607_12550_amd as J
from gpu_util import blob_bytes, compress, ctx, decompress, device_cells, note
from oracle import attention as oat, pipeline as opl

pytestmark = pytest.mark.gpu
TOL = 1e-4


def _cell(rng, m, T, d, decay=1.5):
    core = rng.standard_normal((m, T, 16)) @ (rng.standard_normal((16, d)) * np.arange(1, d + 1) ** -decay)
    return core + 0.05 * rng.standard_normal((m, T, d))


def _oracle_blob(X, H, r_T, r_d, bits, group, seed, fb=2):
    ref = opl.compress_cell(X, r_T=r_T, r_d=r_d, bits=bits, group=group, seed=seed, factor_bytes=fb)
    return opl.write_blob(ref, in_dtype="bf16", n_heads=H)


def _run(kblobs, vblobs, layers, Q, d):
    n, n_q = Q.shape[0], Q.shape[1]
    kb = [torch.from_numpy(np.frombuffer(b, np.uint8).copy()).cuda() for b in kblobs]
    vb = [torch.from_numpy(np.frombuffer(b, np.uint8).copy()).cuda() for b in vblobs]
    kh = np.stack([np.frombuffer(b[:128], np.uint8) for b in kblobs])
    vh = np.stack([np.frombuffer(b[:128], np.uint8) for b in vblobs])
    rk = max(opl.read_blob(b)["r_T"] for b in kblobs)
    rv = max(opl.read_blob(b)["r_T"] for b in vblobs)
    T = opl.read_blob(kblobs[0])["T"]
    ws = torch.empty(J.jolt_attend_workspace_size(n, n_q, T, d, rk, rv), dtype=torch.uint8, device="cuda")
    Qd = torch.from_numpy(Q.astype(np.float32)).cuda()
    Od = torch.empty_like(Qd)
    note("jolt_attend", n, "items, n_q", n_q, "T", T, "d", d, "ranks", rk, rv)
    J.jolt_attend(ctx(), kb, vb, kh, vh, layers, Qd, Od, 1.0 / np.sqrt(d), ws)
    torch.cuda.synchronize()
    return Od.cpu().numpy().astype(np.float64)


def _check(got, want):
    """Per query head j: every output entry within 1e-4 of that head's output norm."""
    assert got.shape == want.shape
    for j in range(want.shape[0]):
        nj = np.linalg.norm(want[j])
        err = np.abs(got[j] - want[j]).max()
        assert err <= TOL * nj, (j, err, nj)
    assert np.linalg.norm(got - want) <= TOL * np.linalg.norm(want)


@pytest.mark.parametrize("case", ["gqa_ragged", "residual_only_keys", "single_token", "two_items_fp32_factors"])
def test_attention_on_oracle_blobs(case):
    rng = np.random.default_rng(3)
    if case == "gqa_ragged":          # 2 layers x 4 heads, T = 300 (ragged last chunk), 2 queries per head
        L, H, T, d, n_q, layers = 2, 4, 300, 128, 8, [1]
        kp, vp, fb = (40, 48, 4), (24, 64, 2), 2
    elif case == "residual_only_keys":   # keys: no backbone; values: no residual; one full chunk
        L, H, T, d, n_q, layers = 1, 4, 64, 128, 4, [0]
        kp, vp, fb = (0, 0, 8), (16, 16, 0), 2
    elif case == "single_token":
        L, H, T, d, n_q, layers = 1, 2, 1, 64, 8, [0]
        kp, vp, fb = (1, 8, 2), (1, 8, 4), 2
    else:                                # two items on different layers, fp32 factors
        L, H, T, d, n_q, layers = 3, 2, 200, 64, 8, [2, 0]
        kp, vp, fb = (32, 32, 4), (48, 16, 8), 4
    n = len(layers)
    kblobs, vblobs = [], []
    for i in range(n):
        K = _cell(rng, L * H, T, d, 1.5)
        V = _cell(rng, L * H, T, d, 0.7)
        kblobs.append(_oracle_blob(K, H, *kp, group=32, seed=11 + i, fb=fb))
        vblobs.append(_oracle_blob(V, H, *vp, group=32, seed=23 + i, fb=fb))
    Q = rng.standard_normal((n, n_q, d)) * 0.5
    got = _run(kblobs, vblobs, layers, Q, d)
    for i in range(n):
        want = oat.attend(opl.decode_blob(kblobs[i]), opl.decode_blob(vblobs[i]), layers[i], H, Q[i],
                          1.0 / np.sqrt(d))
        _check(got[i], want)


def test_attention_on_gpu_blobs_matches_the_materialising_path():
    """Keys and values of a Mistral-shaped layer group (4 layers x 8 heads, T = 512) compressed
    on the GPU; attention on the factors vs decompression followed by attention."""
    H, L, T, d = 8, 4, 512, 128
    k = kvsynth.make_cache(n_layers=L, n_heads=H, T=T, d=d, dtype="f32")
    cells = [k[t][:, 0].reshape(L * H, T, d).astype(np.float64) for t in (0, 1)]
    xs, ex, desc = device_cells(cells, "bf16")
    desc = J.cell_desc(dtype=J.JOLT_BF16, n_layers=L, n_heads=H, T=T, d=d,
                       stride_layer=H * T * d, stride_head=T * d, stride_token=d)
    params = [J.Params(96, 64, 4, 64, J.JOLT_FACTOR_F16, 0, 5), J.Params(64, 96, 8, 64, J.JOLT_FACTOR_F16, 0, 6)]
    blobs, _ = compress(xs, desc, params)
    kb, vb = blob_bytes(blobs[0]), blob_bytes(blobs[1])
    rng = np.random.default_rng(5)
    n_q = 32
    layers = [0, 1, 2, 3]
    Q = rng.standard_normal((4, n_q, d))
    got = _run([kb] * 4, [vb] * 4, layers, Q, d)
    Kh, Vh = decompress(blobs[:1], desc, "f32")[0], decompress(blobs[1:], desc, "f32")[0]
    Ko, Vo = opl.decode_blob(kb), opl.decode_blob(vb)
    for i, l in enumerate(layers):
        _check(got[i], oat.attend(Ko, Vo, l, H, Q[i], 1.0 / np.sqrt(d)))       # oracle decode
        _check(got[i], oat.attend(Kh, Vh, l, H, Q[i], 1.0 / np.sqrt(d)))       # GPU decode


def test_attention_rejects_bad_calls():
    rng = np.random.default_rng(0)
    X = _cell(rng, 4, 64, 64)
    b = _oracle_blob(X, 4, 8, 8, 2, 32, 1)
    kb = torch.from_numpy(np.frombuffer(b, np.uint8).copy()).cuda()
    h = np.frombuffer(b[:128], np.uint8)[None]
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    Q = torch.zeros((1, 6, 64), device="cuda")
    with pytest.raises(J.JoltError):        # 6 query heads over 4 key-value heads
        J.jolt_attend(ctx(), [kb], [kb], h, h, [0], Q, Q.clone(), 0.125, ws)
    Q = torch.zeros((1, 4, 64), device="cuda")
    with pytest.raises(J.JoltError):        # layer outside the cell
        J.jolt_attend(ctx(), [kb], [kb], h, h, [1], Q, Q.clone(), 0.125, ws)

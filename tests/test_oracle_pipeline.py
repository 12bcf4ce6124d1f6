"""Pins of the oracle's end-to-end cell path, blob format and budgeted mode."""
import numpy as np
import pytest

import kvsynth
from conftest import lowrank_cell
from oracle import alloc, pipeline as pl
from oracle.rounding import to_bf16


@pytest.fixture(scope="module")
def keys_cell():
    x = kvsynth.layer_kv(layer=0, tensor=0, n_heads=4, T=128, d=128, alpha=1.5)
    return x[0].astype(np.float64)


def test_full_rank_fp32_factors_nearly_lossless(keys_cell):           # P1 with rounding
    X = keys_cell
    out = pl.compress_cell(X, r_T=128, r_d=128, bits=8, group=64, factor_bytes=4)
    # fp32 factor rounding leaves a ~1e-7 residual; its fp16 scale underflows to
    # zero, so the residual stage can only keep or lower the error
    assert pl.rel_error(X, out["Xtilde"]) < 1e-6
    assert pl.rel_error(X, out["Xhat"]) <= pl.rel_error(X, out["Xtilde"])


def test_residual_bits_reduce_error(keys_cell):
    X = keys_cell
    errs = [pl.rel_error(X, pl.compress_cell(X, r_T=32, r_d=32, bits=b)["Xhat"])
            for b in (0, 2, 4, 8)]
    assert errs[0] > errs[1] > errs[2] > errs[3]


def test_closed_loop_residual_uses_stored_factors(keys_cell):
    """The residual is taken against the decoder's X~ (stored fp16 factors), so
    at b = 8 the only error left is the residual's quantisation error."""
    X = keys_cell
    out = pl.compress_cell(X, r_T=16, r_d=16, bits=8)
    R = X - out["Xtilde"]
    q_err = np.sum((out["Xhat"] - X) ** 2) / np.sum(R * R)
    assert q_err < 1e-4


def test_blob_roundtrip_and_decode(keys_cell):
    X = keys_cell
    for fb, bits in ((2, 2), (2, 0), (4, 4), (2, 8)):
        out = pl.compress_cell(X, r_T=24, r_d=40, bits=bits, factor_bytes=fb, seed=11)
        blob = pl.write_blob(out, in_dtype="bf16", n_heads=4)
        lay = pl.blob_layout(4, 128, 128, 24, 40, bits, 64, fb)
        assert len(blob) == lay["total"]
        assert all(lay[k] % 256 == 0 for k in ("UT", "Ud", "G", "gexp", "scales", "codes"))
        b = pl.read_blob(blob)
        assert (b["r_T"], b["r_d"], b["bits"], b["seed"]) == (24, 40, bits, 11)
        np.testing.assert_allclose(pl.decode_blob(blob), out["Xhat"], rtol=0, atol=1e-13)


def test_determinism_and_seed_dependence(keys_cell):                  # P15
    X = keys_cell
    a = pl.write_blob(pl.compress_cell(X, r_T=16, r_d=16, bits=4, seed=3), in_dtype="bf16", n_heads=4)
    b = pl.write_blob(pl.compress_cell(X, r_T=16, r_d=16, bits=4, seed=3), in_dtype="bf16", n_heads=4)
    c = pl.write_blob(pl.compress_cell(X, r_T=16, r_d=16, bits=4, seed=4), in_dtype="bf16", n_heads=4)
    assert a == b and a != c


def test_flash_cell_matches_exact_at_low_rank(rng):
    X = lowrank_cell(rng, 4, 256, 32, 6, noise=0.02)
    ex = pl.compress_cell(X, r_T=8, r_d=16, bits=4, group=16, method="exact")
    fl = pl.compress_cell(X, r_T=8, r_d=16, bits=4, group=16, method="flash", q=32, p=10,
                          power_iters=1)
    assert abs(pl.rel_error(X, ex["Xhat"]) - pl.rel_error(X, fl["Xhat"])) < 2e-3


def test_budgeted_cache_meets_budget_and_error_falls_with_budget():
    K, V = kvsynth.make_cache(n_layers=2, n_heads=2, T=64, d=32, alpha_K=1.5, alpha_V=0.7)
    cells = []
    for arr in (K, V):
        x = kvsynth.bf16_bits_to_f32(arr).astype(np.float64)      # [L][B][H][T][d]
        cells.append(x[:, 0].reshape(-1, 64, 32))
    eps2 = alloc.calibrate_eps2(group=32, d=32, n_samples=1 << 16)
    errs = []
    for ratio in (1.5, 2.0, 3.0):
        res = pl.compress_cells(cells, ratio=ratio, eps2=eps2, group=32)
        assert res["allocation"]["total_bytes"] <= res["budget"]
        errs.append(np.mean([pl.rel_error(X, p["Xhat"]) for X, p in zip(cells, res["parts"])]))
    assert errs[0] < errs[1] < errs[2]


def test_bf16_output_cast():
    x = np.array([1.0 + 2 ** -9, -3.0000001, 1e-3])
    np.testing.assert_array_equal(pl.cast_output(x, "bf16"), to_bf16(x))

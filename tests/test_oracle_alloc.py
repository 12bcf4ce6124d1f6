"""Pins of the oracle's byte model, cap policy and Lagrangian allocator (sections 4, 5, 8)."""
import itertools

import numpy as np
import pytest

from conftest import golden, lowrank_cell
from oracle import alloc, pipeline, tucker as tk


def test_byte_model_matches_paper_footprint():
    """Section 8: Mistral-7B at ctx-2048 occupies 268.4 MB uncompressed, and the compressed
    footprints at 2/3/4/8x land at the printed sizes (1.99-7.98x).  The oracle's own byte
    model prices the uncompressed cache (every entry at b = 16 bits, no factors) and its
    allocator, fed the cells of that cache (16 cells: 8 layer groups x K/V, 32 slices of
    2048 x 128) under budget = cache / R, never exceeds the budget and spends it to within
    2% (the Lagrangian dual only reaches points of each cell's lower convex hull, so with 16
    cells it can stop short of the budget: 2.008x, 3.000x, 4.074x and 8.044x here), while the
    paper's printed footprints sit within 0.5% of cache / R."""
    g = golden("paper_memory_footprint.json")
    mdl = g["model"]
    group_layers = 4
    m = group_layers * mdl["kv_heads"]
    n_cells = 2 * mdl["layers"] // group_layers
    T, d, c = mdl["ctx"], mdl["head_dim"], mdl["bytes_per_scalar"]
    # uncompressed: eq. (1) with no factors and 8 c bits per entry, no scale term
    per_cell = alloc.byte_cost(m, T, d, 0, 0, 8 * c, c, 64, count_scales=False)
    total = n_cells * per_cell
    assert round(total / 1e6, 1) == g["uncompressed_MB"]
    # spectra of that shape (power laws, a different decay per cell), the paper's group 64
    rng = np.random.default_rng(0)
    cells = []
    for i in range(n_cells):
        aT, ad = rng.uniform(0.8, 1.6), rng.uniform(0.5, 1.5)
        lam_T = np.arange(1, T + 1, dtype=np.float64) ** -aT
        lam_d = np.arange(1, d + 1, dtype=np.float64) ** -ad
        lam_d *= lam_T.sum() / lam_d.sum()
        cells.append(alloc.CellSpectrum(m=m, T=T, d=d, c=c, g=64, E=float(lam_T.sum()),
                                        lam_T=lam_T, lam_d=lam_d, rT_max=T))
    eps2 = {0: 1.0, 2: 0.26, 4: 0.010, 8: 3.5e-5}
    lo, hi = g["achieved_ratio_range"]
    assert lo <= min(map(float, g["compressed_MB"])) and max(map(float, g["compressed_MB"])) <= hi + 0.05
    for R, mb in g["compressed_MB"].items():
        res = alloc.allocate(cells, total / float(R), eps2)
        assert not res["infeasible"]
        spent = alloc.allocation_cost(cells, res["alloc"])
        assert spent == res["total_bytes"] <= total / float(R)
        achieved = total / spent
        assert achieved >= float(R) and achieved / float(R) - 1 < 0.02, (R, achieved)
        # the paper's printed footprint, priced against the same uncompressed bytes
        assert abs(total / (mb * 1e6) / float(R) - 1) < 0.005
        assert lo - 0.005 <= total / (mb * 1e6) <= hi + 0.005


def test_byte_cost_eq1_terms():
    """eq. (1): core m r_T r_d, token factor T r_T, feature factor d r_d scalars at
    c bytes, plus b/8 bytes per cached entry; scales add 2 bytes per group."""
    m, T, d = 8, 256, 128
    assert alloc.byte_cost(m, T, d, 0, 0, 0, 2, 64) == 0
    assert alloc.byte_cost(m, T, d, 64, 64, 0, 4, 64) == (8 * 64 * 64 + 256 * 64 + 128 * 64) * 4
    assert alloc.byte_cost(m, T, d, 0, 0, 4, 2, 64, count_scales=False) == m * T * d // 2
    assert alloc.byte_cost(m, T, d, 64, 64, 2, 4, 64) == 229376 + 65536 + 8192
    # doubling every rank roughly quadruples the core term only
    a = alloc.byte_cost(m, T, d, 16, 16, 0, 2, 64)
    b = alloc.byte_cost(m, T, d, 32, 32, 0, 2, 64)
    assert b - 2 * a == 2 * m * 16 * 16 * 2


def test_cap_policy_matches_paper():
    for c in golden("paper_cap_policy.json")["cases"]:
        assert alloc.q_cap(c["T"], c["R"]) == c["q"], c
    for T in (64, 256, 512, 1000, 1024):       # "a no-op for T <= 1024"
        assert alloc.q_cap(T, 2) == 32 and alloc.q_cap(T, 6) == 64
    qs = [alloc.q_cap(T, 3) for T in range(1, 40000, 97)]
    assert (np.diff(qs) >= 0).all() and max(qs) == 512


def _cells(rng, n, m=2, T=24, d=16):
    out = []
    for i in range(n):
        X = lowrank_cell(rng, m, T, d, 4, noise=0.2 + 0.3 * i, decay=0.5 + i)
        sp = pipeline.spectrum(X)
        out.append(alloc.CellSpectrum(m=m, T=T, d=d, c=2, g=8, E=sp["E"], lam_T=sp["lam_T"],
                                      lam_d=sp["lam_d"], rT_max=T))
    return out


def _enumerate(cells, eps2, step):
    per = []
    for c in cells:
        opts = [(0, 0, b) for b in alloc.BIT_GRID]
        opts += [(rT, rd, b) for rT in range(step, c.rT_max + 1, step)
                 for rd in range(step, c.d + 1, step) for b in alloc.BIT_GRID]
        tauT = tk.tail_fractions(c.lam_T, c.E)
        taud = tk.tail_fractions(c.lam_d, c.E)
        per.append([(alloc.byte_cost(c.m, c.T, c.d, rT, rd, b, c.c, c.g),
                     eps2[b] * min(1.0, tauT[rT] + taud[rd]), (rT, rd, b)) for rT, rd, b in opts])
    return per


def test_everett_optimality_against_brute_force(rng):                 # P11
    eps2 = {0: 1.0, 2: 0.26, 4: 0.0101, 8: 3.5e-5}
    cells = _cells(rng, 3)
    per = _enumerate(cells, eps2, 8)
    total_in = sum(c.m * c.T * c.d * 2 for c in cells)
    for ratio in (1.5, 2.0, 3.0, 5.0, 9.0):
        res = alloc.allocate(cells, total_in / ratio, eps2)
        S = res["total_bytes"]
        assert S <= total_in / ratio
        # no allocation that spends at most S bytes has a smaller summed model error
        best = min(sum(p[1] for p in combo) for combo in itertools.product(*per)
                   if sum(p[0] for p in combo) <= S)
        assert res["model_error"] <= best + 1e-15


def test_spend_nonincreasing_in_lambda(rng):
    eps2 = {0: 1.0, 2: 0.26, 4: 0.0101, 8: 3.5e-5}
    cells = _cells(rng, 4)
    total_in = sum(c.m * c.T * c.d * 2 for c in cells)
    spends = []
    for ratio in (1.2, 1.5, 2, 3, 4, 6, 10, 20):
        spends.append(alloc.allocate(cells, total_in / ratio, eps2)["total_bytes"])
    assert (np.diff(spends) <= 0).all()


def test_generous_budget_gives_min_error_and_tiny_budget_flags(rng):
    eps2 = {0: 1.0, 2: 0.26, 4: 0.0101, 8: 3.5e-5}
    cells = _cells(rng, 2)
    res = alloc.allocate(cells, 1e12, eps2)
    assert res["lam"] == 0.0 and res["model_error"] <= 1e-12
    tiny = alloc.allocate(cells, 1.0, eps2, floors=(8, 8, 0))
    assert tiny["infeasible"] and all(a[0] >= 8 for a in tiny["alloc"])
    zero = alloc.allocate(cells, 0.0, eps2)
    assert not zero["infeasible"] and zero["alloc"] == [(0, 0, 0)] * 2


# ------------------------------------------------------------------ ablation allocators (section 7)
EPS2 = {0: 1.0, 2: 0.26, 4: 0.0101, 8: 3.5e-5}


def test_rank_only_is_the_optimum_without_residual(rng):
    """Rank-only spends nothing on residual bits and, at the bytes it spends, no
    residual-free allocation has a smaller summed model error (brute force)."""
    cells = _cells(rng, 3)
    per = [[p for p in grid if p[2][2] == 0] for grid in _enumerate(cells, EPS2, 8)]
    total_in = sum(c.m * c.T * c.d * 2 for c in cells)
    for ratio in (2.0, 4.0, 8.0):
        res = alloc.allocate(cells, total_in / ratio, EPS2, bits=(0,))
        assert all(b == 0 for _, _, b in res["alloc"])
        best = min(sum(p[1] for p in combo) for combo in itertools.product(*per)
                   if sum(p[0] for p in combo) <= res["total_bytes"])
        assert res["model_error"] <= best + 1e-15


def test_greedy_single_cell_takes_the_best_point_within_budget(rng):
    """With one cell the frontier walk stops at the least-error point that fits: the
    brute-force optimum of a single cell."""
    cell = _cells(rng, 1)
    per = _enumerate(cell, EPS2, 8)[0]
    full = cell[0].m * cell[0].T * cell[0].d * 2
    for ratio in (1.3, 2.0, 3.0, 5.0, 12.0):
        B = full / ratio
        res = alloc.allocate_greedy(cell, B, EPS2, [0])
        best = min(p[1] for p in per if p[0] <= B)
        assert res["total_bytes"] <= B
        assert res["model_error"] == best


def test_greedy_pools_spend_their_own_share(rng):
    """Keys and values are separate pools: each spends at most its share of the budget,
    and changing one pool's cells leaves the other pool's allocation unchanged."""
    cells = _cells(rng, 4)
    pools = [0, 0, 1, 1]
    total_in = sum(c.m * c.T * c.d * 2 for c in cells)
    for ratio in (2.0, 4.0):
        B = total_in / ratio
        res = alloc.allocate_greedy(cells, B, EPS2, pools)
        spend = [alloc.byte_cost(c.m, c.T, c.d, rT, rd, b, c.c, c.g)
                 for c, (rT, rd, b) in zip(cells, res["alloc"])]
        assert spend[0] + spend[1] <= B / 2 and spend[2] + spend[3] <= B / 2
        other = _cells(np.random.default_rng(99), 4)
        res2 = alloc.allocate_greedy(cells[:2] + other[2:], B, EPS2, pools)
        assert res2["alloc"][:2] == res["alloc"][:2]
    # the joint dual may move bytes between the pools and is never worse on the model
    # error at the bytes it spends than any allocation within those bytes (Everett)
    j = alloc.allocate(cells, total_in / 4.0, EPS2)
    g = alloc.allocate_greedy(cells, total_in / 4.0, EPS2, pools)
    if g["total_bytes"] <= j["total_bytes"]:
        assert j["model_error"] <= g["model_error"] + 1e-15


def test_uniform_is_the_best_shared_point(rng):
    """Uniform rank: every cell gets the same (r_T, r_d, b), the shared point of least
    summed model error that fits the budget (brute force over the shared points)."""
    cells = _cells(rng, 3)
    per = _enumerate(cells, EPS2, 8)
    total_in = sum(c.m * c.T * c.d * 2 for c in cells)
    for ratio in (1.5, 3.0, 6.0):
        B = total_in / ratio
        res = alloc.allocate_uniform(cells, B, EPS2)
        assert len(set(res["alloc"])) == 1
        shared = [(sum(g[k][0] for g in per), sum(g[k][1] for g in per)) for k in range(len(per[0]))]
        best = min(e for s, e in shared if s <= B)
        assert res["total_bytes"] <= B and res["model_error"] == pytest.approx(best, rel=0, abs=1e-15)

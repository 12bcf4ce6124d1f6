"""Joint Lagrangian allocation of Tucker ranks and residual bits (fp64 oracle).

Section 4, "Joint Lagrangian allocation":

* eq. (1) byte cost of a cell at (r_T, r_d, b):
  s = (m r_T r_d + T r_T + d r_d) c + (b/8) m T d, plus - in this library's
  reading - 2 bytes per quantiser group for the fp16 scales the paper calls a
  negligible per-row term (switchable);
* eq. (2) error model e = eps^2(b) * tau(r_T, r_d), with eps^2(0) = 1 and
  eps^2(b) calibrated once on a Gaussian round trip; tau is the relative
  Frobenius mass the truncation discards, read by default as
  min(1, tau_T(r_T) + tau_d(r_d)) from the mode spectra of the original cell
  (the ST-HOSVD upper bound; (0, 0) discards everything, tau = 1).  When the
  cell carries the truncated feature spectra mu (row k: r_T = (k + 1) step,
  see tucker.truncated_feature_spectra) tau is the exact ST-HOSVD value
  (E - sum_{i < r_d} mu_k[i]) / E and the r_T grid stops at the table's end;
* eq. (3) minimise the summed error subject to the summed cost <= B;
* eq. (4) Lagrangian relaxation: for fixed lambda each cell minimises
  e + lambda s over its finite grid independently, and one bisection on
  lambda drives the total cost to the budget.

Section 5, "Cap selection": q_cap = min(max(q_min(R), ceil(T/32)), 512) with
q_min = 32 for R <= 4 and 64 otherwise.

Deterministic conventions (so that two independent implementations agree
bit for bit on the same spectra):

* grid: r_T in {0} U {k*step <= r_T_max}, r_d in {k*step <= d} (r_d = 0 only
  with r_T = 0), b in the bit grid; optional floors restrict it;
* grid points are ordered by (cost, bits, r_T, r_d) and a cell takes the first
  point of minimal e + lambda s in that order (ties go to the cheaper point);
* e = eps2[b] * min(1, tau_T[r_T] + tau_d[r_d]); value = e + lambda * s, all in
  IEEE double without fused multiply-add;
* bisection on lambda in [0, 1e3]: if the lambda = 0 allocation fits, it is
  returned; if even lambda = 1e3 (the cheapest allocation) does not fit, that
  allocation is returned with the infeasible flag set; otherwise
  mid = 0.5 (lo + hi) replaces hi when S(mid) <= B and lo otherwise, until
  hi - lo <= 1e-15 hi or 200 halvings, and the allocation at hi is returned.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .philox import calibration_samples, rotation_signs
from .residual import residual_roundtrip
from .tucker import tail_fractions

BIT_GRID = (0, 2, 4, 8)
LAMBDA_HI = 1e3
MAX_HALVINGS = 200


def q_cap(T: int, R: float) -> int:
    q_min = 32 if R <= 4 else 64
    return int(min(max(q_min, math.ceil(T / 32)), 512))


def byte_cost(m: int, T: int, d: int, r_T: int, r_d: int, b: int, c: int, g: int,
              count_scales: bool = True) -> int:
    s = (m * r_T * r_d + T * r_T + d * r_d) * c
    if b > 0:
        s += (b * m * T * d) // 8
        if count_scales:
            s += 2 * ((m * T * d) // g)
    return int(s)


@dataclass
class CellSpectrum:
    m: int
    T: int
    d: int
    c: int                 # bytes per stored factor scalar
    g: int                 # quantiser group size
    E: float
    lam_T: np.ndarray      # token-mode eigenvalues (flash: q_eff values + tail)
    lam_d: np.ndarray      # feature-mode eigenvalues (d values)
    rT_max: int            # largest admissible token rank
    extra: dict = field(default_factory=dict)
    mu: np.ndarray | None = None   # K x d truncated feature spectra (exact tau) or None


def st_tau_table(E: float, mu: np.ndarray) -> np.ndarray:
    """Exact ST-HOSVD tau: tab[k][r_d] = (E - sum_{i < r_d} mu[k][i]) / E in [0, 1].

    The head sums run from i = 0 upward, one term at a time; E = 0 gives 0.
    """
    K, d = mu.shape
    tab = np.zeros((K, d + 1))
    if not E > 0.0:
        return tab
    for k in range(K):
        acc = 0.0
        tab[k][0] = 1.0
        for i in range(d):
            acc += float(mu[k][i])
            tab[k][i + 1] = min(1.0, max(0.0, (E - acc) / E))
    return tab


def cell_grid(cell, eps2: dict, *, bits=BIT_GRID, step: int = 8, floors=(0, 0, 0),
              count_scales: bool = True):
    """Grid points of one cell ordered by (cost, b, r_T, r_d): arrays s, e and P = [s, b, r_T, r_d]."""
    tau_T = tail_fractions(cell.lam_T, cell.E)
    tau_d = tail_fractions(cell.lam_d, cell.E)
    fT, fd, fb = floors
    rT_hi = cell.rT_max
    if cell.mu is not None:
        tab = st_tau_table(cell.E, np.asarray(cell.mu, dtype=np.float64))
        rT_hi = min(rT_hi, step * tab.shape[0])
    rTs = [0] + list(range(step, rT_hi + 1, step))
    rds = list(range(step, cell.d + 1, step))
    pts = []
    for b in bits:
        if b < fb:
            continue
        for rT in rTs:
            if rT < fT:
                continue
            for rd in ([0] if rT == 0 else rds):
                if rT > 0 and rd < fd:
                    continue
                pts.append((byte_cost(cell.m, cell.T, cell.d, rT, rd, b, cell.c,
                                      cell.g, count_scales), b, rT, rd))
    if not pts:
        raise ValueError("empty allocation grid (floors exclude every point)")
    pts.sort()
    P = np.array(pts, dtype=np.int64)
    s = P[:, 0].astype(np.float64)
    eb = np.array([float(eps2[int(x)]) for x in P[:, 1]])
    if cell.mu is None:
        tau = np.minimum(1.0, tau_T[P[:, 2]] + tau_d[P[:, 3]])
    else:
        tau = np.array([(1.0 if cell.E > 0.0 else 0.0) if rT == 0 else tab[rT // step - 1][rd]
                        for rT, rd in zip(P[:, 2], P[:, 3])])
    e = eb * tau
    return s, e, P


def _result(grids, idx, lam, infeasible):
    alloc = [tuple(int(v) for v in g[2][i][[2, 3, 1]]) for g, i in zip(grids, idx)]
    total = float(sum(g[0][i] for g, i in zip(grids, idx)))
    err = float(sum(g[1][i] for g, i in zip(grids, idx)))
    return dict(alloc=alloc, lam=lam, total_bytes=total, model_error=err,
                infeasible=infeasible)


def allocate(cells, budget: float, eps2: dict, *, bits=BIT_GRID, step: int = 8,
             floors=(0, 0, 0), count_scales: bool = True):
    """Solve eq. (3) through eq. (4); returns dict(alloc=[(r_T, r_d, b)], ...)."""
    grids = [cell_grid(c, eps2, bits=bits, step=step, floors=floors, count_scales=count_scales)
             for c in cells]

    def choose(lam):
        idx = [int(np.argmin(e + lam * s)) for (s, e, _) in grids]
        total = float(sum(g[0][i] for g, i in zip(grids, idx)))
        return idx, total

    idx0, S0 = choose(0.0)
    if S0 <= budget:
        return _result(grids, idx0, 0.0, False)
    lo, hi = 0.0, LAMBDA_HI
    idx_hi, S_hi = choose(hi)
    if S_hi > budget:
        return _result(grids, idx_hi, hi, True)
    for _ in range(MAX_HALVINGS):
        if hi - lo <= 1e-15 * hi:
            break
        mid = 0.5 * (lo + hi)
        idx_mid, S_mid = choose(mid)
        if S_mid <= budget:
            hi, idx_hi = mid, idx_mid
        else:
            lo = mid
    return _result(grids, idx_hi, hi, False)


# --------------------------------------------------------------------- ablation allocators
# Section 7 ablations (A1, A5) compare the joint dual with three simpler schemes.  The
# paper describes them in words; the readings written out here (identically in the
# library) are:
#
# * rank-only: the joint dual with no residual, i.e. the bit grid {0};
# * greedy: every cell starts at its cheapest grid point and repeatedly takes the upgrade,
#   among all cells, with the largest error reduction per extra byte.  A cell's upgrades
#   walk its Pareto frontier (the points, in grid order, whose error is below that of
#   every cheaper point), one frontier point at a time; an upgrade that would exceed the
#   remaining budget is skipped.  There is no global multiplier: the cells are split into
#   pools (keys and values) and each pool spends its own share of the budget, in
#   proportion to its cells' m T d.  Equal efficiencies go to the lower cell index; an
#   upgrade of zero extra bytes is taken first;
# * uniform: one (r_T, r_d, b) shared by every cell, the one of least summed error whose
#   summed cost fits the budget (ties to the smaller cost, then b, r_T, r_d).
def _pareto(s, e):
    keep, best = [], math.inf
    for k in range(len(s)):
        if e[k] < best:
            keep.append(k)
            best = e[k]
    return keep


def allocate_greedy(cells, budget: float, eps2: dict, pools, *, bits=BIT_GRID, step: int = 8,
                    floors=(0, 0, 0), count_scales: bool = True):
    grids = [cell_grid(c, eps2, bits=bits, step=step, floors=floors, count_scales=count_scales)
             for c in cells]
    fronts = [_pareto(g[0], g[1]) for g in grids]
    cur = [0] * len(cells)
    size = [c.m * c.T * c.d for c in cells]
    total_size = sum(size)
    infeasible = False
    for pool in sorted(set(pools)):
        members = [i for i, p in enumerate(pools) if p == pool]
        share = budget * sum(size[i] for i in members) / total_size
        spent = sum(grids[i][0][fronts[i][0]] for i in members)
        if spent > share:
            infeasible = True
            continue
        while True:
            best, best_eff = -1, -math.inf
            for i in members:
                f = fronts[i]
                if cur[i] + 1 >= len(f):
                    continue
                k0, k1 = f[cur[i]], f[cur[i] + 1]
                ds = grids[i][0][k1] - grids[i][0][k0]
                if spent + ds > share:
                    continue
                de = grids[i][1][k0] - grids[i][1][k1]
                eff = math.inf if ds == 0 else de / ds
                if eff > best_eff:
                    best, best_eff = i, eff
            if best < 0:
                break
            f = fronts[best]
            spent += grids[best][0][f[cur[best] + 1]] - grids[best][0][f[cur[best]]]
            cur[best] += 1
    idx = [fronts[i][cur[i]] for i in range(len(cells))]
    return _result(grids, idx, 0.0, infeasible)


def allocate_uniform(cells, budget: float, eps2: dict, *, bits=BIT_GRID, step: int = 8,
                     floors=(0, 0, 0), count_scales: bool = True):
    grids = [cell_grid(c, eps2, bits=bits, step=step, floors=floors, count_scales=count_scales)
             for c in cells]
    where = []
    for s, e, P in grids:
        where.append({(int(b), int(rT), int(rd)): k for k, (_, b, rT, rd) in enumerate(P)})
    common = set(where[0])
    for w in where[1:]:
        common &= set(w)
    cands = []
    for t in common:
        S = 0.0
        Err = 0.0
        for g, w in zip(grids, where):
            S += g[0][w[t]]
            Err += g[1][w[t]]
        cands.append((S, t[0], t[1], t[2], Err))
    if not cands:
        raise ValueError("no grid point common to every cell")
    cands.sort()
    fit = [c for c in cands if c[0] <= budget]
    infeasible = not fit
    if fit:
        pick, best = None, math.inf
        for c in fit:
            if c[4] < best:
                pick, best = c, c[4]
    else:
        pick = cands[0]
    t = (pick[1], pick[2], pick[3])
    return _result(grids, [w[t] for w in where], 0.0, infeasible)


def allocation_cost(cells, alloc, *, count_scales=True) -> float:
    return float(sum(byte_cost(c.m, c.T, c.d, rT, rd, b, c.c, c.g, count_scales)
                     for c, (rT, rd, b) in zip(cells, alloc)))


def calibrate_eps2(*, group: int, d: int, seed: int = 0, n_samples: int = 1 << 20,
                   bits=(2, 4, 8)) -> dict:
    """eps^2(b) = ||x^ - x||^2 / ||x||^2 of a Gaussian round trip (eq. (2) calibration)."""
    x = calibration_samples(seed, n_samples).reshape(-1, d)
    signs = rotation_signs(seed, d)
    out = {0: 1.0}
    den = float(np.sum(x * x))
    for b in bits:
        xh = residual_roundtrip(x, signs, b, group)
        out[b] = float(np.sum((xh - x) ** 2)) / den
    return out

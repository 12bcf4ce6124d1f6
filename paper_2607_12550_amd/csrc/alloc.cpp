// Joint Lagrangian allocation of Tucker ranks and residual bits (section 4,
// eq. (1)-(4)); host only.
//
// Cost (eq. (1)):  s = (m r_T r_d + T r_T + d r_d) c + [b > 0] (b m T d / 8 + 2 m T d / g)
//                  (the scale term is optional: the paper treats it as negligible).
// Error (eq. (2)): e = eps2(b) * tau(r_T, r_d).  By default tau = min(1, tau_T(r_T) +
//                  tau_d(r_d)) from the mode spectra of the cell, tau(r) = (sum of
//                  eigenvalues past r) / E (the ST-HOSVD bound).  With the truncated
//                  feature spectra mu_k of the cell (row k at r_T = (k + 1) step) tau is
//                  the exact discarded mass (E - sum_{i < r_d} mu_k[i]) / E, head sums
//                  accumulated from i = 0 upward, clipped to [0, 1].
// Problem (eq. (3)) is solved through the relaxation of eq. (4): for a fixed lambda
// every cell independently takes the grid point minimising e + lambda s, and one
// bisection on lambda drives the total cost to the budget.
//
// Determinism: grid points are ordered by (cost, bits, r_T, r_d) and the first
// point of minimal value wins; tails are suffix sums accumulated from the smallest
// eigenvalue upward; the bisection halves [0, 1e3] until hi - lo <= 1e-15 hi (at
// most 200 halvings) and returns the allocation at hi.  This file is compiled
// without floating-point contraction so the arithmetic is plain IEEE double.
//
// Speed: the grids of the cells are built and sorted (one 64-bit key per point holding the
// cost and the generation index, so an unstable sort yields the stable order), and each
// bisection step evaluated, on up to 16 host threads (each cell by one thread, totals summed
// in cell order, so the result does not depend on the split; a bisection step over small
// frontiers runs on the calling thread), and each bisection step scans only the Pareto
// frontier of a grid.  A point q off the frontier has an earlier
// point p with s_p <= s_q and e_p <= e_q; rounding is monotone, so for every lambda >= 0
// e_p + lambda s_p <= e_q + lambda s_q in floating point too, and q can never be the first
// point of minimal value: the scan over the frontier returns what the full scan returns.
//
// The ablation allocators of section 7 (rank-only, greedy, uniform rank) use the same
// grid, costs and model errors; their definitions are stated with JOLT_ALLOC_* in the
// public header.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <map>
#include <atomic>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <set>
#include <thread>
#include <tuple>
#include <vector>

#include "../../include/jolt.h"
#include "host_util.h"

namespace {

struct Point {
  int64_t s;
  int32_t b, rT, rd;
  double e;
};

std::vector<double> tail_fractions(const double *lam, int n, double E) {
  std::vector<double> suf(n + 1, 0.0);
  double acc = 0.0;
  for (int i = n - 1; i >= 0; --i) {
    acc += lam[i];
    suf[i] = acc;
  }
  if (!(E > 0.0)) return std::vector<double>(n + 1, 0.0);
  for (int i = 0; i <= n; ++i) suf[i] = suf[i] / E;
  return suf;
}

// exact ST-HOSVD tau, n_mu rows of d + 1: tab[k][r_d] = (E - sum_{i < r_d} mu_k[i]) / E
std::vector<double> exact_tau_table(const double *mu, int n_mu, int d, double E) {
  std::vector<double> tab((size_t)std::max(n_mu, 0) * (d + 1), 0.0);
  if (!(E > 0.0)) return tab;
  for (int k = 0; k < n_mu; ++k) {
    double acc = 0.0;
    double *row = tab.data() + (size_t)k * (d + 1);
    row[0] = 1.0;
    for (int i = 0; i < d; ++i) {
      acc += mu[(size_t)k * d + i];
      row[i + 1] = std::min(1.0, std::max(0.0, (E - acc) / E));
    }
  }
  return tab;
}

int64_t byte_cost(int64_t m, int64_t T, int64_t d, int64_t rT, int64_t rd, int64_t b, int64_t c,
                  int64_t g, bool scales) {
  int64_t s = (m * rT * rd + T * rT + d * rd) * c;
  if (b > 0) {
    s += (b * m * T * d) / 8;
    if (scales) s += 2 * ((m * T * d) / g);
  }
  return s;
}

// Runs a per-cell task for cells 0 .. n-1 on the calling thread and nthr - 1 workers that
// persist across run() calls; run() returns when every cell is done.
class CellPool {
 public:
  CellPool(int nthr, int n) : n_(n) {
    for (int t = 1; t < nthr; ++t) workers_.emplace_back([this] { loop(); });
  }
  ~CellPool() {
    {
      std::lock_guard<std::mutex> g(mu_);
      stop_ = true;
      ++gen_;
    }
    cv_.notify_all();
    for (auto &w : workers_) w.join();
  }
  void run(const std::function<void(int)> &f) {
    {
      std::lock_guard<std::mutex> g(mu_);
      task_ = &f;
      next_ = 0;
      busy_ = (int)workers_.size();
      ++gen_;
    }
    cv_.notify_all();
    drain(f);
    std::unique_lock<std::mutex> g(mu_);
    done_.wait(g, [this] { return busy_ == 0; });
    task_ = nullptr;
  }

 private:
  void drain(const std::function<void(int)> &f) {
    for (int ci = next_++; ci < n_; ci = next_++) f(ci);
  }
  void loop() {
    uint64_t seen = 0;
    for (;;) {
      const std::function<void(int)> *f;
      {
        std::unique_lock<std::mutex> g(mu_);
        cv_.wait(g, [&] { return gen_ != seen; });
        seen = gen_;
        if (stop_) return;
        f = task_;
      }
      drain(*f);
      {
        std::lock_guard<std::mutex> g(mu_);
        if (--busy_ == 0) done_.notify_one();
      }
    }
  }
  const int n_;
  std::vector<std::thread> workers_;
  std::mutex mu_;
  std::condition_variable cv_, done_;
  const std::function<void(int)> *task_ = nullptr;
  std::atomic<int> next_{0};
  int busy_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

// Ascending sort of keys below 2^bits (LSD radix, 11-bit digits).
void radix_sort(std::vector<uint64_t> &key, int bits) {
  constexpr int DB = 11, NB = 1 << DB;
  std::vector<uint64_t> tmp(key.size());
  uint32_t cnt[NB];
  for (int sh = 0; sh < bits; sh += DB) {
    std::fill(cnt, cnt + NB, 0u);
    for (uint64_t k : key) ++cnt[(k >> sh) & (NB - 1)];
    uint32_t pos = 0;
    for (uint32_t &c : cnt) { const uint32_t n = c; c = pos; pos += n; }
    for (uint64_t k : key) tmp[cnt[(k >> sh) & (NB - 1)]++] = k;
    key.swap(tmp);
  }
}

// Pareto frontier of a grid in grid order: the points whose error is below that of every
// earlier (cheaper or equal-cost, earlier-ordered) point
std::vector<int> pareto(const std::vector<Point> &pts) {
  std::vector<int> keep;
  double best = std::numeric_limits<double>::infinity();
  for (int k = 0; k < (int)pts.size(); ++k)
    if (pts[k].e < best) { keep.push_back(k); best = pts[k].e; }
  return keep;
}

}  // namespace

extern "C" int jolt_allocate(const jolt_cell_spectrum *cells, int n_cells, const jolt_alloc_opts *o,
                             int32_t *r_T, int32_t *r_d, int32_t *bits, double *lambda_star,
                             double *total_bytes, double *model_error, int32_t *infeasible) {
  if (!cells || !o || !r_T || !r_d || !bits || n_cells < 0)
    return jolt_fail(JOLT_E_INVAL, "jolt_allocate: null argument or negative cell count");
  if (o->step < 1) return jolt_fail(JOLT_E_INVAL, "jolt_allocate: step must be >= 1");
  if (!(o->budget_bytes >= 0.0)) return jolt_fail(JOLT_E_INVAL, "jolt_allocate: budget must be >= 0");
  if (o->strategy < JOLT_ALLOC_JOINT || o->strategy > JOLT_ALLOC_UNIFORM)
    return jolt_fail(JOLT_E_INVAL, "jolt_allocate: unknown strategy %d", o->strategy);
  const int bit_values[4] = {0, 2, 4, 8};
  const int mask = o->strategy == JOLT_ALLOC_RANK_ONLY ? (o->bit_mask & 1) : o->bit_mask;
  std::vector<std::vector<Point>> grids(n_cells);
  for (int ci = 0; ci < n_cells; ++ci) {
    const jolt_cell_spectrum &c = cells[ci];
    if (c.m < 1 || c.T < 1 || c.d < 1 || (c.c != 2 && c.c != 4) || c.g < 1 || c.n_lam_T < 1 ||
        c.rT_max < 0 || c.rT_max > c.n_lam_T || !c.lam_T || !c.lam_d)
      return jolt_fail(JOLT_E_INVAL, "jolt_allocate: malformed cell spectrum %d", ci);
    if (c.n_mu < 0 || (c.n_mu > 0 && !c.mu))
      return jolt_fail(JOLT_E_INVAL, "jolt_allocate: malformed truncated spectra of cell %d", ci);
  }
  // grid of one cell, sorted in grid order
  auto build = [&](int ci) {
    const jolt_cell_spectrum &c = cells[ci];
    const std::vector<double> tT = tail_fractions(c.lam_T, c.n_lam_T, c.E);
    const std::vector<double> td = tail_fractions(c.lam_d, c.d, c.E);
    const std::vector<double> tx = exact_tau_table(c.mu, c.n_mu, c.d, c.E);
    const int rT_hi = c.n_mu > 0 ? std::min<int64_t>(c.rT_max, (int64_t)c.n_mu * o->step) : c.rT_max;
    std::vector<Point> &pts = grids[ci];
    pts.reserve((size_t)4 * (rT_hi / o->step + 1) * (c.d / o->step + 1));
    for (int bi = 0; bi < 4; ++bi) {
      if (!(mask & (1 << bi))) continue;
      const int b = bit_values[bi];
      if (b < o->floor_bits) continue;
      const int step = o->step, rd0 = std::max(step, (o->floor_rd + step - 1) / step * step);
      // the residual's cost, the same at every (r_T, r_d): s = backbone cost + res
      const int64_t res = byte_cost(c.m, c.T, c.d, 0, 0, b, c.c, c.g, o->count_scale_bytes != 0);
      std::vector<int> rTs{0};
      for (int r = o->step; r <= rT_hi; r += o->step) rTs.push_back(r);
      for (int rT : rTs) {
        if (rT < o->floor_rT) continue;
        if (rT == 0) {
          Point p{res, b, 0, 0, 0.0};
          const double tau = c.n_mu > 0 ? (c.E > 0.0 ? 1.0 : 0.0) : std::min(1.0, tT[0] + td[0]);
          p.e = o->eps2[bi] * tau;
          pts.push_back(p);
          continue;
        }
        const int64_t s_rT = (int64_t)c.T * rT, s_rd = (int64_t)c.m * rT + c.d;   // s = (s_rT + s_rd rd) c + res
        const double eps = o->eps2[bi], tT_r = tT[rT];
        const double *txr = c.n_mu > 0 ? tx.data() + (size_t)(rT / step - 1) * (c.d + 1) : nullptr;
        for (int rd = rd0; rd <= c.d; rd += step) {
          const double tau = txr ? txr[rd] : std::min(1.0, tT_r + td[rd]);
          pts.push_back(Point{(s_rT + s_rd * rd) * c.c + res, b, rT, rd, eps * tau});
        }
      }
    }
    // the points were made in (b, r_T, r_d) order, so ordering by (s, generation index) gives
    // grid order; both go into one 64-bit key when s leaves room for the index
    const size_t np = pts.size();
    int gb = 1;
    while (((size_t)1 << gb) < np) ++gb;
    int64_t smax = 0;
    for (const Point &q : pts) smax = std::max(smax, q.s);
    if (smax >= 0 && gb < 40 && (uint64_t)smax < ((uint64_t)1 << (63 - gb))) {
      std::vector<uint64_t> key(np);
      for (size_t k = 0; k < np; ++k) key[k] = ((uint64_t)pts[k].s << gb) | (uint64_t)k;
      radix_sort(key, 64 - __builtin_clzll(((uint64_t)smax << gb) | ((uint64_t)1 << gb)));
      std::vector<Point> sorted(np);
      const uint64_t low = ((uint64_t)1 << gb) - 1;
      for (size_t k = 0; k < np; ++k) sorted[k] = pts[key[k] & low];
      pts.swap(sorted);
    } else {
      std::stable_sort(pts.begin(), pts.end(), [](const Point &a, const Point &b) { return a.s < b.s; });
    }
  };
  const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
  CellPool pool(std::max(1, std::min<int>(n_cells, (int)std::min(16u, hw))), n_cells);
  pool.run(build);
  for (int ci = 0; ci < n_cells; ++ci)
    if (grids[ci].empty()) return jolt_fail(JOLT_E_INVAL, "jolt_allocate: empty grid for cell %d", ci);
  std::vector<int> idx(n_cells), idx_hi(n_cells);
  auto emit = [&](const std::vector<int> &sel, double lam, int infeas) {
    double tb = 0.0, te = 0.0;
    for (int ci = 0; ci < n_cells; ++ci) {
      const Point &p = grids[ci][sel[ci]];
      r_T[ci] = p.rT; r_d[ci] = p.rd; bits[ci] = p.b;
      tb += (double)p.s; te += p.e;
    }
    if (lambda_star) *lambda_star = lam;
    if (total_bytes) *total_bytes = tb;
    if (model_error) *model_error = te;
    if (infeasible) *infeasible = infeas;
    return JOLT_OK;
  };
  const double B = o->budget_bytes;
  if (o->strategy == JOLT_ALLOC_GREEDY) {
    std::vector<std::vector<int>> front(n_cells);
    for (int ci = 0; ci < n_cells; ++ci) front[ci] = pareto(grids[ci]);
    std::vector<int> cur(n_cells, 0);
    double total_size = 0.0;
    for (int ci = 0; ci < n_cells; ++ci) total_size += (double)cells[ci].m * cells[ci].T * cells[ci].d;
    std::set<int> pools;
    for (int ci = 0; ci < n_cells; ++ci) pools.insert(cells[ci].pool);
    int infeas = 0;
    for (int pool : pools) {
      std::vector<int> mem;
      double size = 0.0, spent = 0.0;
      for (int ci = 0; ci < n_cells; ++ci)
        if (cells[ci].pool == pool) {
          mem.push_back(ci);
          size += (double)cells[ci].m * cells[ci].T * cells[ci].d;
        }
      const double share = B * size / total_size;
      for (int ci : mem) spent += (double)grids[ci][front[ci][0]].s;
      if (spent > share) { infeas = 1; continue; }
      for (;;) {
        int best = -1;
        double best_eff = -std::numeric_limits<double>::infinity();
        for (int ci : mem) {
          const std::vector<int> &f = front[ci];
          if (cur[ci] + 1 >= (int)f.size()) continue;
          const Point &p0 = grids[ci][f[cur[ci]]], &p1 = grids[ci][f[cur[ci] + 1]];
          const double ds = (double)p1.s - (double)p0.s;
          if (spent + ds > share) continue;
          const double de = p0.e - p1.e;
          const double eff = ds == 0.0 ? std::numeric_limits<double>::infinity() : de / ds;
          if (eff > best_eff) { best = ci; best_eff = eff; }
        }
        if (best < 0) break;
        const std::vector<int> &f = front[best];
        spent += (double)grids[best][f[cur[best] + 1]].s - (double)grids[best][f[cur[best]]].s;
        ++cur[best];
      }
    }
    for (int ci = 0; ci < n_cells; ++ci) idx[ci] = front[ci][cur[ci]];
    return emit(idx, 0.0, infeas);
  }
  if (o->strategy == JOLT_ALLOC_UNIFORM) {
    // points shared by every cell, keyed by (b, r_T, r_d)
    std::vector<std::map<std::tuple<int, int, int>, int>> where(n_cells);
    for (int ci = 0; ci < n_cells; ++ci)
      for (int k = 0; k < (int)grids[ci].size(); ++k)
        where[ci][std::make_tuple(grids[ci][k].b, grids[ci][k].rT, grids[ci][k].rd)] = k;
    struct Cand { double S; int b, rT, rd; double err; };
    std::vector<Cand> cands;
    if (n_cells > 0) {
      for (const auto &kv : where[0]) {
        bool shared = true;
        for (int ci = 1; ci < n_cells && shared; ++ci) shared = where[ci].count(kv.first) > 0;
        if (!shared) continue;
        double S = 0.0, err = 0.0;
        for (int ci = 0; ci < n_cells; ++ci) {
          const Point &p = grids[ci][where[ci].at(kv.first)];
          S += (double)p.s;
          err += p.e;
        }
        cands.push_back(Cand{S, std::get<0>(kv.first), std::get<1>(kv.first), std::get<2>(kv.first), err});
      }
      if (cands.empty()) return jolt_fail(JOLT_E_INVAL, "jolt_allocate: no grid point common to every cell");
    }
    std::sort(cands.begin(), cands.end(), [](const Cand &a, const Cand &b) {
      return std::make_tuple(a.S, a.b, a.rT, a.rd) < std::make_tuple(b.S, b.b, b.rT, b.rd);
    });
    int pick = -1;
    double best = std::numeric_limits<double>::infinity();
    for (int k = 0; k < (int)cands.size(); ++k)
      if (cands[k].S <= B && cands[k].err < best) { pick = k; best = cands[k].err; }
    const int infeas = (pick < 0 && !cands.empty()) ? 1 : 0;
    if (pick < 0) pick = 0;
    for (int ci = 0; ci < n_cells; ++ci)
      idx[ci] = where[ci].at(std::make_tuple(cands[pick].b, cands[pick].rT, cands[pick].rd));
    return emit(idx, 0.0, infeas);
  }
  // the frontier of each grid, led by its first point in every case (a NaN error there
  // would make the full scan keep point 0)
  std::vector<std::vector<int>> front(n_cells);
  for (int ci = 0; ci < n_cells; ++ci) {
    front[ci] = pareto(grids[ci]);
    if (front[ci].empty() || front[ci][0] != 0) front[ci].insert(front[ci].begin(), 0);
  }
  // each frontier's (e, s) pairs contiguous, so a bisection step streams through them
  std::vector<std::vector<double>> fe(n_cells), fs(n_cells);
  for (int ci = 0; ci < n_cells; ++ci) {
    fe[ci].resize(front[ci].size());
    fs[ci].resize(front[ci].size());
    for (size_t q = 0; q < front[ci].size(); ++q) {
      fe[ci][q] = grids[ci][front[ci][q]].e;
      fs[ci][q] = (double)grids[ci][front[ci][q]].s;
    }
  }
  double lam_cur = 0.0;
  std::vector<int> *out_cur = nullptr;
  const std::function<void(int)> pick = [&](int ci) {
    const double *e = fe[ci].data(), *sz = fs[ci].data();
    const size_t nf = fe[ci].size();
    size_t best = 0;
    double bv = e[0] + lam_cur * sz[0];
    for (size_t q = 1; q < nf; ++q) {
      const double v = e[q] + lam_cur * sz[q];
      if (v < bv) { bv = v; best = q; }
    }
    (*out_cur)[ci] = front[ci][best];
  };
  // small frontiers are scanned on the calling thread (waking the pool would cost more)
  size_t front_total = 0;
  for (int ci = 0; ci < n_cells; ++ci) front_total += front[ci].size();
  const bool serial = front_total < 50000;
  auto choose = [&](double lam, std::vector<int> &out) {
    lam_cur = lam;
    out_cur = &out;
    if (serial) {
      for (int ci = 0; ci < n_cells; ++ci) pick(ci);
    } else {
      pool.run(pick);
    }
    double total = 0.0;
    for (int ci = 0; ci < n_cells; ++ci) total += (double)grids[ci][out[ci]].s;
    return total;
  };
  if (choose(0.0, idx) <= B) return emit(idx, 0.0, 0);
  double lo = 0.0, hi = 1e3;
  if (choose(hi, idx_hi) > B) return emit(idx_hi, hi, 1);
  for (int it = 0; it < 200; ++it) {
    if (hi - lo <= 1e-15 * hi) break;
    const double mid = 0.5 * (lo + hi);
    if (choose(mid, idx) <= B) { hi = mid; idx_hi = idx; }
    else lo = mid;
  }
  return emit(idx_hi, hi, 0);
}

// Batched symmetric eigensolver for the mode Gram matrices (token Gram C = X_(2) X_(2)^T,
// feature Grams, FlashJoLT's B B^T).  Section 4 takes the token- and feature-mode
// singular vectors of the cell; they are the eigenvectors of these Grams.
//
//   1. Householder tridiagonalisation A = Q T Q^T (fp32, lower reflectors,
//      Q = H_0 H_1 ... H_{n-2}, H_i = I - tau_i v_i v_i^T, v_i(i+1) = 1).
//   2. All eigenvalues of T by Sturm-count bisection in fp64 (one thread each).
//   3. The top-k eigenvectors of T by inverse iteration in fp64 (one thread each,
//      tridiagonal LU with partial pivoting), re-orthogonalised (modified
//      Gram-Schmidt, two passes) inside clusters of nearly equal eigenvalues.
//   4. U = Q Z applied as blocked WY reflectors (I - V T V^T) with GEMMs.
// fp64 in steps 2-3 costs little on CDNA (full-rate fp64) and makes the
// tridiagonal eigenvectors orthogonal to ~1e-12 even for close eigenvalues.
#include <algorithm>
#include <cfloat>

#include "common.h"
#include "kernels.h"

namespace {

constexpr int SYTD2_THREADS = 1024;

JOLT_DEV double block_sum(double v, double *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < nw; ++w) s += red[w];
  return s;
}

// Workgroup sum with one barrier: successive calls alternate between two halves of red
// (2 x waves entries), so a call never overwrites values an earlier call is still reading.
JOLT_DEV double block_sum1(double v, double *red, int &flip) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  double *r = red + flip * nw;
  flip ^= 1;
  if (lane == 0) r[wave] = v;
  __syncthreads();
  double s = 0.0;
  for (int w = 0; w < nw; ++w) s += r[w];
  return s;
}

// One workgroup per matrix; full symmetric storage in global memory (L2-resident for
// the sizes this kernel serves).  Writes d, e, tau and leaves v_i in column i of A
// (rows i+1..n-1, v_i(i+1) = 1) with zeros above, the dense form the blocked
// back-transformation multiplies by.
//
// Blocked in panels of SB columns (the LAPACK latrd scheme inside one workgroup): the
// panel's reflectors V and the vectors W (A_i v_i corrected for the panel's earlier
// reflectors, then w += K v) are kept in LDS by absolute row.  Column i is brought up to
// date with the panel's earlier reflectors only when it becomes current; the mat-vec reads
// the trailing matrix as it was at the panel start and subtracts V (W^T v) + W (V^T v); the
// trailing matrix past the panel takes the rank-2 SB update once, at the panel end.  Each
// column then reads the trailing matrix once instead of three times (mat-vec, and the
// read and write of an immediate rank-2 update).
constexpr int SB = 16, SBL = SB + 1;     // panel width, LDS row stride of V and W

size_t sytd2_lds_bytes(int n) { return ((size_t)2 * n + (size_t)2 * n * SBL + 2 * SB) * sizeof(float); }

__global__ void __launch_bounds__(SYTD2_THREADS) k_sytd2(EigBatch b) {
  const int mat = blockIdx.x, n = b.n;
  float *A = b.A + (int64_t)mat * b.mat_stride;
  double *dd = b.d + (int64_t)mat * n, *ee = b.e + (int64_t)mat * n;
  float *tau = b.tau + (int64_t)mat * n;
  extern __shared__ float sh[];
  float *v = sh, *w = sh + n;
  float *Vp = w + n, *Wp = Vp + (size_t)n * SBL, *yv = Wp + (size_t)n * SBL;
  __shared__ double red[2 * (SYTD2_THREADS / 64)];
  __shared__ double s_alpha;                        // x[0] of the current column
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = SYTD2_THREADS / 64;
  int flip = 0;
  for (int k0 = 0; k0 < n - 1; k0 += SB) {
    const int jb = min(SB, n - 1 - k0);
    for (int q = tid; q < (n - k0) * SBL; q += SYTD2_THREADS) {
      Vp[(size_t)k0 * SBL + q] = 0.f;
      Wp[(size_t)k0 * SBL + q] = 0.f;
    }
    __syncthreads();
    for (int j = 0; j < jb; ++j) {
      const int i = k0 + j, L = n - 1 - i;
      // column i (rows i..n-1) brought up to date with reflectors k0 .. i-1; the squared
      // norm of x[1..] is accumulated on the way
      double part = 0.0;
      for (int r = i + tid; r < n; r += SYTD2_THREADS) {
        float a = A[(int64_t)r * n + i];
        for (int p = 0; p < j; ++p)
          a -= Vp[(size_t)r * SBL + p] * Wp[(size_t)i * SBL + p] + Wp[(size_t)r * SBL + p] * Vp[(size_t)i * SBL + p];
        if (r == i) A[(int64_t)i * n + i] = a;
        else v[r - i - 1] = a;
        if (r == i + 1) s_alpha = a;
        if (r > i + 1) part += (double)a * (double)a;
      }
      // its barrier also publishes v and x[0]; v[0] is overwritten below, so x[0] is read
      // from its own copy (rewritten only after two more barriers)
      const double sigma = block_sum1(part, red, flip);
      const double alpha = s_alpha;
      double beta, tv, scal;
      if (sigma == 0.0) {
        tv = 0.0; beta = alpha; scal = 0.0;
      } else {
        beta = -copysign(sqrt(alpha * alpha + sigma), alpha);
        tv = (beta - alpha) / beta;
        scal = 1.0 / (alpha - beta);
      }
      // v = x scaled (v[0] = 1); every entry has one owner in this loop
      for (int r = i + 1 + tid; r < n; r += SYTD2_THREADS) {
        const int t = r - i - 1;
        float vt = (t == 0) ? 1.f : (float)((double)v[t] * scal);
        if (tv == 0.0) vt = (t == 0) ? 1.f : 0.f;
        v[t] = vt;
        A[(int64_t)r * n + i] = vt;
        Vp[(size_t)r * SBL + j] = vt;
      }
      if (tid == 0) { ee[i] = beta; tau[i] = (float)tv; }
      __syncthreads();
      if (tv == 0.0) continue;                     // W column stays zero
      const float tf = (float)tv;
      // w' = A22 v over the trailing matrix as of the panel start: a wavefront takes four
      // rows at a time (rows r, r + nw, r + 2 nw, r + 3 nw) so that their loads are in
      // flight together; rows past L read row L - 1 and are not stored
      for (int r0 = wave; r0 < L; r0 += 4 * nw) {
        const float *row[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) row[u] = A + (int64_t)(i + 1 + min(r0 + u * nw, L - 1)) * n + (i + 1);
        float sacc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int c = lane; c < L; c += 64) {
          float x[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) x[u] = row[u][c];
          const float vc = v[c];
#pragma unroll
          for (int u = 0; u < 4; ++u) sacc[u] = fmaf(x[u], vc, sacc[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float su = wave_sum(sacc[u]);
          if (lane == 0 && r0 + u * nw < L) w[r0 + u * nw] = su;
        }
      }
      // yv = [W^T v ; V^T v] over rows i+1.. for the panel's earlier reflectors
      for (int q = wave; q < 2 * j; q += nw) {
        const float *col = (q < j ? Wp : Vp) + (q < j ? q : q - j);
        float sacc = 0.f;
        for (int t = lane; t < L; t += 64) sacc = fmaf(col[(size_t)(i + 1 + t) * SBL], v[t], sacc);
        sacc = wave_sum(sacc);
        if (lane == 0) yv[q < j ? q : SB + q - j] = sacc;
      }
      __syncthreads();
      // corrected w = tau (w' - V yv_W - W yv_V), kept in a register by the thread that owns
      // row t, and its dot with v for K
      part = 0.0;
      float wt[(1024 + SYTD2_THREADS - 1) / SYTD2_THREADS];
#pragma unroll
      for (int u = 0; u < (int)(sizeof(wt) / sizeof(float)); ++u) {
        const int t = tid + u * SYTD2_THREADS;
        wt[u] = 0.f;
        if (t < L) {
          float c = w[t];
          const size_t rr = (size_t)(i + 1 + t) * SBL;
          for (int p = 0; p < j; ++p) c -= Vp[rr + p] * yv[p] + Wp[rr + p] * yv[SB + p];
          wt[u] = tf * c;
          part += (double)wt[u] * (double)v[t];
        }
      }
      const float K = (float)(-0.5 * tv * block_sum1(part, red, flip));
#pragma unroll
      for (int u = 0; u < (int)(sizeof(wt) / sizeof(float)); ++u) {
        const int t = tid + u * SYTD2_THREADS;
        if (t < L) Wp[(size_t)(i + 1 + t) * SBL + j] = fmaf(K, v[t], wt[u]);
      }
      __syncthreads();
    }
    // trailing matrix past the panel: A -= V W^T + W V^T (both triangles)
    const int s0 = k0 + jb;
    for (int r = s0 + wave; r < n; r += nw) {
      float vr[SB], wr[SB];
#pragma unroll
      for (int p = 0; p < SB; ++p) { vr[p] = Vp[(size_t)r * SBL + p]; wr[p] = Wp[(size_t)r * SBL + p]; }
      float *row = A + (int64_t)r * n;
      for (int c = s0 + lane; c < n; c += 64) {
        float acc = 0.f;
#pragma unroll
        for (int p = 0; p < SB; ++p) acc = fmaf(vr[p], Wp[(size_t)c * SBL + p], fmaf(wr[p], Vp[(size_t)c * SBL + p], acc));
        row[c] -= acc;
      }
    }
    __syncthreads();
  }
  // diagonal of T, then zero the strictly upper part and diagonal of the reflector block
  for (int i = tid; i < n; i += SYTD2_THREADS) dd[i] = A[(int64_t)i * n + i];
  if (tid == 0) { ee[n - 1] = 0.0; tau[n - 1] = 0.f; }
  __syncthreads();
  for (int r = wave; r < n; r += nw) {
    float *row = A + (int64_t)r * n;
    for (int c = lane; c < n; c += 64)
      if (c >= r || c == n - 1) row[c] = 0.f;
  }
  if (n == 1 && tid == 0) A[0] = 0.f;
}

JOLT_DEV int sturm_count(const double *d, const double *e, int n, double x, double pivmin) {
  double q = d[0] - x;
  if (fabs(q) <= pivmin) q = -pivmin;
  int cnt = q < 0.0;
  for (int j = 1; j < n; ++j) {
    const double ej = e[j - 1];
    q = d[j] - x - ej * ej / q;
    if (fabs(q) <= pivmin) q = -pivmin;
    cnt += q < 0.0;
  }
  return cnt;
}

JOLT_DEV void gershgorin(const double *d, const double *e, int n, double &gl, double &gu,
                         double &pivmin) {
  gl = DBL_MAX; gu = -DBL_MAX;
  double emax2 = 0.0;
#pragma unroll 8
  for (int i = 0; i < n; ++i) {
    const double r = (i > 0 ? fabs(e[i - 1]) : 0.0) + (i < n - 1 ? fabs(e[i]) : 0.0);
    gl = fmin(gl, d[i] - r);
    gu = fmax(gu, d[i] + r);
    if (i < n - 1) emax2 = fmax(emax2, e[i] * e[i]);
  }
  pivmin = DBL_MIN * fmax(1.0, emax2);
  const double tnorm = fmax(fabs(gl), fabs(gu));
  gl -= 2.0 * DBL_EPSILON * tnorm + 2.0 * pivmin;
  gu += 2.0 * DBL_EPSILON * tnorm + 2.0 * pivmin;
}

// Bisection for all eigenvalues: one workgroup per (matrix, 256 eigenvalues), one
// eigenvalue per thread; d and e^2 are staged in LDS.  Each sweep evaluates the Sturm count
// at three points that split the interval in four (multisection), so a thread advances
// three independent recurrences per step -- work in flight for this latency-bound chain --
// and gains two bits per sweep.  The interval is narrowed to the first quarter whose upper
// point counts more than k eigenvalues, as three successive bisections on the same counts
// would.  The Gershgorin interval and pivmin are reduced over the workgroup (min / max,
// independent of order).  With NP = 1 the sweep is plain bisection at the midpoint: a third
// fewer recurrence steps per bit, for batches large enough to keep the fp64 units busy
// without the extra recurrences.
constexpr int EV_THREADS = 256;
// 1/x from the hardware estimate refined by two Newton steps (each squares the relative
// error, so the result is within a few units in the last place).
JOLT_DEV double recip(double x) {
  double r = __builtin_amdgcn_rcp(x);
  double e = fma(-x, r, 1.0);
  r = fma(r, e, r);
  e = fma(-x, r, 1.0);
  return fma(r, e, r);
}
// 1/x to within 2^-48 relative: the gfx950 estimate is within 2^-24.4 (measured over 2^20
// inputs of exponents -200..200), one Newton step squares that.  A Sturm step
// q' = d - x - e^2 / q with such a quotient is the exact step for e^2 scaled by 1 + 2^-48,
// so each count is that of a tridiagonal within about 2^-48 ||T|| of the given one, far
// below the 1e-11 ||T|| to which the eigenvalues are resolved (|x| >= pivmin > 0 here).
JOLT_DEV double recip_sturm(double x) {
  const double r = __builtin_amdgcn_rcp(x);
  return fma(r, fma(-x, r, 1.0), r);
}

template <int NP>
__global__ void __launch_bounds__(EV_THREADS) k_tri_eigvals(EigBatch b) {
  static_assert(NP == 1 || NP == 3, "bisection or quarter-point multisection");
  extern __shared__ double lds[];
  __shared__ double red[3][EV_THREADS / 64];
  const int mat = blockIdx.y, n = b.n, tid = threadIdx.x;
  double *dl = lds, *e2 = lds + n;
  const double *d = b.d + (int64_t)mat * n, *e = b.e + (int64_t)mat * n;
  // Gershgorin bounds and pivmin (as the serial gershgorin(): min / max over rows)
  double g_lo = DBL_MAX, g_hi = -DBL_MAX, emax2 = 0.0;
  for (int i = tid; i < n; i += EV_THREADS) {
    const double di = d[i], ei = i < n - 1 ? e[i] : 0.0, ep = i > 0 ? e[i - 1] : 0.0;
    dl[i] = di;
    e2[i] = ei * ei;
    const double r = fabs(ep) + fabs(ei);
    g_lo = fmin(g_lo, di - r);
    g_hi = fmax(g_hi, di + r);
    emax2 = fmax(emax2, ei * ei);
  }
  for (int o = 32; o >= 1; o >>= 1) {
    g_lo = fmin(g_lo, __shfl_xor(g_lo, o, 64));
    g_hi = fmax(g_hi, __shfl_xor(g_hi, o, 64));
    emax2 = fmax(emax2, __shfl_xor(emax2, o, 64));
  }
  if ((tid & 63) == 0) { red[0][tid >> 6] = g_lo; red[1][tid >> 6] = g_hi; red[2][tid >> 6] = emax2; }
  __syncthreads();
  double gl = red[0][0], gu = red[1][0];
  emax2 = red[2][0];
  for (int w = 1; w < EV_THREADS / 64; ++w) {
    gl = fmin(gl, red[0][w]); gu = fmax(gu, red[1][w]); emax2 = fmax(emax2, red[2][w]);
  }
  const double pivmin = DBL_MIN * fmax(1.0, emax2);
  {
    const double tnorm = fmax(fabs(gl), fabs(gu));
    gl -= 2.0 * DBL_EPSILON * tnorm + 2.0 * pivmin;
    gu += 2.0 * DBL_EPSILON * tnorm + 2.0 * pivmin;
  }
  // the tridiagonal comes from an fp32 reduction, so resolving eigenvalues beyond a
  // 1e-11 fraction of ||T|| adds nothing; this bounds the sweeps at about 20
  const double atol = 1e-11 * fmax(fabs(gl), fabs(gu));
  const int k = blockIdx.x * EV_THREADS + tid;
  double lo = gl, hi = gu;
  bool live = k < n;
  for (int it = 0; it < 200; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (live && (hi - lo <= 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + 4.0 * pivmin + atol ||
                 mid == lo || mid == hi))
      live = false;
    if (!__any(live)) break;
    // Sturm counts (eigenvalues below x) at the quarter points x[0] < x[1] < x[2], or at the
    // midpoint alone
    const double h4 = 0.25 * (hi - lo);
    double x[NP];
    if (NP == 1) x[0] = mid;
    else { x[0] = lo + h4; x[1] = mid; x[2] = hi - h4; }
    double qv[NP];
    int cnt[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      qv[q] = dl[0] - x[q];
      if (fabs(qv[q]) <= pivmin) qv[q] = -pivmin;
      cnt[q] = qv[q] < 0.0;
    }
#pragma unroll 4
    for (int jj = 1; jj < n; ++jj) {
      const double dj = dl[jj], ej2 = e2[jj - 1];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        double t = dj - x[q] - ej2 * recip_sturm(qv[q]);
        if (fabs(t) <= pivmin) t = -pivmin;
        qv[q] = t;
        cnt[q] += t < 0.0;
      }
    }
    if (live) {
      if (NP == 1) {
        if (cnt[0] > k) hi = x[0];
        else lo = x[0];
      } else {
        if (cnt[0] > k) hi = x[0];
        else if (cnt[NP > 1 ? 1 : 0] > k) { lo = x[0]; hi = x[NP > 1 ? 1 : 0]; }
        else if (cnt[NP - 1] > k) { lo = x[NP > 1 ? 1 : 0]; hi = x[NP - 1]; }
        else lo = x[NP - 1];
      }
    }
  }
  if (k < n) b.lam[(int64_t)mat * n + (n - 1 - k)] = 0.5 * (lo + hi);
}

// inverse iteration on (T - lam I) with partial pivoting; per-thread vectors are laid
// out [array][i][column] so neighbouring threads touch neighbouring addresses.  Each pivot is
// inverted once by recip() (a few ulps) and its reciprocal multiplies in both sweeps: a
// division on the serial chain of every step costs about twice as long, and inverse
// iteration does not need correctly rounded steps.
__global__ void __launch_bounds__(64) k_tri_eigvecs(EigBatch b, InvitWork w, int j0) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = b.n;
  if (idx >= (int64_t)b.n_mat * w.ldlu) return;
  const int mat = (int)(idx / w.ldlu), jj = (int)(idx % w.ldlu), j = j0 + jj;
  if (j >= w.k[mat]) return;
  const double *d = b.d + (int64_t)mat * n, *e = b.e + (int64_t)mat * n;
  const double lam = b.lam[(int64_t)mat * n + j];
  const int64_t ld = w.ldz;
  double *x = w.Z + (int64_t)mat * n * ld + j;
  const int64_t ll = w.ldlu;
  double *u0 = w.lu + ((int64_t)mat * 3 + 0) * n * ll + jj;
  double *u1 = w.lu + ((int64_t)mat * 3 + 1) * n * ll + jj;
  double *u2 = w.lu + ((int64_t)mat * 3 + 2) * n * ll + jj;
  double gl, gu, pivmin;
  gershgorin(d, e, n, gl, gu, pivmin);
  const double tnorm = fmax(fmax(fabs(gl), fabs(gu)), DBL_MIN);
  const double tiny = DBL_EPSILON * tnorm;
  bool zero = true;
  for (int i = 0; i < n && zero; ++i) zero = d[i] == 0.0 && (i == n - 1 || e[i] == 0.0);
  if (zero) {
    // the zero matrix (an all-zero cell): every unit vector is an eigenvector; e_j keeps the
    // k vectors orthonormal without a solve that would divide by the zero pivots
    for (int i = 0; i < n; ++i) x[(int64_t)i * ld] = i == j ? 1.0 : 0.0;
    return;
  }
  // deterministic start vector in [-1, 1]
  auto start = [&](int i) {
    u32x4 r = philox4x32_10(u32x4{(uint32_t)i, (uint32_t)j, (uint32_t)mat, 4u}, 0x6a6f6c74u, 0u);
    return ((double)r.x + 0.5) * 0x1p-31 - 1.0;
  };
  if (w.iters == 0)
    for (int i = 0; i < n; ++i) x[(int64_t)i * ld] = start(i);
  // Each sweep below walks the column serially; its steps are taken in blocks of IB whose
  // loads are issued one block ahead (they never touch an element the current block
  // stores), so the memory latency is paid once per block instead of once per step.  The
  // arithmetic of every step is unchanged.  The first forward sweep draws the start vector
  // itself, and the scaling of a solve's result by 1 / max|x| is applied where the next pass
  // reads it (x holds the vector divided by `pend`), which saves two passes over the column
  // per solve with the same values.
  constexpr int IB = 8;
  double growth = 0.0;                 // max |x| after the last solve (its input has max |x| <= 1)
  double pend = 1.0;
  for (int it = 0; it < w.iters; ++it) {
    const bool gen = it == 0;
    // forward: factor T - lam I = P L U while transforming the right-hand side in x
    double p = d[0] - lam, q = (n > 1) ? e[0] : 0.0;
    double y = gen ? start(0) : x[0] * pend;
    double nc[IB], na1[IB], nb1[IB], ny1[IB];
    auto load_fwd = [&](int i0) {
#pragma unroll
      for (int s = 0; s < IB; ++s) {
        const int i = i0 + s;
        const bool in = i < n - 1;
        nc[s] = in ? e[i] : 0.0;
        na1[s] = in ? d[i + 1] - lam : 0.0;
        nb1[s] = (in && i + 1 < n - 1) ? e[i + 1] : 0.0;
        ny1[s] = in ? (gen ? start(i + 1) : x[(int64_t)(i + 1) * ld] * pend) : 0.0;
      }
    };
    load_fwd(0);
    for (int i0 = 0; i0 < n - 1; i0 += IB) {
      double cc[IB], ca1[IB], cb1[IB], cy1[IB];
#pragma unroll
      for (int s = 0; s < IB; ++s) { cc[s] = nc[s]; ca1[s] = na1[s]; cb1[s] = nb1[s]; cy1[s] = ny1[s]; }
      if (i0 + IB < n - 1) load_fwd(i0 + IB);
#pragma unroll
      for (int s = 0; s < IB; ++s) {
        const int i = i0 + s;
        if (i >= n - 1) break;
        const double c = cc[s];                      // sub-diagonal entry of row i+1
        const double a1 = ca1[s], b1 = cb1[s], y1 = cy1[s];
        if (fabs(p) >= fabs(c)) {
          if (fabs(p) < tiny) p = copysign(tiny, p == 0.0 ? 1.0 : p);
          const double rp = recip(p);
          const double l = c * rp;
          u0[(int64_t)(i) * ll] = rp; u1[(int64_t)(i) * ll] = q; u2[(int64_t)(i) * ll] = 0.0;
          x[(int64_t)i * ld] = y;
          y = y1 - l * y;
          p = a1 - l * q;
          q = b1;
        } else {
          const double rc = recip(c);
          const double l = p * rc;
          u0[(int64_t)(i) * ll] = rc; u1[(int64_t)(i) * ll] = a1; u2[(int64_t)(i) * ll] = b1;
          x[(int64_t)i * ld] = y1;
          const double ynew = y - l * y1;
          const double pnew = q - l * a1;
          q = -l * b1;
          p = pnew;
          y = ynew;
        }
      }
    }
    if (fabs(p) < tiny) p = copysign(tiny, p == 0.0 ? 1.0 : p);
    x[(int64_t)(n - 1) * ld] = y;
    // back substitution, blocks of rows n-2, n-3, ... loaded one block ahead; u0 holds the
    // reciprocals of the pivots, so that no step divides
    double xn1 = y * recip(p), xn2 = 0.0;
    x[(int64_t)(n - 1) * ld] = xn1;
    double amax = fabs(xn1);
    double bx[IB], b0[IB], b1v[IB], b2[IB];
    auto load_back = [&](int i0) {                 // rows i0, i0 - 1, ..., i0 - IB + 1
#pragma unroll
      for (int s = 0; s < IB; ++s) {
        const int i = i0 - s;
        const bool in = i >= 0;
        bx[s] = in ? x[(int64_t)i * ld] : 0.0;
        b0[s] = in ? u0[(int64_t)i * ll] : 1.0;
        b1v[s] = in ? u1[(int64_t)i * ll] : 0.0;
        b2[s] = in ? u2[(int64_t)i * ll] : 0.0;
      }
    };
    load_back(n - 2);
    for (int i0 = n - 2; i0 >= 0; i0 -= IB) {
      double cx[IB], c0[IB], c1[IB], c2[IB];
#pragma unroll
      for (int s = 0; s < IB; ++s) { cx[s] = bx[s]; c0[s] = b0[s]; c1[s] = b1v[s]; c2[s] = b2[s]; }
      if (i0 - IB >= 0) load_back(i0 - IB);
#pragma unroll
      for (int s = 0; s < IB; ++s) {
        const int i = i0 - s;
        if (i < 0) break;
        const double xi = (cx[s] - c1[s] * xn1 - c2[s] * xn2) * c0[s];
        x[(int64_t)i * ld] = xi;
        xn2 = xn1; xn1 = xi;
        amax = fmax(amax, fabs(xi));
      }
    }
    growth = amax;
    pend = amax > 0.0 ? 1.0 / amax : 1.0;
  }
  // convergence: the normalised vector z = y / |y| has residual |(T - lam I) z|_2 <=
  // sqrt(n) / |y|_inf, so a growth of at least 1e4 sqrt(n) / |T| bounds it by 1e-4 |T|
  if (!(growth * tnorm >= 1e4 * sqrt((double)n))) w.status[mat] = 1;
  double nrm = 0.0;
  for (int i0 = 0; i0 < n; i0 += IB) {
    double v[IB];
#pragma unroll
    for (int s = 0; s < IB; ++s) v[s] = i0 + s < n ? x[(int64_t)(i0 + s) * ld] * pend : 0.0;
#pragma unroll
    for (int s = 0; s < IB; ++s) nrm += v[s] * v[s];
  }
  nrm = nrm > 0.0 ? 1.0 / sqrt(nrm) : 0.0;
  for (int i0 = 0; i0 < n; i0 += IB) {
    double v[IB];
#pragma unroll
    for (int s = 0; s < IB; ++s) v[s] = i0 + s < n ? x[(int64_t)(i0 + s) * ld] * pend : 0.0;
#pragma unroll
    for (int s = 0; s < IB; ++s) if (i0 + s < n) x[(int64_t)(i0 + s) * ld] = v[s] * nrm;
  }
}

// Modified Gram-Schmidt (two passes) over each cluster of eigenvalues whose
// consecutive gaps are below tol * ||T||; one workgroup per cluster start.
__global__ void __launch_bounds__(256) k_cluster_mgs(EigBatch b, InvitWork w, int kmax, double rtol) {
  const int mat = blockIdx.y, j0 = blockIdx.x, n = b.n;
  const int k = w.k[mat];
  if (j0 >= k) return;
  const double *lam = b.lam + (int64_t)mat * n;
  const double scale = fmax(fabs(lam[0]), fabs(lam[n - 1]));
  const double tol = rtol * scale;
  auto close = [&](int a) { return lam[a] - lam[a + 1] <= tol; };   // a, a+1 in cluster
  if (j0 > 0 && close(j0 - 1)) return;            // not a cluster start
  int j1 = j0;
  while (j1 + 1 < k && close(j1)) ++j1;
  if (j1 == j0) return;
  __shared__ double red[4];
  const int64_t ld = w.ldz;
  double *Z = w.Z + (int64_t)mat * n * ld;
  for (int c = j0; c <= j1; ++c) {
    for (int pass = 0; pass < 2; ++pass) {
      for (int p = j0; p < c; ++p) {
        double part = 0.0;
        for (int i = threadIdx.x; i < n; i += 256) part += Z[(int64_t)i * ld + p] * Z[(int64_t)i * ld + c];
        const double dot = block_sum(part, red);
        for (int i = threadIdx.x; i < n; i += 256) Z[(int64_t)i * ld + c] -= dot * Z[(int64_t)i * ld + p];
        __syncthreads();
      }
    }
    double part = 0.0;
    for (int i = threadIdx.x; i < n; i += 256) part += Z[(int64_t)i * ld + c] * Z[(int64_t)i * ld + c];
    const double nr = block_sum(part, red);
    const double s = nr > 0.0 ? 1.0 / sqrt(nr) : 0.0;
    for (int i = threadIdx.x; i < n; i += 256) Z[(int64_t)i * ld + c] *= s;
    __syncthreads();
  }
}

__global__ void k_z_to_f32(EigBatch b, InvitWork w, int kmax, float *U, int64_t ldu, int64_t u_stride) {
  const int mat = blockIdx.y;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = b.n;
  if (idx >= (int64_t)n * kmax) return;
  const int i = (int)(idx / kmax), j = (int)(idx % kmax);
  const int k = w.k[mat];
  float v = 0.f;
  if (j < k) v = (float)w.Z[(int64_t)mat * n * w.ldz + (int64_t)i * w.ldz + j];
  if (j < ldu) U[(int64_t)mat * u_stride + (int64_t)i * ldu + j] = v;
}

// T factor of the block reflector of panel p (columns i0 .. i0+pw-1 of A):
// H_i0 ... H_{i0+pw-1} = I - V T V^T with T upper triangular, built by the forward
// recurrence T[0:j, j] = -tau_j T[0:j, 0:j] (V^T V)[0:j, j] from the precomputed Gram S.
constexpr int NB = 128;
__global__ void __launch_bounds__(NB) k_larft(EigBatch b, const float *S_all, float *Tout) {
  const int mat = blockIdx.y, p = blockIdx.x, n = b.n;
  const int panels = (n + NB - 1) / NB;
  const int i0 = p * NB;
  const int pw = max(0, min(NB, n - refl_off(b) - i0));
  const float *tau = b.tau + (int64_t)mat * n;
  const float *S = S_all + ((int64_t)mat * panels + p) * NB * NB;
  __shared__ float T[NB][NB + 1];
  __shared__ float Ss[NB][NB + 1];              // the panel's Gram, staged once
  const int a = threadIdx.x;
  for (int c = 0; c < NB; ++c) T[a][c] = 0.f;
  for (int r0 = 0; r0 < NB; r0 += 16) {         // sixteen loads in flight per thread
    float x[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) x[k] = S[(r0 + k) * NB + a];
#pragma unroll
    for (int k = 0; k < 16; ++k) Ss[r0 + k][a] = x[k];
  }
  __syncthreads();
  for (int j = 0; j < pw; ++j) {
    const float tj = tau[i0 + j];
    float s = 0.f;
    if (a < j)
      for (int c = a; c < j; ++c) s = fmaf(T[a][c], Ss[c][j], s);
    __syncthreads();
    if (a < j) T[a][j] = -tj * s;
    if (a == j) T[j][j] = tj;
    __syncthreads();
  }
  float *To = Tout + ((int64_t)mat * panels + p) * NB * NB;
  for (int c = 0; c < NB; ++c) To[a * NB + c] = T[a][c];
}

}  // namespace

hipError_t launch_sytrd_small(const EigBatch &b, hipStream_t st) {
  if (b.n > SYTD2_THREADS) return hipErrorInvalidValue;   // one corrected w entry per thread
  const size_t shm = sytd2_lds_bytes(b.n);
  if (shm > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_sytd2),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_sytd2, dim3(b.n_mat), dim3(SYTD2_THREADS), shm, st, b);
  return hipGetLastError();
}

hipError_t launch_tridiag_eigvals(const EigBatch &b, hipStream_t st) {
  const int per_block = EV_THREADS;
  dim3 grid((b.n + per_block - 1) / per_block, b.n_mat);
  const size_t shm = (size_t)2 * b.n * sizeof(double);
  // bisection once the batch fills every SIMD with two wavefronts (32 matrices of order
  // 4096), multisection below that
  const bool bisect = (int64_t)b.n_mat * b.n >= (int64_t)32 * 4096;
  const void *fn = bisect ? reinterpret_cast<const void *>(&k_tri_eigvals<1>)
                          : reinterpret_cast<const void *>(&k_tri_eigvals<3>);
  if (shm > 65536) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
  }
  if (bisect) hipLaunchKernelGGL(k_tri_eigvals<1>, grid, dim3(EV_THREADS), shm, st, b);
  else hipLaunchKernelGGL(k_tri_eigvals<3>, grid, dim3(EV_THREADS), shm, st, b);
  return hipGetLastError();
}

hipError_t launch_tridiag_eigvecs(const EigBatch &b, const InvitWork &w, int kmax, hipStream_t st) {
  if (kmax <= 0) return hipSuccess;
  const int64_t total = (int64_t)b.n_mat * w.ldlu;
  hipError_t err = hipSuccess;
  for (int j0 = 0; j0 < kmax; j0 += w.ldlu) {
    hipLaunchKernelGGL(k_tri_eigvecs, dim3((unsigned)((total + 63) / 64)), dim3(64), 0, st, b, w, j0);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(k_cluster_mgs, dim3(kmax, b.n_mat), dim3(256), 0, st, b, w, kmax, 1e-10);
  return hipGetLastError();
}

int backtransform_nb() { return NB; }

constexpr int BT_KCHUNK = 512;   // rows per split-K chunk of W1 = V^T U

size_t backtransform_scratch_floats(int n_mat, int n, int kmax) {
  const size_t panels = (n + NB - 1) / NB;
  const size_t chunks = (n + BT_KCHUNK - 1) / BT_KCHUNK;
  return 2 * (size_t)n_mat * panels * NB * NB        // S = V^T V and T per panel
         + (size_t)n_mat * chunks * NB * kmax         // W1 partials
         + (size_t)n_mat * NB * kmax;                 // W2
}

size_t backtransform_table_entries(int n_mat, int n) {
  const size_t panels = (n + NB - 1) / NB;
  const size_t chunks = (n + BT_KCHUNK - 1) / BT_KCHUNK;
  return panels * (size_t)n_mat * (1 + chunks + 2);
}

hipError_t launch_backtransform(const EigBatch &b, const InvitWork &w, int kmax, const int *k_host, float *U,
                                int64_t ldu, int64_t u_stride, float *scratch, GemmProblem *tab_dev,
                                GemmProblem *tab_host, hipStream_t st, bool u_ready) {
  const int n = b.n, panels = (n + NB - 1) / NB, nm = b.n_mat, off = refl_off(b);
  const int chunks_max = (n + BT_KCHUNK - 1) / BT_KCHUNK;
  {
    dim3 g((unsigned)(((int64_t)n * kmax + 255) / 256), nm);
    if (!u_ready) hipLaunchKernelGGL(k_z_to_f32, g, dim3(256), 0, st, b, w, kmax, U, ldu, u_stride);
  }
  float *Sf = scratch;
  float *Tf = Sf + (size_t)nm * panels * NB * NB;
  float *W1 = Tf + (size_t)nm * panels * NB * NB;            // [m][chunk * NB][kmax]
  float *W2 = W1 + (size_t)nm * chunks_max * NB * kmax;       // [m][NB][kmax]
  const int64_t w1_mat = (int64_t)chunks_max * NB * kmax;
  // table: [S: panels x nm] then per panel [W1: nm x chunks | W2: nm | U: nm]
  const size_t per_panel = (size_t)nm * (chunks_max + 2);
  GemmProblem *gS = tab_host;
  for (int p = 0; p < panels; ++p) {
    const int i0 = p * NB, pw = std::max(0, std::min(NB, n - off - i0)), rows = std::max(0, n - (i0 + off));
    const int chunks = std::max(1, (rows + BT_KCHUNK - 1) / BT_KCHUNK);
    GemmProblem *g = tab_host + (size_t)panels * nm + (size_t)p * per_panel;
    for (int m = 0; m < nm; ++m) {
      const float *A = b.A + (int64_t)m * b.mat_stride;
      const int km = std::min(std::max(k_host[m], 0), kmax);   // this matrix's vectors
      GemmProblem S{};
      S.A = GemmOperand{A + (int64_t)(i0 + off) * n + i0, n, 0, 0, 0, 1};
      S.B = GemmOperand{A + (int64_t)(i0 + off) * n + i0, n, 0, 0, 0, 1};
      S.C = Sf + ((size_t)m * panels + p) * NB * NB; S.ldc = NB;
      S.M = std::max(pw, 0); S.N = std::max(pw, 0); S.K = rows; S.alpha = 1.f; S.beta = 0.f;
      gS[(size_t)p * nm + m] = S;
      // W1 partial c = V[rows of chunk c]^T U[rows of chunk c]   (pw x kmax each)
      for (int c = 0; c < chunks_max; ++c) {
        GemmProblem P{};
        const int r0 = c * BT_KCHUNK, r1 = std::min(rows, r0 + BT_KCHUNK);
        P.A = GemmOperand{A + (int64_t)(i0 + off + r0) * n + i0, n, 0, 0, 0, 1};
        P.B = GemmOperand{U + (int64_t)m * u_stride + (int64_t)(i0 + off + r0) * ldu, ldu, 0, 0, 0, 1};
        P.C = W1 + m * w1_mat + (int64_t)c * NB * kmax; P.ldc = kmax;
        P.M = (c < chunks) ? pw : 0; P.N = km; P.K = std::max(0, r1 - r0);
        P.alpha = 1.f; P.beta = 0.f;
        g[(size_t)m * chunks_max + c] = P;
      }
      // W2 = [T T ... T] [W1_0; W1_1; ...]: the split-K sum folded into this product
      // (A's columns wrap onto T with a zero segment stride)
      GemmProblem Q{};
      Q.A = seg_operand(Tf + ((size_t)m * panels + p) * NB * NB, NB, 0, 0, NB, 1);
      Q.B = GemmOperand{W1 + m * w1_mat, kmax, 0, 0, 0, 1};
      Q.C = W2 + (size_t)m * NB * kmax; Q.ldc = kmax;
      Q.M = pw; Q.N = km; Q.K = chunks * NB; Q.alpha = 1.f; Q.beta = 0.f;
      g[(size_t)nm * chunks_max + m] = Q;
      GemmProblem R{};
      R.A = GemmOperand{A + (int64_t)(i0 + off) * n + i0, n, 0, 0, 0, 1};
      R.B = GemmOperand{W2 + (size_t)m * NB * kmax, kmax, 0, 0, 0, 1};
      R.C = U + (int64_t)m * u_stride + (int64_t)(i0 + off) * ldu; R.ldc = ldu;
      R.M = rows; R.N = km; R.K = pw; R.alpha = -1.f; R.beta = 1.f;
      g[(size_t)nm * (chunks_max + 1) + m] = R;
    }
  }
  const size_t ntab = (size_t)panels * nm + (size_t)panels * per_panel;
  hipError_t err = hipMemcpyAsync(tab_dev, tab_host, sizeof(GemmProblem) * ntab, hipMemcpyHostToDevice, st);
  if (err != hipSuccess) return err;
  // W1 rows past a short panel's width must read as zero in the folded sum: the last
  // (shortest) panel is applied first, right after this clear
  err = hipMemsetAsync(W1, 0, sizeof(float) * (size_t)nm * w1_mat, st);
  if (err != hipSuccess) return err;
  err = launch_gemm(tab_dev, nm * panels, NB, NB, 1, GT_F32, GT_F32, false, false, st);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(k_larft, dim3(panels, nm), dim3(NB), 0, st, b, Sf, Tf);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  for (int p = panels - 1; p >= 0; --p) {
    const int i0 = p * NB, pw = std::max(0, std::min(NB, n - off - i0));
    if (pw <= 0) continue;
    const int rows = n - (i0 + off);
    GemmProblem *g = tab_dev + (size_t)panels * nm + (size_t)p * per_panel;
    err = launch_gemm(g, nm * chunks_max, pw, kmax, 1, GT_F32, GT_F32, false, false, st);
    if (err != hipSuccess) return err;
    err = launch_gemm(g + (size_t)nm * chunks_max, nm, pw, kmax, 1, GT_F32, GT_F32, true, false, st);
    if (err != hipSuccess) return err;
    err = launch_gemm(g + (size_t)nm * (chunks_max + 1), nm, rows, kmax, 1, GT_F32, GT_F32, true, false, st);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

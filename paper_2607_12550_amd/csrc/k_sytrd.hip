// Blocked Householder tridiagonalisation for large symmetric matrices (the exact
// token Gram C = X_(2) X_(2)^T of section 4 at T in the thousands), batched over
// matrices of one size.
//
// Panel of nb columns (the latrd scheme): for column i = k0 + j, o = i + 1,
//   x  = A[:, i] - V[:, :j] W[i, :j]^T - W[:, :j] V[i, :j]^T     (column as updated so far)
//   Householder of x[o:]: alpha = x_o, sigma = ||x[o+1:]||^2, beta, tau, scal = 1/(alpha - beta)
//   v  = e_o + scal * x_tail           (x_tail = x with entries <= o zeroed)
//   y  = A22 v - V (W^T v) - W (V^T v),   A22 = A[o:, o:] as at the panel start
//   w  = tau y - (tau^2 / 2)(y^T v) v,    W[:, j] = w
// then A22 -= V W^T + W V^T as one MFMA GEMM with K = 2 nb (full storage is kept).
//
// By linearity A22 v = scal * A22 x_tail + A22[:, o], so the memory-bound mat-vec
// runs on the unnormalised x_tail; sigma and the correction dot products W^T x_tail,
// V^T x_tail are formed where x_tail is produced.  Per column:
//   k_symv_tiles  lower-triangle 128 x 128 tiles of A22 (each read once; an off-diagonal
//                 tile feeds two row blocks through per-slot partials, so row sums are
//                 formed in a fixed order);
//   k_col_step    per 128-row block: tau, v, y, w (y^T v assembled from global sums the
//                 launch already has), then the next column's x and the block partials of
//                 its sigma and dot products;
//   k_col_first   the first column of a panel (x is column k0 of A).
// Panels are stored twice, P = [V; W] and Q = [W; V] (rows = panel columns, packed to
// the panel's width jb), so the rank-2jb update is the single product P^T Q.  Every row
// a kernel or the update reads (rows >= the current column's o) has been written in
// the current panel, so the panel buffers never need clearing.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace {

constexpr int TB = 128;   // mat-vec tile
constexpr int RB = 128;   // rows per workgroup of the column kernels
constexpr int TRD_MAX_N = 8192;
static_assert(TRD_MAX_N / TB <= 64, "the slots of one row fit the lanes of a wavefront");

JOLT_DEV void tri_decode(int t, int &I, int &J) {
  int i = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while ((i + 1) * (i + 2) / 2 <= t) ++i;
  while (i * (i + 1) / 2 > t) --i;
  I = i;
  J = t - i * (i + 1) / 2;
}

struct MatView {
  float *A, *P, *Q, *xt, *part, *dpart, *qpart, *sc;
  double *d, *e;
  float *tau;
};

JOLT_DEV MatView view(const SytrdArgs &a, int mat) {
  const int n = a.n, nb = a.nb;
  MatView m;
  m.A = a.A + (int64_t)mat * a.mat_stride;
  float *base = a.work + (int64_t)mat * a.work_stride;
  m.P = base;
  m.Q = m.P + (int64_t)2 * nb * n;
  m.xt = m.Q + (int64_t)2 * nb * n;
  m.part = m.xt + n;
  m.dpart = m.part + (int64_t)a.slots * n;                  // two buffers (column parity)
  m.qpart = m.dpart + (int64_t)2 * a.slots * (2 * nb + 1);
  m.sc = m.qpart + (int64_t)a.slots * (a.slots + 1) / 2;   // per parity: [0] alpha, [1] diagonal
  m.d = a.d + (int64_t)mat * n;
  m.e = a.e + (int64_t)mat * n;
  m.tau = a.tau + (int64_t)mat * n;
  return m;
}

// A22 x_tail partials for tile (I, J) of the trailing block.  Tiles are 128 x 128 on a grid
// whose origin `base` is o rounded down to a multiple of 32 (so the 128-float row segment a
// tile reads covers exactly four 128-byte cache lines);
// entries with row or column < o are masked to zero.  Thread (ty, tx) of the 16 x 16 grid
// holds 8 rows x 8 columns in registers, the columns being the two runs 4 tx .. 4 tx + 3 and
// 64 + 4 tx .. 64 + 4 tx + 3 of the tile, so that each 16-byte load of a wave covers two
// whole cache lines of a row; row sums reduce across tx (lane shuffles), column sums across
// ty (shuffles, then LDS across the four waves).  Each tile also writes its term of
// x_tail^T A22 x_tail (x_I^T A_II x_I on the diagonal, 2 x_I^T A_IJ x_J off it), which is
// sum_r x_r (row sum)_r + sum_c x_c (column sum)_c over the tile in both cases.
// base[byte offset]: with base uniform and the offset a 32-bit vector, the load takes the
// scalar-base + vector-offset form
JOLT_DEV float ld_off(const float *base, uint32_t boff) {
  return *reinterpret_cast<const float *>(reinterpret_cast<const char *>(base) + boff);
}

JOLT_DEV void householder(float alpha, double sigma, double &beta, double &tv, double &scal) {
  if (sigma == 0.0) { tv = 0.0; beta = alpha; scal = 0.0; return; }
  beta = -copysign(sqrt((double)alpha * alpha + sigma), (double)alpha);
  tv = (beta - alpha) / beta;
  scal = 1.0 / (alpha - beta);
}

// Column i = k0 + j of a panel, after the mat-vec of its x_tail: reflector i from the block
// partials, w_i, and, when the panel continues (more != 0), column i + 1 as updated by
// reflectors k0 .. i together with the block partials of its sigma and dot products.
// w_i = tau y - (tau^2 / 2)(y^T v) v needs the global y^T v; it is assembled from sums this
// launch already has, so that no second launch per column is needed:
//   y^T v     = v^T A22 v - 2 (V^T v).(W^T v),
//   v^T A22 v = A22[o, o] + 2 scal (A22 x_tail)[o] + scal^2 x_tail^T A22 x_tail,
// with (A22 x_tail)[o] summed from the slot partials of row o and the last term from the
// mat-vec's per-tile partials.  Each workgroup also forms y[o] (hence w_i[o], which the
// next column's update needs) by wave sums, and the owner of row o stores that same value.
// The column scalars (alpha, diagonal) and the dot partials alternate between two
// buffers by column parity: this launch reads column i's and writes column i + 1's.
__global__ void __launch_bounds__(RB, 2) k_col_step(SytrdArgs a, int i, int j, int jbw, int more) {
  const int mat = blockIdx.y, n = a.n, nb = a.nb, o = i + 1;
  const int base = o & ~31, nt = (n - base + TB - 1) / TB, ntile = nt * (nt + 1) / 2;
  const int nprev = (n - i + RB - 1) / RB;     // row blocks of the launch that made column i's x
  const MatView M = view(a, mat);
  const int64_t dstride = 2 * nb + 1, dbuf = (int64_t)a.slots * dstride;
  const float *dcur = M.dpart + (i & 1) * dbuf;
  float *dnext = M.dpart + ((i + 1) & 1) * dbuf;
  const float *scur = M.sc + 2 * (i & 1);
  float *snext = M.sc + 2 * ((i + 1) & 1);
  __shared__ float pw[32], pv[32], cw[32], cv[32];
  __shared__ double red[RB / 64];
  __shared__ double sh_sigma;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float *V = M.P, *W = M.P + (int64_t)jbw * n;
  float *Qv = M.Q + (int64_t)jbw * n;
  const int r = o + blockIdx.x * RB + tid;
  const int rr = r < n ? r : o;                 // in-range row for the loads
  // Every load that does not depend on this column's Householder scalars is issued before
  // any is used and without a branch: entries past the live range read an entry this launch
  // does not write and are masked afterwards.  The kernel then waits on one memory round
  // trip before its first barrier.  Each load is a uniform row base plus a per-thread byte
  // offset shared by its group, so the addresses cost no 64-bit vector arithmetic.
  const uint32_t off_r = 4u * (uint32_t)rr, off_p = 4u * (uint32_t)(rr - base);
  const float *pp = M.part + (rr - base);
  float ts[32];
#pragma unroll
  for (int q = 0; q < 32; ++q) ts[q] = ld_off(M.part + (int64_t)min(q, nt - 1) * n, off_p);
  const float a_o = ld_off(M.A + (int64_t)o * n, off_r);   // A22[:, 0] (row o by symmetry)
  const float a_oo = M.A[(int64_t)o * n + o];
  const float x_r = ld_off(M.xt, off_r);
  // row f of V and W is not written by this launch (it writes row j only)
  const int f = j == 0 ? 1 : 0;
  float vrow[32], wrow[32];
#pragma unroll
  for (int p = 0; p < 32; ++p) {
    vrow[p] = ld_off(V + (int64_t)(p < j ? p : f) * n, off_r);
    wrow[p] = ld_off(W + (int64_t)(p < j ? p : f) * n, off_r);
  }
  const uint32_t off_c = 4u * (uint32_t)(tid < j ? tid : f) * (uint32_t)n;
  float w_o = ld_off(W + o, off_c);
  float v_o = ld_off(V + o, off_c);
  const float alpha = scur[0];
  const uint32_t off_d = 4u * (uint32_t)min(tid, 2 * j);   // dot of this thread: 0 sigma, then W, V
  const float *dp = dcur + min(tid, 2 * j);
  float td[32];
#pragma unroll
  for (int b = 0; b < 32; ++b) td[b] = ld_off(dcur + (int64_t)min(b, nprev - 1) * dstride, off_d);
  // slot `lane` of row o
  const float pov = ld_off(M.part + (o - base), 4u * (uint32_t)min(lane, nt - 1) * (uint32_t)n);
  constexpr int QU = 8;
  float qv[QU];
#pragma unroll
  for (int k = 0; k < QU; ++k) qv[k] = ld_off(M.qpart, 4u * (uint32_t)min(tid + RB * k, ntile - 1));

  float ysl = 0.f;
#pragma unroll
  for (int q = 0; q < 32; ++q) ysl += q < nt ? ts[q] : 0.f;
  for (int q = 32; q < nt; ++q) ysl += pp[(int64_t)q * n];
#pragma unroll
  for (int p = 0; p < 32; ++p)
    if (p >= j) { vrow[p] = 0.f; wrow[p] = 0.f; }
  if (tid >= j) { w_o = 0.f; v_o = 0.f; }
  // sigma and the dots, summed over the row blocks in the order b = 0, 1, ... (fp64)
  if (tid < 2 * j + 1) {
    double sd = 0.0;
#pragma unroll
    for (int b = 0; b < 32; ++b) sd += b < nprev ? (double)td[b] : 0.0;
    for (int b = 32; b < nprev; ++b) sd += (double)dp[(int64_t)b * dstride];
    if (tid == 0) sh_sigma = sd;
    else if (tid <= j) pw[tid - 1] = (float)sd;
    else pv[tid - 1 - j] = (float)sd;
  }
  if (tid < j) { cw[tid] = w_o; cv[tid] = v_o; }
  // x_tail^T A22 x_tail: per-thread sums over tiles t = tid + RB k, then the block (fp64)
  double qs = 0.0;
#pragma unroll
  for (int k = 0; k < QU; ++k) qs += tid + RB * k < ntile ? (double)qv[k] : 0.0;
  for (int t = tid + RB * QU; t < ntile; t += RB) qs += (double)M.qpart[t];
  qs = wave_sum(qs);
  if (lane == 0) red[wave] = qs;
  __syncthreads();
  const double qsum = red[0] + red[1];
  double beta, tv, scal;
  householder(alpha, sh_sigma, beta, tv, scal);
  const float sc = (float)scal, tf = (float)tv;
  // W^T v = scal W^T x_tail + W[o, :] and V^T v = scal V^T x_tail + V[o, :] (v = e_o +
  // scal x_tail, x_tail[o] = 0) are formed where used, from the raw dots and row o in LDS.
  // y[o] (lane p < j takes correction p, lane q < nt slot q of row o; wave sums, so every
  // wave has the same value) and alpha2 = -(tau^2 / 2) y^T v
  float tcorr = 0.f;
  double tpvw = 0.0;
  if (lane < j) {
    const float pwf = fmaf(sc, pw[lane], cw[lane]), pvf = fmaf(sc, pv[lane], cv[lane]);
    tcorr = fmaf(cv[lane], pwf, cw[lane] * pvf);
    tpvw = (double)pvf * (double)pwf;
  }
  const float ysl_o = wave_sum(lane < nt ? pov : 0.f);
  const float y_o = fmaf(sc, ysl_o, a_oo) - wave_sum(tcorr);
  const double pvw = wave_sum(tpvw);
  const double vav = (double)a_oo + 2.0 * scal * (double)ysl_o + scal * scal * qsum;
  const float alpha2 = tv == 0.0 ? 0.f : (float)(-0.5 * (double)tf * (double)tf * (vav - 2.0 * pvw));
  float vr = 0.f, w = 0.f;
  if (r < n) {
    vr = (r == o) ? 1.f : (tv == 0.0 ? 0.f : sc * x_r);
    float y = fmaf(sc, ysl, a_o);
#pragma unroll
    for (int p = 0; p < 32; ++p)
      if (p < j) y -= fmaf(vrow[p], fmaf(sc, pw[p], cw[p]), wrow[p] * fmaf(sc, pv[p], cv[p]));
    if (r == o) y = y_o;                          // row o: the value every workgroup uses
    const float wp = (tv == 0.0) ? 0.f : tf * y;
    w = fmaf(alpha2, vr, wp);
    V[(int64_t)j * n + r] = vr;
    Qv[(int64_t)j * n + r] = vr;
    M.A[(int64_t)r * n + i] = vr;                 // reflector kept for the back-transformation
    W[(int64_t)j * n + r] = w;
    M.Q[(int64_t)j * n + r] = w;
  }
  if (blockIdx.x == 0 && tid == 0) { M.d[i] = scur[1]; M.e[i] = beta; M.tau[i] = (float)tv; }
  if (!more) return;

  // column o = i + 1: x[r] = A[o][r] - sum_{p <= j} (V[p][r] W[p][o] + W[p][r] V[p][o]), r >= o,
  // with V[j][o] = 1 and W[j][o] = tau y[o] + alpha2
  const int jp = j + 1;
  const float cw_j = fmaf(alpha2, 1.f, tv == 0.0 ? 0.f : tf * y_o);
  float xtail = 0.f;
  if (r < n) {
    float x = a_o;
#pragma unroll
    for (int p = 0; p < 32; ++p)
      if (p < j) x -= fmaf(vrow[p], cw[p], wrow[p] * cv[p]);
    x -= fmaf(vr, cw_j, w);
    if (r == o) snext[1] = x;
    if (r == o + 1) snext[0] = x;
    xtail = (r > o + 1) ? x : 0.f;
    M.xt[r] = xtail;
  }
  // partials over this block's rows of the next column's sigma = x_tail^T x_tail and of
  // W_p^T x_tail, V_p^T x_tail (p <= j), in that order
  __shared__ float prod[2 * 32 + 1][RB];
  const int nk = 2 * jp + 1;
  prod[0][tid] = xtail * xtail;
#pragma unroll
  for (int p = 0; p < 32; ++p)
    if (p < jp) {
      const float vp = p == j ? vr : vrow[p], wq = p == j ? w : wrow[p];
      prod[1 + p][tid] = wq * xtail;
      prod[1 + jp + p][tid] = vp * xtail;
    }
  __syncthreads();
  if (tid < nk) {
    // four interleaved partial sums, combined in a fixed order
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int t = 0; t < RB; t += 4)
#pragma unroll
      for (int q = 0; q < 4; ++q) s4[q] += prod[tid][t + q];
    dnext[(int64_t)blockIdx.x * dstride + tid] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
  }
}
__global__ void __launch_bounds__(256) k_symv_tiles(SytrdArgs a, int i) {
  // odd columns walk the matrices and tiles in reverse, so a pass starts on the data the
  // previous pass touched last (still cache-resident when the matrices exceed the caches)
  const bool rev = i & 1;
  const int mat = rev ? gridDim.y - 1 - blockIdx.y : blockIdx.y;
  const int n = a.n, o = i + 1;
  const int base = o & ~31, Lb = n - base;
  const MatView M = view(a, mat);
  const int tile = rev ? gridDim.x - 1 - blockIdx.x : blockIdx.x;
  int I, J;
  tri_decode(tile, I, J);
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4, lane = tid & 63, wave = tid >> 6;
  const int r0 = I * TB + ty * 8;                             // relative to base
  // column of register c (relative to base): two runs of four
  auto ccol = [&](int c) { return J * TB + (c < 4 ? tx * 4 + c : 64 + tx * 4 + c - 4); };
  const float *xt = M.xt;
  float xr[8], xc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int gr = base + r0 + k, gc = base + ccol(k);
    xr[k] = (gr >= o + 1 && gr < n) ? xt[gr] : 0.f;     // x_tail is zero at o and above it
    xc[k] = (gc >= o + 1 && gc < n) ? xt[gc] : 0.f;
  }
  float rs[8], cs[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) { rs[k] = 0.f; cs[k] = 0.f; }
  const bool diag = (I == J);
  // All 16 row loads are issued before any is consumed: rows outside [o, n) read a clamped
  // in-range row and are zeroed afterwards, so no load sits behind a branch.
  const int gc0 = base + ccol(0), gc4 = base + ccol(4);
  float v[8][8];
  if (gc4 + 4 <= n) {
    float4 u[8][2];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int gr = min(max(base + r0 + k, o), n - 1);
      const float *row = M.A + (int64_t)gr * n;
      u[k][0] = *reinterpret_cast<const float4 *>(row + gc0);
      u[k][1] = *reinterpret_cast<const float4 *>(row + gc4);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int gr = base + r0 + k;
      const float rm = (gr >= o && gr < n) ? 1.f : 0.f;
      v[k][0] = u[k][0].x * rm; v[k][1] = u[k][0].y * rm; v[k][2] = u[k][0].z * rm; v[k][3] = u[k][0].w * rm;
      v[k][4] = u[k][1].x * rm; v[k][5] = u[k][1].y * rm; v[k][6] = u[k][1].z * rm; v[k][7] = u[k][1].w * rm;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int gr = base + r0 + k;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int gc = base + ccol(c);
        v[k][c] = (gr >= o && gr < n && gc < n) ? M.A[(int64_t)gr * n + gc] : 0.f;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) {
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int gc = base + ccol(c);
      const float e = (gc >= o) ? v[k][c] : 0.f;
      if (diag) {
        // lower part only: row sums take col <= row, column sums take col < row
        const bool le = ccol(c) <= (r0 + k), lt = ccol(c) < (r0 + k);
        rs[k] = fmaf(le ? e : 0.f, xc[c], rs[k]);
        cs[c] = fmaf(lt ? e : 0.f, xr[k], cs[c]);
      } else {
        rs[k] = fmaf(e, xc[c], rs[k]);
        cs[c] = fmaf(e, xr[k], cs[c]);
      }
    }
  }
  // row sums: reduce over tx (16 consecutive lanes)
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float v = rs[k];
    v += __shfl_xor(v, 1, 64); v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 4, 64); v += __shfl_xor(v, 8, 64);
    rs[k] = v;
  }
  // column sums: reduce over ty (lanes 16 apart in a wave, then the four waves)
  __shared__ float csh[4][TB];
  __shared__ float rsh[TB];
  __shared__ float qsh[4];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    float v = cs[c];
    v += __shfl_xor(v, 16, 64); v += __shfl_xor(v, 32, 64);
    cs[c] = v;
  }
  {
    // this wave's term of x_tail^T A22 x_tail: its 32 rows' sums and its column partials
    float qc = 0.f;
    if (tx == 0) {
#pragma unroll
      for (int k = 0; k < 8; ++k) qc = fmaf(xr[k], rs[k], qc);
    }
    if (lane < 16) {
#pragma unroll
      for (int c = 0; c < 8; ++c) qc = fmaf(xc[c], cs[c], qc);
    }
    qc = wave_sum(qc);
    if (lane == 0) qsh[wave] = qc;
  }
  if (lane < 16) {
#pragma unroll
    for (int c = 0; c < 8; ++c) csh[wave][ccol(c) - J * TB] = cs[c];
  }
  if (tx == 0) {
#pragma unroll
    for (int k = 0; k < 8; ++k) rsh[ty * 8 + k] = rs[k];
  }
  __syncthreads();
  float *part = M.part;
  if (tid == 0) M.qpart[tile] = (qsh[0] + qsh[1]) + (qsh[2] + qsh[3]);
  if (tid < TB) {
    const float colsum = csh[0][tid] + csh[1][tid] + csh[2][tid] + csh[3][tid];
    const int rr = I * TB + tid, cc = J * TB + tid;
    if (diag) {
      if (rr < Lb) part[(int64_t)I * n + rr] = rsh[tid] + colsum;
    } else {
      if (rr < Lb) part[(int64_t)J * n + rr] = rsh[tid];
      if (cc < Lb) part[(int64_t)I * n + cc] = colsum;
    }
  }
}

// First column k0 of a panel (no reflector of the panel applies yet): x = A[k0][r] for
// r >= k0, its scalars and the block partials of its sigma, into the buffers of column k0's
// parity.
__global__ void __launch_bounds__(RB) k_col_first(SytrdArgs a, int k0) {
  const int mat = blockIdx.y, n = a.n;
  const MatView M = view(a, mat);
  const int64_t dstride = 2 * a.nb + 1;
  float *dnext = M.dpart + (k0 & 1) * (int64_t)a.slots * dstride;
  float *snext = M.sc + 2 * (k0 & 1);
  const int tid = threadIdx.x;
  const int r = k0 + blockIdx.x * RB + tid;
  float xtail = 0.f;
  if (r < n) {
    const float x = M.A[(int64_t)k0 * n + r];
    if (r == k0) snext[1] = x;
    if (r == k0 + 1) snext[0] = x;
    xtail = (r > k0 + 1) ? x : 0.f;
    M.xt[r] = xtail;
  }
  __shared__ float prod[RB];
  prod[tid] = xtail * xtail;
  __syncthreads();
  if (tid == 0) {
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < RB; t += 4)
#pragma unroll
      for (int q = 0; q < 4; ++q) s4[q] += prod[t + q];
    dnext[(int64_t)blockIdx.x * dstride] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
  }
}

// After a lower-triangle trailing update, copy the lower triangle into the upper part of
// rows s .. s+nb (the rows the next panel reads as rows): A[r][c] = A[c][r] for c > r.
// One workgroup per 64-column chunk; the (nb+1) x 64 block is transposed through LDS.
__global__ void __launch_bounds__(256) k_mirror_strip(SytrdArgs a, int s) {
  const int mat = blockIdx.y, n = a.n, nb = a.nb;
  float *A = a.A + (int64_t)mat * a.mat_stride;
  const int rows = min(nb + 1, n - s);
  const int c0 = s + blockIdx.x * 64;
  __shared__ float t[64][65];
  const int tid = threadIdx.x;
  for (int q = tid; q < 64 * 64; q += 256) {
    const int cc = q / 64, rr = q % 64;          // read A[c0 + cc][s + rr]: rows contiguous in rr
    const int c = c0 + cc, r = s + rr;
    t[cc][rr] = (rr < rows && c < n && c > r) ? A[(int64_t)c * n + r] : 0.f;
  }
  __syncthreads();
  for (int q = tid; q < 64 * 64; q += 256) {
    const int rr = q / 64, cc = q % 64;          // write A[s + rr][c0 + cc]
    const int c = c0 + cc, r = s + rr;
    if (rr < rows && c < n && c > r) A[(int64_t)r * n + c] = t[cc][rr];
  }
}

__global__ void __launch_bounds__(64) k_sytrd_finish(SytrdArgs a) {
  const int mat = blockIdx.x, n = a.n;
  float *A = a.A + (int64_t)mat * a.mat_stride;
  if (threadIdx.x == 0) {
    a.d[(int64_t)mat * n + n - 1] = A[(int64_t)(n - 1) * n + (n - 1)];
    a.e[(int64_t)mat * n + n - 1] = 0.0;
    a.tau[(int64_t)mat * n + n - 1] = 0.f;
  }
}

// zero the upper triangle and diagonal of the reflector block (dense V for the back-transform)
__global__ void k_reflector_clean(SytrdArgs a) {
  const int mat = blockIdx.y, n = a.n;
  float *A = a.A + (int64_t)mat * a.mat_stride;
  const int64_t total = (int64_t)n * n;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(q / n), c = (int)(q % n);
    if (c >= r || c == n - 1) A[q] = 0.f;
  }
}

size_t per_mat_floats(int n, int nb) {
  const size_t slots = (n + TB - 1) / TB;
  return 4 * (size_t)nb * n + (size_t)n + slots * n + 2 * slots * (2 * nb + 1) + slots * (slots + 1) / 2 + 64;
}

}  // namespace

size_t sytrd_large_work_floats(int n_mat, int n, int nb) {
  return (size_t)n_mat * ((per_mat_floats(n, nb) + 63) / 64 * 64);
}

size_t sytrd_large_table_entries(int n_mat, int n, int nb) {
  const int panels = (n - 1 + nb - 1) / nb;
  return (size_t)panels * n_mat;
}

void sytrd_large_tables(const EigBatch &b, float *work, int nb, GemmProblem *tab_host) {
  const int n = b.n, nm = b.n_mat;
  const int64_t ws = (int64_t)((per_mat_floats(n, nb) + 63) / 64 * 64);
  const int panels = (n - 1 + nb - 1) / nb;
  // one fused rank-2jb update per panel: A22 -= P^T Q with P = [V; W], Q = [W; V]
  for (int p = 0; p < panels; ++p) {
    const int k0 = p * nb, jb = std::min(nb, n - 1 - k0), s = k0 + jb, rem = n - s;
    for (int m = 0; m < nm; ++m) {
      float *A = b.A + (int64_t)m * b.mat_stride;
      const float *P = work + (int64_t)m * ws;
      const float *Q = P + (int64_t)2 * nb * n;
      GemmProblem g{};
      g.A = GemmOperand{P + s, n, 0, 0, 0, 1};    // A(m = r, k = p) = P[p][s + r]
      g.B = GemmOperand{Q + s, n, 0, 0, 0, 1};    // B(k = p, n = c) = Q[p][s + c]
      g.C = A + (int64_t)s * n + s; g.ldc = n;
      g.M = rem; g.N = rem; g.K = 2 * jb; g.alpha = -1.f; g.beta = 1.f;
      g.lower_only = 1;   // the upper part of the next panel's rows is restored by k_mirror_strip
      tab_host[(size_t)p * nm + m] = g;
    }
  }
}

hipError_t launch_sytrd_large(const EigBatch &b, float *work, int nb, const GemmProblem *tab_dev,
                              hipStream_t st, int m0, int m1) {
  // matrices m0 .. m1-1 of the batch (all by default)
  const int n = b.n;
  if (m1 < 0) m1 = b.n_mat;
  const int nm = m1 - m0;
  if (nm <= 0 || m0 < 0 || m1 > b.n_mat) return hipErrorInvalidValue;
  if (nb > 32) return hipErrorInvalidValue;     // k_col_step holds the 2 nb + 1 dots of a block
  if (n > TRD_MAX_N) return hipErrorInvalidValue;
  const int64_t wstride = (int64_t)((per_mat_floats(n, nb) + 63) / 64 * 64);
  SytrdArgs a{};
  a.A = b.A + (int64_t)m0 * b.mat_stride; a.mat_stride = b.mat_stride; a.n = n; a.nb = nb;
  a.d = b.d + (int64_t)m0 * n; a.e = b.e + (int64_t)m0 * n; a.tau = b.tau + (int64_t)m0 * n;
  a.work = work + m0 * wstride;
  a.work_stride = wstride;
  a.slots = (n + TB - 1) / TB;
  const int panels = (n - 1 + nb - 1) / nb;
  hipError_t err = hipSuccess;
  // only the lower triangle (and the diagonal tiles) of the input is read: the upper part of
  // the first panel's rows is restored from it here, that of later panels after each update
  hipLaunchKernelGGL(k_mirror_strip, dim3((n + 63) / 64, nm), dim3(256), 0, st, a, 0);
  for (int p = 0; p < panels; ++p) {
    const int k0 = p * nb, jb = std::min(nb, n - 1 - k0);
    hipLaunchKernelGGL(k_col_first, dim3((n - k0 + RB - 1) / RB, nm), dim3(RB), 0, st, a, k0);
    for (int j = 0; j < jb; ++j) {
      const int i = k0 + j, o = i + 1, L = n - o;
      const int nt = (n - (o & ~31) + TB - 1) / TB, nblk = (L + RB - 1) / RB;
      hipLaunchKernelGGL(k_symv_tiles, dim3(nt * (nt + 1) / 2, nm), dim3(256), 0, st, a, i);
      hipLaunchKernelGGL(k_col_step, dim3(nblk, nm), dim3(RB), 0, st, a, i, j, jb, j + 1 < jb ? 1 : 0);
    }
    const int s = k0 + jb;
    if (s < n) {
      err = launch_update3(tab_dev + (size_t)p * b.n_mat + m0, nm, n - s, st);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL(k_mirror_strip, dim3((n - s + 63) / 64, nm), dim3(256), 0, st, a, s);
    }
  }
  hipLaunchKernelGGL(k_sytrd_finish, dim3(nm), dim3(64), 0, st, a);
  hipLaunchKernelGGL(k_reflector_clean, dim3(1024, nm), dim3(256), 0, st, a);
  return hipGetLastError();
}

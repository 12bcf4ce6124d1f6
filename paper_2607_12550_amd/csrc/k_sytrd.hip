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
//   k_col_finish  per 128-row block: tau, v, y, w_pre = tau y, partial w_pre^T v;
//   k_col_next    per 128-row block: w = w_pre + alpha2 v, the next column's x and the
//                 block partials of its sigma and dot products.
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

JOLT_DEV void tri_decode(int t, int &I, int &J) {
  int i = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while ((i + 1) * (i + 2) / 2 <= t) ++i;
  while (i * (i + 1) / 2 > t) --i;
  I = i;
  J = t - i * (i + 1) / 2;
}

struct MatView {
  float *A, *P, *Q, *xt, *wpre, *part, *dpart, *wpart, *sc;
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
  m.wpre = m.xt + n;
  m.part = m.wpre + n;
  m.dpart = m.part + (int64_t)a.slots * n;
  m.wpart = m.dpart + (int64_t)a.slots * (2 * nb + 1);
  m.sc = m.wpart + a.slots;          // [0] alpha, [1] diagonal
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
// ty (shuffles, then LDS across the four waves).  Tiles (I, 0) also produce the
// dot partials [sigma, W_p^T x, V_p^T x] over their 128 rows.
JOLT_DEV void householder(float alpha, double sigma, double &beta, double &tv, double &scal) {
  if (sigma == 0.0) { tv = 0.0; beta = alpha; scal = 0.0; return; }
  beta = -copysign(sqrt((double)alpha * alpha + sigma), (double)alpha);
  tv = (beta - alpha) / beta;
  scal = 1.0 / (alpha - beta);
}

__global__ void __launch_bounds__(RB) k_col_finish(SytrdArgs a, int i, int j, int jbw) {
  const int mat = blockIdx.y, n = a.n, nb = a.nb, o = i + 1;
  const int base = o & ~31, nt = (n - base + TB - 1) / TB;
  const int nprev = (n - i + RB - 1) / RB;     // row blocks of the k_col_next launch that made x
  const MatView M = view(a, mat);
  __shared__ float pw[64], pv[64];
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
  // trip before its barrier.
  const float *pp = M.part + (rr - base);
  float ts[32];
#pragma unroll
  for (int q = 0; q < 32; ++q) ts[q] = pp[(int64_t)min(q, nt - 1) * n];
  const float a_o = M.A[(int64_t)o * n + rr];   // A22[:, 0] (row o by symmetry)
  const float x_r = M.xt[rr];
  // row f of V is not written by this launch (it writes row j only)
  const int f = j == 0 ? 1 : 0;
  float vrow[32], wrow[32];
#pragma unroll
  for (int p = 0; p < 32; ++p) {
    vrow[p] = V[(int64_t)(p < j ? p : f) * n + rr];
    wrow[p] = W[(int64_t)(p < j ? p : 0) * n + rr];
  }
  float w_o = W[(int64_t)(tid < j ? tid : 0) * n + o];
  float v_o = V[(int64_t)(tid < j ? tid : f) * n + o];
  const float alpha = M.sc[0];
  const int64_t dstride = 2 * nb + 1;
  const float *dp = M.dpart + min(tid, 2 * j);  // dot of this thread: 0 sigma, then W, V
  float td[32];
#pragma unroll
  for (int b = 0; b < 32; ++b) td[b] = dp[(int64_t)min(b, nprev - 1) * dstride];
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
  __syncthreads();
  double beta, tv, scal;
  householder(alpha, sh_sigma, beta, tv, scal);
  const float sc = (float)scal, tf = (float)tv;
  // W^T v = scal W^T x_tail + W[o, :]  (v = e_o + scal x_tail, x_tail[o] = 0)
  if (tid < j) {
    pw[tid] = sc * pw[tid] + w_o;
    pv[tid] = sc * pv[tid] + v_o;
  }
  __syncthreads();
  double dot = 0.0;
  if (r < n) {
    const float vr = (r == o) ? 1.f : (tv == 0.0 ? 0.f : sc * x_r);
    float y = sc * ysl + a_o;
#pragma unroll
    for (int p = 0; p < 32; ++p)
      if (p < j) y -= vrow[p] * pw[p] + wrow[p] * pv[p];
    const float wp = (tv == 0.0) ? 0.f : tf * y;
    M.wpre[r] = wp;
    V[(int64_t)j * n + r] = vr;
    Qv[(int64_t)j * n + r] = vr;
    M.A[(int64_t)r * n + i] = vr;                 // reflector kept for the back-transformation
    dot = (double)wp * (double)vr;
  }
  dot = wave_sum(dot);
  if (lane == 0) red[wave] = dot;
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < RB / 64; ++w) s += red[w];
    M.wpart[blockIdx.x] = (float)s;
    if (blockIdx.x == 0) { M.d[i] = M.sc[1]; M.e[i] = beta; M.tau[i] = (float)tv; }
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
  int I, J;
  tri_decode(rev ? gridDim.x - 1 - blockIdx.x : blockIdx.x, I, J);
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
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    float v = cs[c];
    v += __shfl_xor(v, 16, 64); v += __shfl_xor(v, 32, 64);
    cs[c] = v;
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

__global__ void __launch_bounds__(RB) k_col_next(SytrdArgs a, int i, int j, int ip, int jp,
                                                 int prep_only, int jbw) {
  const int mat = blockIdx.y, n = a.n;
  const MatView M = view(a, mat);
  float *V = M.P, *W = M.P + (int64_t)jbw * n;
  __shared__ float cw[64], cv[64];
  __shared__ float alpha2_s;
  const int tid = threadIdx.x;
  // rows from ip (= i + 1 = o of column i unless prep_only) in blocks of 128, one per thread
  const int r = (prep_only ? ip : i + 1) + blockIdx.x * RB + tid;
  const int rr = r < n ? r : n - 1;             // in-range row for the loads
  const bool next = ip < n - 1;
  // Every load that does not need alpha2 is issued before any is used and without a branch
  // (panel rows p < j of V and W at this row and at row ip, row ip of A, what rebuilds w_j
  // and the block partials of w^T v): entries past the live range read an entry this
  // launch does not write and are masked afterwards.
  const int ipc = min(ip, n - 1);
  // row g of W is not written by this launch (it writes row j only, and none in prep_only)
  const int g = j == 0 ? 1 : 0;
  float vrow[32], wrow[32];
#pragma unroll
  for (int p = 0; p < 32; ++p) {
    const bool ld = p < jp && (prep_only || p < j);
    vrow[p] = V[(int64_t)(ld ? p : 0) * n + rr];
    wrow[p] = W[(int64_t)(ld ? p : g) * n + rr];
  }
  float a_ip = M.A[(int64_t)ipc * n + rr];
  const bool ldc = tid < jp, ldw = ldc && (prep_only || tid < j);
  float cv_t = V[(int64_t)(ldc ? tid : 0) * n + ipc];
  float cw_t = W[(int64_t)(ldw ? tid : g) * n + ipc];
  float wpre_r = 0.f, vj_r = 0.f, wpre_ip = 0.f, vj_ip = 0.f, tau_i = 0.f, tw[32];
  const int nblk = (n - (i + 1) + RB - 1) / RB;   // row blocks of column i's k_col_finish
  if (!prep_only) {
    wpre_r = M.wpre[rr];
    vj_r = V[(int64_t)j * n + rr];
    wpre_ip = M.wpre[ipc];
    vj_ip = V[(int64_t)j * n + ipc];
    tau_i = M.tau[i];
#pragma unroll
    for (int b = 0; b < 32; ++b) tw[b] = M.wpart[min(b, nblk - 1)];
  }
#pragma unroll
  for (int p = 0; p < 32; ++p)
    if (!(next && p < jp && (prep_only || p < j))) { vrow[p] = 0.f; wrow[p] = 0.f; }
  if (!next) a_ip = 0.f;
  if (!(next && ldc)) cv_t = 0.f;
  if (!(next && ldw)) cw_t = 0.f;
  float alpha2 = 0.f, w = 0.f;
  if (!prep_only) {
    vrow[j] = vj_r;
    if (tid == 0) {
      double sw = 0.0;
#pragma unroll
      for (int b = 0; b < 32; ++b) sw += b < nblk ? (double)tw[b] : 0.0;
      for (int b = 32; b < nblk; ++b) sw += (double)M.wpart[b];
      alpha2_s = (float)(-0.5 * (double)tau_i * sw);
    }
    __syncthreads();
    alpha2 = alpha2_s;
    w = wpre_r + alpha2 * vj_r;
    wrow[j] = w;
    if (r < n) {
      W[(int64_t)j * n + r] = w;
      M.Q[(int64_t)j * n + r] = w;
    }
    if (!next) return;
    // reflector j's w[ip] is rebuilt here because another workgroup of this launch writes it
    if (tid == j) cw_t = wpre_ip + alpha2 * vj_ip;
  }
  if (tid < jp) { cw[tid] = cw_t; cv[tid] = cv_t; }
  __syncthreads();
  // x[r] = A[ip][r] - sum_p (V[p][r] W[p][ip] + W[p][r] V[p][ip]) for r >= ip (row ip = column ip)
  float xtail = 0.f;
  if (r < n) {
    float x = a_ip;
#pragma unroll
    for (int p = 0; p < 32; ++p)
      if (p < jp) x -= vrow[p] * cw[p] + wrow[p] * cv[p];
    if (r == ip) M.sc[1] = x;
    if (r == ip + 1) M.sc[0] = x;
    xtail = (r > ip + 1) ? x : 0.f;
    M.xt[r] = xtail;
  }
  // partials over this block's rows of the next column's sigma = x_tail^T x_tail and of
  // W_p^T x_tail, V_p^T x_tail (p < jp), in that order; summed over blocks by k_col_finish
  __shared__ float prod[2 * 32 + 1][RB];
  const int nk = 2 * jp + 1;
  prod[0][tid] = xtail * xtail;
#pragma unroll
  for (int p = 0; p < 32; ++p)
    if (p < jp) { prod[1 + p][tid] = wrow[p] * xtail; prod[1 + jp + p][tid] = vrow[p] * xtail; }
  __syncthreads();
  if (tid < nk) {
    // four interleaved partial sums, combined in a fixed order
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int t = 0; t < RB; t += 4)
#pragma unroll
      for (int q = 0; q < 4; ++q) s4[q] += prod[tid][t + q];
    M.dpart[(int64_t)blockIdx.x * (2 * a.nb + 1) + tid] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
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
  return 4 * (size_t)nb * n + 2 * (size_t)n + slots * n + slots * (2 * nb + 1) + slots + 64;
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
  if (nb > 32) return hipErrorInvalidValue;     // k_col_next's partial buffer holds 2 nb + 1 dots
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
    hipLaunchKernelGGL(k_col_next, dim3((n - k0 + RB - 1) / RB, nm), dim3(RB), 0, st, a, -1, 0, k0, 0, 1, jb);
    for (int j = 0; j < jb; ++j) {
      const int i = k0 + j, o = i + 1, L = n - o;
      const int nt = (n - (o & ~31) + TB - 1) / TB, nblk = (L + RB - 1) / RB;
      hipLaunchKernelGGL(k_symv_tiles, dim3(nt * (nt + 1) / 2, nm), dim3(256), 0, st, a, i);
      hipLaunchKernelGGL(k_col_finish, dim3(nblk, nm), dim3(RB), 0, st, a, i, j, jb);
      const bool more = j + 1 < jb;
      hipLaunchKernelGGL(k_col_next, dim3(nblk, nm), dim3(RB), 0, st, a, i, j, more ? i + 1 : n, j + 1, 0, jb);
    }
    const int s = k0 + jb;
    if (s < n) {
      err = launch_gemm(tab_dev + (size_t)p * b.n_mat + m0, nm, n - s, n - s, 1, GT_F32, GT_F32, false, false, st);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL(k_mirror_strip, dim3((n - s + 63) / 64, nm), dim3(256), 0, st, a, s);
    }
  }
  hipLaunchKernelGGL(k_sytrd_finish, dim3(nm), dim3(64), 0, st, a);
  hipLaunchKernelGGL(k_reflector_clean, dim3(1024, nm), dim3(256), 0, st, a);
  return hipGetLastError();
}

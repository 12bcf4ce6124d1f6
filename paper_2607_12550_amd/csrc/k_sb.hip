// Two-stage tridiagonalisation of the large symmetric matrices of the exact token mode
// (C = X_(2) X_(2)^T of section 4, T in the thousands), batched over matrices of one size.
//
// Stage 1 (dense to band, half-bandwidth SB = 32), per panel of SB columns k0 .. k0 + 31
// with the rows below the band r0 = k0 + SB .. n - 1 (m = n - r0 of them):
//   QR of the m x SB panel by Householder reflectors, Q = H_0 ... H_31 = I - V T V^T
//   (V explicit, unit lower trapezoidal; T upper triangular), R into the band;
//   X = A22 V T, Y = V^T X, Z = X - (1/2) V T^T Y;
//   A22 <- Q^T A22 Q = A22 - V Z^T - Z V^T   (the rank-2SB update on the matrix cores).
// The trailing matrix is read and written once per panel instead of once per column, so
// the one-stage reduction's per-column mat-vec over A22 disappears.
//
// Stage 2 (band to tridiagonal) chases bulges: sweep s annihilates column s below its
// subdiagonal with a reflector on rows s+1 .. s+SB, applied on both sides of the diagonal
// block and from the right to the block below; the fill this makes in that block's first
// column is annihilated by the next reflector of the sweep, and so on to the end of the
// band.  Each step touches three SB x SB blocks (the previous bulge block, the diagonal
// block and the block below) of a band buffer holding 2 SB entries per column; sweep s + 1
// may run step k once sweep s has completed step k + 2 (k + 3 here, so that the next step's
// blocks can be loaded during the current one).  One workgroup per matrix, one wavefront per
// sweep in flight, the dependencies between wavefronts kept in LDS.
//
// Eigenvectors: z of the tridiagonal -> Q2 z (the stage-2 reflectors in blocks of 32 sweeps
// at one step, groups of sweeps last to first, steps in increasing order within a group) ->
// Q1 (Q2 z) (stage-1 reflectors by the blocked WY back-transform, with the unit of
// reflector i at row i + SB).
//
// Which of this and the one-stage reduction runs is the caller's choice (by batch size:
// the bulge chase is a chain of about n^2 / 64 dependent steps per matrix, hidden only when
// enough matrices run side by side).
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace {

constexpr int SB = 32;            // half-bandwidth of the intermediate band
constexpr int SBW = 2 * SB;       // band-buffer entries per column (band and bulge)
constexpr int PQ_NT = 1024;       // panel QR: threads per matrix
constexpr int SY_ROWS = 128;      // rows of X per workgroup of the symmetric product
constexpr int SY_NT = 256;
constexpr int BG_WAVES = 8;       // bulge chase: wavefronts (sweeps in flight) per matrix
constexpr int BT_BLOCK = 128;     // reflectors per block of the stage-1 back-transform

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__host__ __device__ inline int steps_max(int n) { return n >= 3 ? (n - 3) / SB + 1 : 1; }

struct SbView {
  float *A, *P, *Q, *X, *Yp, *Sp, *AB, *V2, *VTb;
  double *d, *e;
  float *tau;
};

__host__ __device__ inline size_t sb_per_mat(int n) {
  const size_t km = n >= 3 ? (size_t)((n - 3) / SB + 1) : 1;
  const size_t nblk = (size_t)((n + SY_ROWS - 1) / SY_ROWS);
  const size_t f = 4 * (size_t)SB * n + (size_t)n * SB + 2 * nblk * SB * SB + (size_t)n * SBW +
                   (size_t)n * km * SB + km * (km + 1) / 2 * 2 * SB * SB + 64;
  return (f + 63) / 64 * 64;
}

JOLT_DEV SbView sview(const SbArgs &a, int mat) {
  const int n = a.n;
  SbView v;
  v.A = a.A + (int64_t)mat * a.mat_stride;
  float *w = a.work + (int64_t)mat * a.work_stride;
  const int nblk = (n + SY_ROWS - 1) / SY_ROWS;
  v.P = w;
  v.Q = v.P + (int64_t)2 * SB * n;
  v.X = v.Q + (int64_t)2 * SB * n;
  v.Yp = v.X + (int64_t)n * SB;
  v.Sp = v.Yp + (int64_t)nblk * SB * SB;
  v.AB = v.Sp + (int64_t)nblk * SB * SB;
  v.V2 = v.AB + (int64_t)n * SBW;
  v.VTb = v.V2 + (int64_t)n * steps_max(n) * SB;     // V T of each block of 32 sweeps
  v.d = a.d + (int64_t)mat * n;
  v.e = a.e + (int64_t)mat * n;
  v.tau = a.tau + (int64_t)mat * n;
  return v;
}

JOLT_DEV void house(float alpha, float sigma, float &tau, float &beta, float &scal) {
  if (sigma == 0.f) { tau = 0.f; beta = alpha; scal = 0.f; return; }
  const double b = -copysign(sqrt((double)alpha * alpha + (double)sigma), (double)alpha);
  tau = (float)((b - alpha) / b);
  beta = (float)b;
  scal = (float)(1.0 / (alpha - b));
}

// base[idx] with a uniform base and a 32-bit element index: the access takes the
// scalar-base + vector-offset form, so no 64-bit address is kept per access
JOLT_DEV float ldx(const float *base, uint32_t idx) {
  return *reinterpret_cast<const float *>(reinterpret_cast<const char *>(base) + 4u * idx);
}
JOLT_DEV void stx(float *base, uint32_t idx, float v) {
  *reinterpret_cast<float *>(reinterpret_cast<char *>(base) + 4u * idx) = v;
}

// Lane exchanges without LDS: the sum over the lane pair (l, l + 32) by v_permlane32_swap
// (two copies of x leave the lower lane's value in r[0] and the upper's in r[1], in both
// lanes), a lane's value as a wave-uniform scalar by readlane, and the sum over lanes
// 0 .. 31 by DPP moves within rows of 16 (quad swaps, half-row and row mirrors) plus two
// readlanes.
JOLT_DEV float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
JOLT_DEV float lane_value(float x, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l)); }
JOLT_DEV float dpp_add(float x, int ctrl_sel) {
  int y;
  switch (ctrl_sel) {
    case 0: y = __builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false); break;   // lanes ^ 1
    case 1: y = __builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false); break;   // lanes ^ 2
    case 2: y = __builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false); break;  // half-row mirror
    default: y = __builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false); break; // row mirror
  }
  return x + __int_as_float(y);
}
JOLT_DEV float sum_lanes32(float x) {
  x = dpp_add(x, 0);
  x = dpp_add(x, 1);
  x = dpp_add(x, 2);
  x = dpp_add(x, 3);
  return lane_value(x, 0) + lane_value(x, 16);
}

// Workgroup barrier for LDS traffic only: waits for this wavefront's LDS operations, not for
// its global loads, so that loads issued before the barrier stay in flight across it.
JOLT_DEV void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

JOLT_DEV void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------- stage 1: panel QR
// One workgroup per matrix.  The panel stays in memory (the matrix's rows r0 .. n - 1,
// columns k0 .. k0 + 31); each column costs one pass over its live rows, which applies
// reflector j and forms the sums the next column needs: with g_c = sum_{r > j+1} x_r[j+1] x_r[c]
// (rows as updated by reflector j), sigma_{j+1} = g_{j+1} and
//   d_c = v_{j+1}^T P[:, c] = scal g_c + P[j+1][c]   for every c != j + 1,
// which are the apply-dots for c > j + 1 (columns left of j are neither read nor written
// by the pass; the block factor T is formed later from V^T V).
// Eight lanes share a row (four columns each), so a wavefront reads eight whole rows per
// load; the entries x_r[j] and x_r[j+1] are exchanged within the eight lanes.
// Writes: the diagonal block and R into the band buffer (zeros past the band), V explicit
// into the panel (unit at row j, zeros above, and zeros in the rows [blk + SB, r0) of the
// panel's columns, blk = k0 rounded down to the back-transform's block of 128 reflectors)
// and tau.
JOLT_DEV float pick4(const float (&x)[4], int u) {
  return u == 0 ? x[0] : (u == 1 ? x[1] : (u == 2 ? x[2] : x[3]));
}

__global__ void __launch_bounds__(PQ_NT) k_sb_panel(SbArgs a, int p, int mat0) {
  const int mat = mat0 + blockIdx.x, n = a.n;
  const SbView M = sview(a, mat);
  const int k0 = p * SB, r0 = k0 + SB, w = min(SB, n - k0), m = n - r0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float red[PQ_NT / 64][SB];
  __shared__ float rowj[SB], dv[SB];
  __shared__ float sc[4];
  for (int q = tid; q < SB * SBW; q += PQ_NT) {
    const int j = q / SBW, dd = q - j * SBW, row = k0 + j + dd;
    if (j >= w || row >= n) continue;
    if (dd < SB - j) M.AB[(int64_t)(k0 + j) * SBW + dd] = M.A[(int64_t)row * n + k0 + j];
    else if (dd > SB) M.AB[(int64_t)(k0 + j) * SBW + dd] = 0.f;
  }
  if (m <= 0) {
    if (tid < w) M.tau[k0 + tid] = 0.f;
    return;
  }
  const int jmax = min(m, SB);
  const int grp0 = lane & ~7, c4 = (lane & 7) * 4;
  const int rfirst = wave * 8 + (lane >> 3);
  constexpr int RSTEP = PQ_NT / 8;
  const bool vec = (n % 4 == 0) && ((reinterpret_cast<uintptr_t>(M.A) & 15) == 0);
  __syncthreads();
  for (int j = -1; j < jmax; ++j) {
    const int nj = j + 1;
    float tj = 0.f, sj = 0.f, bj = 0.f, d4[4] = {0.f, 0.f, 0.f, 0.f};
    if (j >= 0) {
      tj = sc[0]; bj = sc[1]; sj = sc[2];
#pragma unroll
      for (int u = 0; u < 4; ++u) d4[u] = dv[c4 + u];
    }
    float g4[4] = {0.f, 0.f, 0.f, 0.f};
    // eight rows per batch: their loads are issued together (the rows a thread stores are
    // never reloaded within the pass, but the compiler cannot prove it across iterations)
    constexpr int RB8 = 8;
    for (int rb = rfirst; rb < m; rb += RB8 * RSTEP) {
      float xb[RB8][4];
#pragma unroll
      for (int e = 0; e < RB8; ++e) {
        const int r = rb + e * RSTEP;
        const float *rp = M.A + (int64_t)(r0 + r) * n + k0 + c4;
        xb[e][0] = xb[e][1] = xb[e][2] = xb[e][3] = 0.f;
        if (r < m && r >= j && c4 + 3 >= j) {      // columns left of j take no part
          if (vec) {
            const jf4 v = gload_f4(rp);
            xb[e][0] = v[0]; xb[e][1] = v[1]; xb[e][2] = v[2]; xb[e][3] = v[3];
          } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) xb[e][u] = rp[u];
          }
        }
      }
#pragma unroll
      for (int e = 0; e < RB8; ++e) {
        const int r = rb + e * RSTEP;
        if (r >= m || r < j) continue;             // the eight lanes of a row agree
        float *rp = M.A + (int64_t)(r0 + r) * n + k0 + c4;
        float (&x)[4] = xb[e];
        if (j >= 0) {
          const float xj = __shfl(pick4(x, j & 3), grp0 | (j >> 2), 64);
          const float vr = (r == j) ? 1.f : xj * sj;
          const float tv = tj * vr;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int c = c4 + u;
            if (c > j) x[u] = fmaf(-tv, d4[u], x[u]);
            if (c == j) x[u] = vr;
          }
          if (r == j) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int c = c4 + u;
              if (c == j) M.AB[(int64_t)(k0 + j) * SBW + SB] = bj;
              if (c > j) { M.AB[(int64_t)(k0 + c) * SBW + SB + j - c] = x[u]; x[u] = 0.f; }
            }
          }
          if (c4 + 3 >= j) {                       // columns left of j are unchanged
            if (vec) {
              jf4 v;
              v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
              gstore_f4(rp, v);
            } else {
#pragma unroll
              for (int u = 0; u < 4; ++u) rp[u] = x[u];
            }
          }
        }
        if (nj < jmax) {
          if (r == nj) {
#pragma unroll
            for (int u = 0; u < 4; ++u) rowj[c4 + u] = x[u];
          }
          if (r > nj) {
            const float xn = __shfl(pick4(x, nj & 3), grp0 | (nj >> 2), 64);
#pragma unroll
            for (int u = 0; u < 4; ++u) g4[u] = fmaf(xn, x[u], g4[u]);
          }
        }
      }
    }
    if (nj >= jmax) break;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      g4[u] += shfl_xor(g4[u], 8);
      g4[u] += shfl_xor(g4[u], 16);
      g4[u] += shfl_xor(g4[u], 32);
    }
    if (lane < 8) {
#pragma unroll
      for (int u = 0; u < 4; ++u) red[wave][c4 + u] = g4[u];
    }
    __syncthreads();
    if (wave == 0) {
      float gsum = 0.f, rj = 0.f;
      if (lane < SB) {
#pragma unroll
        for (int q = 0; q < PQ_NT / 64; ++q) gsum += red[q][lane];
        rj = rowj[lane];
      }
      const float alpha = __shfl(rj, nj, 64), sig = __shfl(gsum, nj, 64);
      float t, b, sl;
      house(alpha, sig, t, b, sl);
      if (lane < SB) dv[lane] = (lane == nj) ? 0.f : fmaf(sl, gsum, rj);
      if (lane == 0) { sc[0] = t; sc[1] = b; sc[2] = sl; M.tau[k0 + nj] = t; }
    }
    __syncthreads();
  }
  if (tid >= jmax && tid < SB) M.tau[k0 + tid] = 0.f;
  __syncthreads();
  // zeros above the panel's reflectors inside their back-transform block
  const int z0 = (k0 / BT_BLOCK) * BT_BLOCK + SB;
  for (int q = tid; q < (r0 - z0) * SB; q += PQ_NT) {
    const int row = z0 + q / SB, c = q % SB;
    if (row < n) M.A[(int64_t)row * n + k0 + c] = 0.f;
  }
}

// ------------------------------------------------- stage 1: X = A22 V T and V^T X partials
// A22 = A[r0:, r0:] (lower triangle stored), V = the panel's explicit reflectors.  A
// workgroup owns 128 rows of X and sweeps all columns of A22 in chunks of 32: chunks left
// of its diagonal block are read as stored, chunks right of it transposed from the rows
// below, the diagonal chunks entry by entry.  fp32 MFMA 32x32x2 (four wavefronts, 32 rows
// each).  Epilogue: X1 stored, and this block's terms of V^T X1 and V^T V (the block
// factor T and X = X1 T are formed by the Z kernel).
struct SyLds {
  float As[SY_ROWS][SB + 1];
  float Vs[SB][SB + 1];
  float Vb[SY_ROWS][SB + 1];
};

__global__ void __launch_bounds__(SY_NT) k_sb_symm(SbArgs a, int p, int mat0) {
  const int mat = mat0 + blockIdx.y, n = a.n;
  const SbView M = sview(a, mat);
  const int k0 = p * SB, r0 = k0 + SB, m = n - r0;
  const int i0 = blockIdx.x * SY_ROWS;
  if (m < 2 || i0 >= m) return;
  __shared__ SyLds sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lr = lane & 31, lh = lane >> 5;
  const float *A22 = M.A + (int64_t)r0 * n + r0;
  float ra[16], rv[4];
  auto fetch = [&](int kc) {
    if (kc + SB <= i0) {                        // left of the diagonal block: stored rows
      const int j = tid & 31, ib = tid >> 5;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int R = i0 + ib + 8 * q, C = kc + j;
        ra[q] = (R < m) ? A22[(int64_t)R * n + C] : 0.f;
      }
    } else if (kc >= i0 + SY_ROWS) {            // right of it: the transposed rows below
      const int i = tid & 127, jb = tid >> 7;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int R = i0 + i, C = kc + jb + 2 * q;
        ra[q] = (R < m && C < m) ? A22[(int64_t)C * n + R] : 0.f;
      }
    } else {
      const int j = tid & 31, ib = tid >> 5;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int R = i0 + ib + 8 * q, C = kc + j;
        float v = 0.f;
        if (R < m && C < m) v = (R >= C) ? A22[(int64_t)R * n + C] : A22[(int64_t)C * n + R];
        ra[q] = v;
      }
    }
    const int c = tid & 31, kb = tid >> 5;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = kc + kb + 8 * q;
      rv[q] = (k < m) ? M.A[(int64_t)(r0 + k) * n + k0 + c] : 0.f;
    }
  };
  auto stash = [&](int kc) {
    if (kc >= i0 + SY_ROWS) {
      const int i = tid & 127, jb = tid >> 7;
#pragma unroll
      for (int q = 0; q < 16; ++q) sm.As[i][jb + 2 * q] = ra[q];
    } else {
      const int j = tid & 31, ib = tid >> 5;
#pragma unroll
      for (int q = 0; q < 16; ++q) sm.As[ib + 8 * q][j] = ra[q];
    }
    const int c = tid & 31, kb = tid >> 5;
#pragma unroll
    for (int q = 0; q < 4; ++q) sm.Vs[kb + 8 * q][c] = rv[q];
  };
  f32x16_t acc;
#pragma unroll
  for (int q = 0; q < 16; ++q) acc[q] = 0.f;
  fetch(0);
  for (int kc = 0; kc < m; kc += SB) {
    __syncthreads();
    stash(kc);
    __syncthreads();
    if (kc + SB < m) fetch(kc + SB);
#pragma unroll
    for (int s = 0; s < SB / 2; ++s)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.As[32 * wave + lr][2 * s + lh], sm.Vs[2 * s + lh][lr], acc,
                                                 0, 0, 0);
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 16; ++q) sm.As[32 * wave + 8 * (q >> 2) + 4 * lh + (q & 3)][lr] = acc[q];
  for (int q = tid; q < SY_ROWS * SB; q += SY_NT) {
    const int i = q / SB, c = q % SB;
    sm.Vb[i][c] = (i0 + i < m) ? M.A[(int64_t)(r0 + i0 + i) * n + k0 + c] : 0.f;
  }
  __syncthreads();
  {
    const int xi = tid >> 1, xc = (tid & 1) * 16;
    if (i0 + xi < m) {
#pragma unroll
      for (int u = 0; u < 16; ++u) M.X[(int64_t)(i0 + xi) * SB + xc + u] = sm.As[xi][xc + u];
    }
  }
  const int ya = tid >> 3, yc = (tid & 7) * 4;
  float yo[4] = {0.f, 0.f, 0.f, 0.f}, so[4] = {0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < SY_ROWS; ++i) {
    const float v = sm.Vb[i][ya];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      yo[u] = fmaf(v, sm.As[i][yc + u], yo[u]);
      so[u] = fmaf(v, sm.Vb[i][yc + u], so[u]);
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    M.Yp[((int64_t)blockIdx.x * SB + ya) * SB + yc + u] = yo[u];
    M.Sp[((int64_t)blockIdx.x * SB + ya) * SB + yc + u] = so[u];
  }
}

// ------------------------------------- stage 1: Z = X - (1/2) V (T^T Y) and the update panels
// From the block terms: S = V^T V and Y1 = V^T X1 summed in a fixed order, T by the
// recurrence T[0:c, c] = -tau_c T[0:c, 0:c] S[0:c, c] (one row per thread, in registers),
// Y = Y1 T, M = T^T Y; then per row X = X1 T and Z = X - (1/2) V M.  Writes
// P = [V; Z] and Q = [Z; V] (rows = panel columns, indexed by matrix row), so that the
// rank-2SB update A22 -= V Z^T + Z V^T is the single product P^T Q.
__global__ void __launch_bounds__(SY_NT) k_sb_zform(SbArgs a, int p, int mat0) {
  const int mat = mat0 + blockIdx.y, n = a.n;
  const SbView M = sview(a, mat);
  const int k0 = p * SB, r0 = k0 + SB, m = n - r0;
  const int i0 = blockIdx.x * SY_ROWS;
  if (m < 2 || i0 >= m) return;
  const int nblk = (m + SY_ROWS - 1) / SY_ROWS;
  __shared__ float Ys[SB][SB + 1], Ss[SB][SB + 1], Tw[SB][SB + 1], Ms[SB][SB + 1];
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid * 4 + u;
    float sy = 0.f, ss = 0.f;
    for (int b = 0; b < nblk; ++b) {
      sy += M.Yp[(int64_t)b * SB * SB + e];
      ss += M.Sp[(int64_t)b * SB * SB + e];
    }
    Ys[e / SB][e % SB] = sy;
    Ss[e / SB][e % SB] = ss;
  }
  __syncthreads();
  if (tid < SB) {
    // row i of T in registers (its entries left of the diagonal are zero, so every column
    // sums over all earlier entries)
    const int i = tid;
    float trow[SB];
#pragma unroll
    for (int c = 0; c < SB; ++c) {
      const float tc = M.tau[k0 + c];
      float acc = 0.f;
#pragma unroll
      for (int d = 0; d < c; ++d) acc = fmaf(trow[d], Ss[d][c], acc);
      trow[c] = (i < c) ? -tc * acc : (i == c ? tc : 0.f);
    }
#pragma unroll
    for (int c = 0; c < SB; ++c) Tw[i][c] = trow[c];
  }
  __syncthreads();
  // Y = Y1 T into Ms, then M = T^T Y into Ys
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid * 4 + u, ra = e / SB, c = e % SB;
    float acc = 0.f;
    for (int k = 0; k <= c; ++k) acc = fmaf(Ys[ra][k], Tw[k][c], acc);
    Ms[ra][c] = acc;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid * 4 + u, ra = e / SB, c = e % SB;
    float acc = 0.f;
    for (int k = 0; k <= ra; ++k) acc = fmaf(Tw[k][ra], Ms[k][c], acc);
    Ys[ra][c] = acc;
  }
  __syncthreads();
  const int i = tid >> 1, cb = (tid & 1) * 16;
  const int r = i0 + i;
  if (r >= m) return;
  float v[SB], x1[SB];
  const float *vp = M.A + (int64_t)(r0 + r) * n + k0;
#pragma unroll
  for (int c = 0; c < SB; ++c) { v[c] = vp[c]; x1[c] = M.X[(int64_t)r * SB + c]; }
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int c = cb + u;
    float sx = 0.f, sm_ = 0.f;
#pragma unroll
    for (int q = 0; q < SB; ++q) {
      sx = fmaf(x1[q], Tw[q][c], sx);
      sm_ = fmaf(v[q], Ys[q][c], sm_);
    }
    const float z = fmaf(-0.5f, sm_, sx);
    float vc = 0.f;
#pragma unroll
    for (int q = 0; q < SB; ++q) vc = (q == c) ? v[q] : vc;
    M.P[(int64_t)c * n + r0 + r] = vc;
    M.P[(int64_t)(SB + c) * n + r0 + r] = z;
    M.Q[(int64_t)c * n + r0 + r] = z;
    M.Q[(int64_t)(SB + c) * n + r0 + r] = vc;
  }
}

// ---------------------------------------------------------------- stage 2: bulge chase
// Band buffer AB[col][dd] = A[col + dd][col], dd < 2 SB.  Step k of sweep s works on the
// rows R = [r0, r1), r0 = s + 1 + k SB, r1 = min(r0 + SB, n):
//   L  = A[R, c0 : c0 + SB] (c0 = r0 - SB; at k = 0 only column s): reflector from its first
//        column, applied from the left;
//   D  = A[R, R]: both sides;
//   E  = A[r1 : r1 + SB, R]: from the right.  E is the next step's L and stays in registers.
// Lane (j, h) of a wavefront holds rows 16 h .. 16 h + 15 of column j of L and D, and
// columns 16 h .. 16 h + 15 of row j of E; v, w and E's transpose go through LDS.
// Reflector (s, k) is stored as [tau, v_1 .. v_31] (v_0 = 1) for the back-transform.
__global__ void __launch_bounds__(BG_WAVES * 64) k_sb_bulge(SbArgs a, int mat0) {
  const int mat = mat0 + blockIdx.x, n = a.n;
  const SbView M = sview(a, mat);
  const int km = steps_max(n);
  __shared__ float tb[BG_WAVES][SB][SB + 1];
  __shared__ float vb[BG_WAVES][SB], wb[BG_WAVES][SB];
  __shared__ int prog[BG_WAVES];
  __shared__ int abort_flag;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, lj = lane & 31, h = lane >> 5;
  if (tid < BG_WAVES) prog[tid] = -1;
  if (tid == 0) abort_flag = 0;
  __syncthreads();
  float *AB = M.AB;
  const int nsw = n - 2;
  // block loads of step k of a sweep: E (row layout) and D (diagonal-offset layout: lane lj
  // holds entry (c + lj, c) of columns c = 16 h ..; each column's lower part is one
  // contiguous band record), both coalesced
  auto load_blocks = [&](int r0, float (&D)[16], float (&E)[16]) {
    const int r1 = min(r0 + SB, n), ln = r1 - r0, ne = min(r1 + SB, n) - r1;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int c = 16 * h + q;
      E[q] = (lj < ne && c < ln) ? ldx(AB, (uint32_t)((r0 + c) * SBW + (ln + lj - c))) : 0.f;
      D[q] = (c + lj < ln) ? ldx(AB, (uint32_t)((r0 + c) * SBW + lj)) : 0.f;
    }
  };
  for (int s = wv; s < nsw; s += BG_WAVES) {
    float L[16], D[16], E[16], Dn[16], En[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) { L[q] = 0.f; Dn[q] = 0.f; En[q] = 0.f; }
    int r0 = s + 1;
    bool stop = false;
    for (int k = 0;; ++k) {
      const int r1 = min(r0 + SB, n), ln = r1 - r0;
      if (ln < 2) break;
      // Step k + 1's blocks are loaded during step k, so sweep s - 1 must have completed
      // step k + 3 (step k itself needs k + 2).
      if (s > 0) {
        const int need = (s - 1) * 1024 + k + 4;
        int spins = 0;
        if (a.spin_max == 0) stop = true;
        while (!stop) {
          const int v = __hip_atomic_load(&prog[(s - 1) % BG_WAVES], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
          if (v >= need) break;
          if (++spins > a.spin_max || __hip_atomic_load(&abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) {
            stop = true;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
        if (stop) break;
      }
      const int r2 = min(r1 + SB, n), ne = r2 - r1;
      if (k == 0) {
        load_blocks(r0, D, E);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int i = 16 * h + q;
          L[q] = (lj == 0 && i < ln) ? ldx(AB, (uint32_t)(s * SBW + 1 + i)) : 0.f;
        }
      } else {
#pragma unroll
        for (int q = 0; q < 16; ++q) { D[q] = Dn[q]; E[q] = En[q]; }
      }
      if (ne >= 2) load_blocks(r1, Dn, En);
      // reflector from L's first column (lanes 0 and 32)
      float part = 0.f;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int i = 16 * h + q;
        if (i >= 1) part = fmaf(L[q], L[q], part);
      }
      const float sigma = lane_value(part, 0) + lane_value(part, 32);
      const float alpha = lane_value(L[0], 0);
      float tau, beta, scal;
      house(alpha, sigma, tau, beta, scal);
      float *vbw = vb[wv], *wbw = wb[wv];
      if (lj == 0) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int i = 16 * h + q;
          vbw[i] = (i == 0) ? 1.f : (i < ln ? L[q] * scal : 0.f);
        }
      }
      wave_sync();
      const float vl = vbw[lj];
      if (h == 0) stx(M.V2, (uint32_t)((s * km + k) * SB + lj), (lj == 0) ? tau : vl);
      // L <- H L (columns 1 .. 31; column 0 becomes beta e_0)
      {
        float wc = 0.f;
#pragma unroll
        for (int q = 0; q < 16; ++q) wc = fmaf(vbw[16 * h + q], L[q], wc);
        wc = pair_sum(wc);
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int i = 16 * h + q;
          L[q] = (lj == 0) ? ((i == 0) ? beta : 0.f) : fmaf(-tau * vbw[i], wc, L[q]);
        }
        if (k == 0) {
          if (lj == 0) {
#pragma unroll
            for (int q = 0; q < 16; ++q) {
              const int i = 16 * h + q;
              if (i < ln) stx(AB, (uint32_t)(s * SBW + 1 + i), L[q]);
            }
          }
        }
      }
      float *tbw = &tb[wv][0][0];
      if (k > 0) {
        // stored by rows (through LDS), so that each store covers whole lines of a record
        const int c0 = r0 - SB;
#pragma unroll
        for (int q = 0; q < 16; ++q) tbw[(16 * h + q) * (SB + 1) + lj] = L[q];
        wave_sync();
        if (lj < ln) {
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int c = 16 * h + q;
            stx(AB, (uint32_t)((c0 + c) * SBW + (SB + lj - c)), tbw[lj * (SB + 1) + c]);
          }
        }
        wave_sync();
      }
      // D <- H D H: p = tau D v and w = p - (tau/2)(p^T v) v by columns (D mirrored through
      // LDS), then D -= v w^T + w v^T in the diagonal-offset layout
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int c = 16 * h + q;
        if (c + lj < SB) { tbw[(c + lj) * (SB + 1) + c] = D[q]; tbw[c * (SB + 1) + c + lj] = D[q]; }
      }
      wave_sync();
      float pj = 0.f;
#pragma unroll
      for (int q = 0; q < 16; ++q) pj = fmaf(tbw[(16 * h + q) * (SB + 1) + lj], vbw[16 * h + q], pj);
      pj = pair_sum(pj) * tau;
      const float pv = sum_lanes32(pj * vl);
      if (h == 0) wbw[lj] = fmaf(-0.5f * tau * pv, vl, pj);
      wave_sync();
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int c = 16 * h + q, i = c + lj;
        if (i < ln) {
          D[q] = fmaf(-vbw[i], wbw[c], fmaf(-wbw[i], vbw[c], D[q]));
          stx(AB, (uint32_t)((r0 + c) * SBW + lj), D[q]);
        }
      }
      // E <- E H (row layout: lane (i, h) holds columns 16 h ..)
      float yi = 0.f;
#pragma unroll
      for (int q = 0; q < 16; ++q) yi = fmaf(E[q], vbw[16 * h + q], yi);
      yi = pair_sum(yi);
#pragma unroll
      for (int q = 0; q < 16; ++q) E[q] = fmaf(-tau * yi, vbw[16 * h + q], E[q]);
      if (ne >= 2) {
        wave_sync();
#pragma unroll
        for (int q = 0; q < 16; ++q) tbw[lj * (SB + 1) + 16 * h + q] = E[q];
        wave_sync();
#pragma unroll
        for (int q = 0; q < 16; ++q) L[q] = tbw[(16 * h + q) * (SB + 1) + lj];
      } else if (ne == 1 && lj == 0) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int c = 16 * h + q;
          if (c < ln) stx(AB, (uint32_t)((r0 + c) * SBW + (ln - c)), E[q]);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      if (lane == 0) __hip_atomic_store(&prog[wv], s * 1024 + k + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (ne < 2) break;
      r0 = r1;
    }
    if (stop) {
      if (lane == 0) __hip_atomic_store(&abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      break;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    if (lane == 0) __hip_atomic_store(&prog[wv], s * 1024 + 1023, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __syncthreads();
  const bool bad = abort_flag != 0;
  for (int i = tid; i < n; i += BG_WAVES * 64) {
    M.d[i] = bad ? __builtin_nan("") : (double)AB[(int64_t)i * SBW];
    M.e[i] = (i + 1 < n) ? (double)AB[(int64_t)i * SBW + 1] : 0.0;
  }
}

// ------------------------------------------- eigenvectors: U = Q2 Z (stage-2 reflectors)
// The reflectors of the G = 32 sweeps s0 .. s0 + 31 at one step k act on the rows
// s0 + g + 1 + 32 k .. + 31 (g = 0 .. 31): a parallelogram block of 63 rows whose product
// H_{s0,k} H_{s0+1,k} ... H_{s0+31,k} is I - V T V^T (V 63 x 32, unit entry of column g in
// row g; T upper triangular).  Applying Q2 = product of all reflectors in the order made to
// the eigenvectors takes the groups from the last to the first and, within a group, the
// blocks in increasing k: a reflector of a later sweep overlaps one of an earlier sweep only
// at a step of the earlier one that is later (sweep s0 + g at step k meets sweep s0 + g' at
// step k + 1 only for g > g'), and reflectors that do not overlap commute.
constexpr int QG = SB;                 // sweeps per block
constexpr int QH = SB + QG - 1;        // rows per block
constexpr int QCW = 64;                // eigenvector columns per workgroup
constexpr int QRING = 128;             // rows of the sliding window (63 in use + 32 prefetched), a power of 2
constexpr int Q_NT = 256;

__host__ __device__ inline int64_t q_group_offset(int gi, int km) {
  return (int64_t)gi * km - (int64_t)gi * (gi - 1) / 2;    // blocks of groups 0 .. gi-1
}

JOLT_DEV bool refl_exists(int s, int k, int n) { return s <= n - 3 && k <= (n - 3 - s) / SB; }

// V T of every block (64 x 32, row-major, row 63 zero); one wavefront per block.  Column g
// of V holds the entries 1 .. 31 of reflector (s0 + g, k) below its unit entry;
// S = V^T V, then T[0:g, g] = -tau_g T[0:g, 0:g] S[0:g, g], T[g][g] = tau_g, then V T.
__global__ void __launch_bounds__(512) k_sb_qt(SbArgs a, int mat0) {
  const int mat = mat0 + blockIdx.y, n = a.n;
  const SbView M = sview(a, mat);
  const int km = steps_max(n);
  const int64_t total = (int64_t)km * (km + 1) / 2;
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane & 31;
  const int64_t blk = (int64_t)blockIdx.x * 8 + wv;
  __shared__ float vs[8][QG][SB + 1];
  __shared__ float ss[8][QG][QG + 1];
  __shared__ float ts[8][QG];
  __shared__ float tt[8][QG][QG + 1];
  if (blk >= total) return;
  int gi = 0;
  while (q_group_offset(gi + 1, km) <= blk) ++gi;
  const int k = (int)(blk - q_group_offset(gi, km)), s0 = gi * QG;
  const bool ex = refl_exists(s0 + g, k, n);
  const uint32_t vb = ex ? (uint32_t)(((s0 + g) * km + k) * SB) : 0u;
  if (lane < 32) {
    for (int i = 0; i < SB; ++i) {
      const float x = ldx(M.V2, vb + i);
      vs[wv][g][i] = (i == 0) ? 1.f : (ex ? x : 0.f);
      if (i == 0) ts[wv][g] = ex ? x : 0.f;
    }
  }
  wave_sync();
  // S = V^T V on the fp32 matrix cores (one 32 x 32 tile over the block's 64 rows): lane
  // (lr, lh) supplies V[j][lr] at j = 2 st + lh as both operands
  {
    const int lr = lane & 31, lh = lane >> 5;
    f32x16_t acc;
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[q] = 0.f;
#pragma unroll
    for (int st = 0; st < 32; ++st) {
      const int j = 2 * st + lh, dj = j - lr;
      const float x = vs[wv][lr][min(max(dj, 0), SB - 1)];
      const float vj = (dj == 0) ? 1.f : ((dj > 0 && dj < SB) ? x : 0.f);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(vj, vj, acc, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) ss[wv][8 * (q >> 2) + 4 * lh + (q & 3)][lr] = acc[q];
  }
  wave_sync();
  float t[QG];
#pragma unroll
  for (int c = 0; c < QG; ++c) t[c] = 0.f;
  const int i = g;
#pragma unroll
  for (int c = 0; c < QG; ++c) {
    const float tc = ts[wv][c];
    float acc = 0.f;
#pragma unroll
    for (int d = 0; d < c; ++d)
      if (d >= i) acc = fmaf(t[d], ss[wv][d][c], acc);
    t[c] = (i < c) ? -tc * acc : (i == c ? tc : 0.f);
  }
  if (lane < 32) {
#pragma unroll
    for (int c = 0; c < QG; ++c) tt[wv][i][c] = t[c];
  }
  wave_sync();
  {
    // V T on the fp32 matrix cores: two 32-row tiles, lane (lr, lh) supplies V[32 jt + lr][g]
    // and T[g][lr] at g = 2 st + lh; V[j][g] is 1 at j = g and entry j - g of column g below it
    const int lr = lane & 31, lh = lane >> 5;
    float *To = M.VTb + (q_group_offset(gi, km) + k) * (2 * QG * QG);
#pragma unroll
    for (int jt = 0; jt < 2; ++jt) {
      f32x16_t acc;
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[q] = 0.f;
      const int j = 32 * jt + lr;
#pragma unroll
      for (int st = 0; st < 16; ++st) {
        const int gg = 2 * st + lh, dj = j - gg;
        const float x = vs[wv][gg][min(max(dj, 0), SB - 1)];
        const float vj = (dj == 0) ? 1.f : ((dj > 0 && dj < SB) ? x : 0.f);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(vj, tt[wv][gg][lr], acc, 0, 0, 0);
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int row = 32 * jt + 8 * (q >> 2) + 4 * lh + (q & 3);
        To[row * QG + lr] = (row < QH) ? acc[q] : 0.f;
      }
    }
  }
}

// U (fp32) = Z (fp64) for the first k[mat] columns
__global__ void k_sb_z2u(int n, const double *Z, int ldz, const int32_t *kcnt, float *U, int64_t ldu,
                         int64_t u_stride, int kmax) {
  const int mat = blockIdx.y, kc = kcnt[mat];
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)n * kmax) return;
  const int r = (int)(q / kmax), c = (int)(q % kmax);
  if (c < kc) U[(int64_t)mat * u_stride + (int64_t)r * ldu + c] = (float)Z[((int64_t)mat * n + r) * ldz + c];
}

// Blocks applied to a slab of QCW columns held in a sliding window of QRING rows; while a
// block is applied the next block's 32 new rows, V entries and T are loaded into registers.
// Inside a group the barriers wait for LDS traffic only (rows that leave the window are not
// read again in the group, V and T are read-only), so those loads and the stores of the
// leaving rows stay in flight; a full barrier separates the groups.
struct QLds {
  float z[QRING][QCW + 1];
  float v[QH + 1][QG + 1];     // row QH stays zero (the products run over 64 rows)
  float vt[QH + 1][QG + 1];    // V T of the block (row QH zero)
  float w[QG][QCW + 1];
  float w2[QG][QCW + 1];
};

__global__ void __launch_bounds__(Q_NT) k_sb_qapply(SbArgs a, int mat0, const int32_t *kcnt, float *U,
                                                    int64_t ldu, int64_t u_stride) {
  const int mat = mat0 + blockIdx.y, n = a.n;
  const int c0 = blockIdx.x * QCW, kc = kcnt[mat];
  if (c0 >= kc) return;
  const SbView M = sview(a, mat);
  const int km = steps_max(n);
  __shared__ QLds sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, lr = lane & 31, lh = lane >> 5;
  const int ct = wave & 1, kh = wave >> 1;
  float *Um = U + (int64_t)mat * u_stride;
  const int ncol = min(QCW, kc - c0);
  for (int e = tid; e < QRING * (QCW + 1); e += Q_NT) (&sm.z[0][0])[e] = 0.f;
  for (int e = tid; e < QG + 1; e += Q_NT) sm.v[QH][e] = 0.f;
  // per-thread shares: rows (32 x QCW: 8 each), V (63 x 32: 8 each), V T (64 x 32: 8 each)
  float rz[8], rv[8], rt[8];
  auto fetch = [&](int s0, int k, int row0, int nrows) {
    // rows row0 .. row0 + nrows - 1 of the slab (nrows <= 32), V and T of block (s0, k)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + u * Q_NT, r = e / QCW, c = e % QCW;
      rz[u] = (r < nrows && row0 + r < n && c < ncol) ? Um[(int64_t)(row0 + r) * ldu + c0 + c] : 0.f;
    }
    const int gi = s0 / QG;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + u * Q_NT, j = e / QG, g = e % QG;
      float x = 0.f;
      if (j < QH) {
        const int i = j - g, row = s0 + 1 + k * SB + j;
        if (i == 0) x = 1.f;
        else if (i > 0 && i < SB && row < n && refl_exists(s0 + g, k, n))
          x = ldx(M.V2, (uint32_t)(((s0 + g) * km + k) * SB + i));
      }
      rv[u] = x;
    }
    const float *Tb = M.VTb + (q_group_offset(gi, km) + k) * (2 * QG * QG);
#pragma unroll
    for (int u = 0; u < 8; ++u) rt[u] = Tb[tid + u * Q_NT];
  };
  auto stash_vt = [&]() {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + u * Q_NT, j = e / QG, g = e % QG;
      if (j < QH) sm.v[j][g] = rv[u];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + u * Q_NT;
      sm.vt[e / QG][e % QG] = rt[u];
    }
  };
  auto stash_rows = [&](int row0) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + u * Q_NT, r = e / QCW, c = e % QCW;
      sm.z[(row0 + r) & (QRING - 1)][c] = rz[u];
    }
  };
  auto store_rows = [&](int row0, int nrows) {
    for (int e = tid; e < nrows * QCW; e += Q_NT) {
      const int r = e / QCW, c = e % QCW;
      if (row0 + r < n && c < ncol) Um[(int64_t)(row0 + r) * ldu + c0 + c] = sm.z[(row0 + r) & (QRING - 1)][c];
    }
  };
  const int ng = km;
  for (int gi = ng - 1; gi >= 0; --gi) {
    const int s0 = gi * QG, kv = km - gi;
    // window start: rows s0 + 1 .. s0 + 63 of block 0
    fetch(s0, 0, s0 + 1, 32);
    __syncthreads();
    stash_rows(s0 + 1);
    stash_vt();
    fetch(s0, 0, s0 + 33, 31);
    __syncthreads();
    stash_rows(s0 + 33);
    for (int k = 0; k < kv; ++k) {
      const int r0 = s0 + 1 + k * SB;
      if (k + 1 < kv) {
        // next block: its V and T, and the 32 rows that enter the window
        fetch(s0, k + 1, r0 + QH, 32);
      }
      lds_barrier();
      // The block's products on the fp32 matrix cores (32x32x2; lane (lr, lh) supplies row or
      // column lr at k = lh, acc[q] is element (8 (q / 4) + 4 lh + q % 4, lr) of the tile).
      // W = V^T Z: tile of columns 32 ct, the 64 block rows split between two wavefronts.
      {
        f32x16_t acc, acc1;
#pragma unroll
        for (int q = 0; q < 16; ++q) { acc[q] = 0.f; acc1[q] = 0.f; }
#pragma unroll
        for (int st = 0; st < 16; st += 2) {          // two independent chains
          const int j = 32 * kh + 2 * st + lh;
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.v[j][lr], sm.z[(r0 + j) & (QRING - 1)][32 * ct + lr], acc, 0, 0, 0);
          acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.v[j + 2][lr], sm.z[(r0 + j + 2) & (QRING - 1)][32 * ct + lr],
                                                      acc1, 0, 0, 0);
        }
        acc += acc1;
        if (kh == 1) {
#pragma unroll
          for (int q = 0; q < 16; ++q) sm.w2[8 * (q >> 2) + 4 * lh + (q & 3)][32 * ct + lr] = acc[q];
        }
        lds_barrier();
        if (kh == 0) {
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const int g = 8 * (q >> 2) + 4 * lh + (q & 3);
            sm.w[g][32 * ct + lr] = acc[q] + sm.w2[g][32 * ct + lr];
          }
        }
      }
      lds_barrier();
      // Z -= (V T) W: tile (rows 32 kh, columns 32 ct) per wavefront
      {
        f32x16_t acc, acc1;
#pragma unroll
        for (int q = 0; q < 16; ++q) { acc[q] = 0.f; acc1[q] = 0.f; }
#pragma unroll
        for (int st = 0; st < 16; st += 2) {
          const int g = 2 * st + lh;
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.vt[32 * kh + lr][g], sm.w[g][32 * ct + lr], acc, 0, 0, 0);
          acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.vt[32 * kh + lr][g + 2], sm.w[g + 2][32 * ct + lr], acc1, 0, 0,
                                                      0);
        }
        acc += acc1;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int j = 32 * kh + 8 * (q >> 2) + 4 * lh + (q & 3);
          if (j < QH) sm.z[(r0 + j) & (QRING - 1)][32 * ct + lr] -= acc[q];
        }
      }
      lds_barrier();
      if (k + 1 < kv) {
        // rows r0 .. r0 + 31 leave the window; the prefetched rows and the next V, T enter
        store_rows(r0, SB);
        lds_barrier();
        stash_rows(r0 + QH);
        stash_vt();
      } else {
        store_rows(r0, min(QH, n - r0));
      }
    }
    __syncthreads();
  }
}

}  // namespace

size_t sb_work_floats(int n_mat, int n) { return (size_t)n_mat * sb_per_mat(n); }

int sb_band() { return SB; }

size_t sb_table_entries(int n_mat, int n) { return (size_t)((n + SB - 1) / SB) * n_mat; }

void sb_tables(const EigBatch &b, float *work, GemmProblem *tab_host) {
  const int n = b.n, nm = b.n_mat, panels = (n + SB - 1) / SB;
  const int64_t ws = (int64_t)sb_per_mat(n);
  for (int p = 0; p < panels; ++p) {
    const int r0 = p * SB + SB, m = n - r0;
    for (int q = 0; q < nm; ++q) {
      GemmProblem g{};
      if (m >= 2) {
        const float *P = work + (int64_t)q * ws;
        const float *Q = P + (int64_t)2 * SB * n;
        g.A = GemmOperand{P + r0, n, 0, 0, 0, 1};    // A(m = r, k = p) = P[p][r0 + r]
        g.B = GemmOperand{Q + r0, n, 0, 0, 0, 1};
        g.C = b.A + (int64_t)q * b.mat_stride + (int64_t)r0 * n + r0;
        g.ldc = n;
        g.M = m; g.N = m; g.K = 2 * SB; g.alpha = -1.f; g.beta = 1.f;
        g.lower_only = 1;
      }
      tab_host[(size_t)p * nm + q] = g;
    }
  }
}

hipError_t launch_sb_reduce(const EigBatch &b, float *work, const GemmProblem *tab_dev, hipStream_t st, int m0,
                            int m1, int spin_max) {
  const int n = b.n;
  if (m1 < 0) m1 = b.n_mat;
  const int nm = m1 - m0;
  if (nm <= 0 || m0 < 0 || m1 > b.n_mat || n < 3 || n > SB_MAX_N) return hipErrorInvalidValue;
  SbArgs a{};
  a.A = b.A;
  a.mat_stride = b.mat_stride;
  a.n = n;
  a.work = work;
  a.work_stride = (int64_t)sb_per_mat(n);
  a.d = b.d;
  a.e = b.e;
  a.tau = b.tau;
  a.spin_max = spin_max < 0 ? 0 : spin_max;
  const int panels = (n + SB - 1) / SB;
  for (int p = 0; p < panels; ++p) {
    const int m = n - (p * SB + SB);
    hipLaunchKernelGGL(k_sb_panel, dim3(nm), dim3(PQ_NT), 0, st, a, p, m0);
    if (m < 2) continue;
    const int nblk = (m + SY_ROWS - 1) / SY_ROWS;
    hipLaunchKernelGGL(k_sb_symm, dim3(nblk, nm), dim3(SY_NT), 0, st, a, p, m0);
    hipLaunchKernelGGL(k_sb_zform, dim3(nblk, nm), dim3(SY_NT), 0, st, a, p, m0);
    hipError_t e = launch_update3(tab_dev + (size_t)p * b.n_mat + m0, nm, m, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_sb_bulge, dim3(nm), dim3(BG_WAVES * 64), 0, st, a, m0);
  return hipGetLastError();
}

hipError_t launch_sb_q2(const EigBatch &b, const float *work, const InvitWork &w, int kmax, float *U, int64_t ldu,
                        int64_t u_stride, hipStream_t st) {
  const int n = b.n, nm = b.n_mat;
  if (kmax <= 0) return hipSuccess;
  if (n < 3 || n > SB_MAX_N) return hipErrorInvalidValue;
  SbArgs a{};
  a.A = b.A;
  a.mat_stride = b.mat_stride;
  a.n = n;
  a.work = const_cast<float *>(work);
  a.work_stride = (int64_t)sb_per_mat(n);
  a.d = b.d;
  a.e = b.e;
  a.tau = b.tau;
  const int km = steps_max(n);
  const int64_t blocks = (int64_t)km * (km + 1) / 2;
  hipLaunchKernelGGL(k_sb_qt, dim3((unsigned)((blocks + 7) / 8), nm), dim3(512), 0, st, a, 0);
  hipLaunchKernelGGL(k_sb_z2u, dim3((unsigned)(((int64_t)n * kmax + 255) / 256), nm), dim3(256), 0, st, n, w.Z, w.ldz,
                     w.k, U, ldu, u_stride, kmax);
  hipLaunchKernelGGL(k_sb_qapply, dim3((kmax + QCW - 1) / QCW, nm), dim3(Q_NT), 0, st, a, 0, w.k, U, ldu, u_stride);
  return hipGetLastError();
}

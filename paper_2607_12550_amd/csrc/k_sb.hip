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
// may run step k once sweep s has completed step k + 2.  One workgroup per matrix, one
// wavefront per sweep in flight, the dependencies between wavefronts kept in LDS.
//
// Eigenvectors: z of the tridiagonal -> Q2 z (stage-2 reflectors, last sweep first; the
// reflectors of one sweep act on disjoint rows) -> Q1 (Q2 z) (stage-1 reflectors by the
// blocked WY back-transform, with the unit of reflector i at row i + SB).
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
constexpr int SPIN_MAX = 1 << 24; // bound of one dependency wait of the bulge chase

typedef float f32x16_t __attribute__((ext_vector_type(16)));

__host__ __device__ inline int steps_max(int n) { return n >= 3 ? (n - 3) / SB + 1 : 1; }

struct SbView {
  float *A, *P, *Q, *X, *Yp, *T, *AB, *V2;
  double *d, *e;
  float *tau;
};

__host__ __device__ inline size_t sb_per_mat(int n) {
  const size_t km = n >= 3 ? (size_t)((n - 3) / SB + 1) : 1;
  const size_t nblk = (size_t)((n + SY_ROWS - 1) / SY_ROWS);
  const size_t f = 4 * (size_t)SB * n + (size_t)n * SB + nblk * SB * SB + SB * SB + (size_t)n * SBW +
                   (size_t)n * km * SB + 64;
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
  v.T = v.Yp + (int64_t)nblk * SB * SB;
  v.AB = v.T + SB * SB;
  v.V2 = v.AB + (int64_t)n * SBW;
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
// which are the apply-dots for c > j + 1 and the entries (V^T v_{j+1})_c of the T
// recurrence T[0:j+1, j+1] = -tau T[0:j+1, 0:j+1] (V^T v_{j+1}) for c < j + 1.
// Eight lanes share a row (four columns each), so a wavefront reads eight whole rows per
// load; the entries x_r[j] and x_r[j+1] are exchanged within the eight lanes.
// Writes: the diagonal block and R into the band buffer (zeros past the band), V explicit
// into the panel (unit at row j, zeros above, and zeros in the rows [blk + SB, r0) of the
// panel's columns, blk = k0 rounded down to the back-transform's block of 128 reflectors),
// tau and T.
JOLT_DEV float pick4(const float (&x)[4], int u) {
  return u == 0 ? x[0] : (u == 1 ? x[1] : (u == 2 ? x[2] : x[3]));
}

__global__ void __launch_bounds__(PQ_NT) k_sb_panel(SbArgs a, int p, int mat0) {
  const int mat = mat0 + blockIdx.x, n = a.n;
  const SbView M = sview(a, mat);
  const int k0 = p * SB, r0 = k0 + SB, w = min(SB, n - k0), m = n - r0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ float red[PQ_NT / 64][SB];
  __shared__ float rowj[SB], dv[SB], Ts[SB][SB + 1];
  __shared__ float sc[4];
  for (int q = tid; q < SB * SBW; q += PQ_NT) {
    const int j = q / SBW, dd = q - j * SBW, row = k0 + j + dd;
    if (j >= w || row >= n) continue;
    if (dd < SB - j) M.AB[(int64_t)(k0 + j) * SBW + dd] = M.A[(int64_t)row * n + k0 + j];
    else if (dd > SB) M.AB[(int64_t)(k0 + j) * SBW + dd] = 0.f;
  }
  for (int q = tid; q < SB * (SB + 1); q += PQ_NT) (&Ts[0][0])[q] = 0.f;
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
    for (int r = rfirst; r < m; r += RSTEP) {
      if (r < j) continue;                       // the eight lanes of a row agree
      float *rp = M.A + (int64_t)(r0 + r) * n + k0 + c4;
      float x[4];
      if (vec) {
        const jf4 v = gload_f4(rp);
        x[0] = v[0]; x[1] = v[1]; x[2] = v[2]; x[3] = v[3];
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) x[u] = rp[u];
      }
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
      wave_sync();
      if (lane < nj) {
        float acc = 0.f;
        for (int c = lane; c < nj; ++c) acc = fmaf(Ts[lane][c], dv[c], acc);
        Ts[lane][nj] = -t * acc;
      }
      if (lane == nj) Ts[nj][nj] = t;
    }
    __syncthreads();
  }
  if (tid >= jmax && tid < SB) M.tau[k0 + tid] = 0.f;
  __syncthreads();
  for (int q = tid; q < SB * SB; q += PQ_NT) M.T[q] = Ts[q / SB][q % SB];
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
// each).  Epilogue: X = X1 T (T upper triangular), and this block's term of Y = V^T X.
struct SyLds {
  float As[SY_ROWS][SB + 1];
  float Vs[SB][SB + 1];
  float Ts[SB][SB + 1];
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
  for (int q = tid; q < SB * SB; q += SY_NT) sm.Ts[q / SB][q % SB] = M.T[q];
  for (int q = tid; q < SY_ROWS * SB; q += SY_NT) {
    const int i = q / SB, c = q % SB;
    sm.Vb[i][c] = (i0 + i < m) ? M.A[(int64_t)(r0 + i0 + i) * n + k0 + c] : 0.f;
  }
  __syncthreads();
  const int xi = tid >> 1, xc = (tid & 1) * 16;
  float xo[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int c = xc + u;
    float s = 0.f;
    for (int k = 0; k <= c; ++k) s = fmaf(sm.As[xi][k], sm.Ts[k][c], s);
    xo[u] = s;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 16; ++u) sm.As[xi][xc + u] = xo[u];
  if (i0 + xi < m) {
#pragma unroll
    for (int u = 0; u < 16; ++u) M.X[(int64_t)(i0 + xi) * SB + xc + u] = xo[u];
  }
  __syncthreads();
  const int ya = tid >> 3, yc = (tid & 7) * 4;
  float yo[4] = {0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < SY_ROWS; ++i) {
    const float v = sm.Vb[i][ya];
#pragma unroll
    for (int u = 0; u < 4; ++u) yo[u] = fmaf(v, sm.As[i][yc + u], yo[u]);
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) M.Yp[((int64_t)blockIdx.x * SB + ya) * SB + yc + u] = yo[u];
}

// ------------------------------------- stage 1: Z = X - (1/2) V (T^T Y) and the update panels
// P = [V; Z] and Q = [Z; V] (rows = panel columns, indexed by matrix row), so that the
// rank-2SB update A22 -= V Z^T + Z V^T is the single product P^T Q.
__global__ void __launch_bounds__(SY_NT) k_sb_zform(SbArgs a, int p, int mat0) {
  const int mat = mat0 + blockIdx.y, n = a.n;
  const SbView M = sview(a, mat);
  const int k0 = p * SB, r0 = k0 + SB, m = n - r0;
  const int i0 = blockIdx.x * SY_ROWS;
  if (m < 2 || i0 >= m) return;
  const int nblk = (m + SY_ROWS - 1) / SY_ROWS;
  __shared__ float Ys[SB][SB + 1], Ts[SB][SB + 1], Ms[SB][SB + 1];
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid * 4 + u;
    float s = 0.f;
    for (int b = 0; b < nblk; ++b) s += M.Yp[(int64_t)b * SB * SB + e];
    Ys[e / SB][e % SB] = s;
    Ts[e / SB][e % SB] = M.T[e];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid * 4 + u, ra = e / SB, c = e % SB;
    float s = 0.f;
    for (int k = 0; k <= ra; ++k) s = fmaf(Ts[k][ra], Ys[k][c], s);
    Ms[ra][c] = s;
  }
  __syncthreads();
  const int i = tid >> 1, cb = (tid & 1) * 16;
  const int r = i0 + i;
  if (r >= m) return;
  float v[SB];
  const float *vp = M.A + (int64_t)(r0 + r) * n + k0;
#pragma unroll
  for (int c = 0; c < SB; ++c) v[c] = vp[c];
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int c = cb + u;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < SB; ++q) s = fmaf(v[q], Ms[q][c], s);
    const float z = fmaf(-0.5f, s, M.X[(int64_t)r * SB + c]);
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
        for (;;) {
          const int v = __hip_atomic_load(&prog[(s - 1) % BG_WAVES], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
          if (v >= need) break;
          if (++spins > SPIN_MAX || __hip_atomic_load(&abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) {
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
      const float sigma = __shfl(part, 0, 64) + __shfl(part, 32, 64);
      const float alpha = __shfl(L[0], 0, 64);
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
        wc += shfl_xor(wc, 32);
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
      pj += shfl_xor(pj, 32);
      pj *= tau;
      float pv = (h == 0) ? pj * vl : 0.f;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) pv += shfl_xor(pv, o);
      pv = __shfl(pv, 0, 64);
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
      yi += shfl_xor(yi, 32);
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
// One workgroup per matrix and slab of C columns of Z, the slab resident in LDS (fp32);
// sweeps from the last to the first, the reflectors of one sweep (disjoint row blocks)
// spread over the wavefronts (wavefront w takes k = w, w + 8, ...), one barrier per sweep.
// A wavefront's reflectors of the next sweep are loaded while the current sweep is applied
// (two register sets, one entry per lane and reflector).  Lane layout per reflector: column lane % C, rows
// lane / C + (64 / C) q of its 32 (so that a wavefront's slab accesses spread over the LDS banks).
constexpr int Q2_NT = 512;
constexpr int Q2_WAVES = Q2_NT / 64;

// A wavefront's reflectors of one sweep: lane l holds entry l % 32 of each ([tau, v_1 ..]);
// one load per reflector, the entries a lane needs come by lane exchange.
template <int TMAX>
struct Q2Set {
  float e[TMAX];
};

template <int TMAX>
JOLT_DEV void q2_fetch(Q2Set<TMAX> &f, const float *V2, int s, int km, int n, int wv, int lane) {
  const int ks = (n - 3 - s) / SB + 1;
#pragma unroll
  for (int t = 0; t < TMAX; ++t) {
    const int k = wv + t * Q2_WAVES;
    const bool live = s >= 0 && k < ks;
    // unconditional load (a valid entry when not live; such entries are never applied), so
    // that the loads stay in flight across the sweep's barrier until their first use
    f.e[t] = ldx(V2, live ? (uint32_t)((s * km + k) * SB + (lane & 31)) : 0u);
  }
}

template <int C, int TMAX>
__global__ void __launch_bounds__(Q2_NT) k_sb_q2(SbArgs a, int mat0, const double *Z, int ldz, const int32_t *kcnt,
                                                 float *U, int64_t ldu, int64_t u_stride) {
  constexpr int RPL = C / 2;                 // rows per lane
  const int mat = mat0 + blockIdx.y, n = a.n;
  const int c0 = blockIdx.x * C;
  const int kc = kcnt[mat];
  if (c0 >= kc) return;
  const SbView M = sview(a, mat);
  const int km = steps_max(n);
  extern __shared__ float us[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const double *Zm = Z + (int64_t)mat * n * ldz;
  for (int q = tid; q < n * C; q += Q2_NT) {
    const int r = q / C, c = q % C;
    us[q] = (c0 + c < kc) ? (float)Zm[(int64_t)r * ldz + c0 + c] : 0.f;
  }
  const int col = lane % C, rg = lane / C;
  // the reflectors of one sweep touch disjoint rows: G at a time are read, reduced and
  // written as a group, so that their LDS traffic and shuffles overlap
  auto apply = [&](const Q2Set<TMAX> &g, int s) {
    constexpr int G = C == 8 ? 8 : 4;
    const int ks = (n - 3 - s) / SB + 1;
#pragma unroll
    for (int t0 = 0; t0 < TMAX; t0 += G) {
      if (wv + t0 * Q2_WAVES >= ks) break;
      float u[G][RPL], vv[G][RPL], dot[G], tv[G];
      int base[G], ln[G];
#pragma unroll
      for (int e = 0; e < G; ++e) {
        const int k = wv + (t0 + e) * Q2_WAVES;
        const int r0 = s + 1 + k * SB;
        ln[e] = (k < ks) ? min(SB, n - r0) : 0;
        base[e] = r0 * C + col;
        dot[e] = 0.f;
#pragma unroll
        for (int q = 0; q < RPL; ++q) {
          const int i = rg + (64 / C) * q;
          // every lane takes part in the exchange (its source lanes must be active)
          const float vi = __shfl(g.e[t0 + e], i, 64);
          vv[e][q] = (i == 0) ? 1.f : vi;
          u[e][q] = (i < ln[e]) ? us[base[e] + i * C] : 0.f;
          dot[e] = fmaf(vv[e][q], u[e][q], dot[e]);
        }
        tv[e] = __shfl(g.e[t0 + e], 0, 64);
      }
#pragma unroll
      for (int o = C; o < 64; o <<= 1)
#pragma unroll
        for (int e = 0; e < G; ++e) dot[e] += shfl_xor(dot[e], o);
#pragma unroll
      for (int e = 0; e < G; ++e) {
        const float td = tv[e] * dot[e];
#pragma unroll
        for (int q = 0; q < RPL; ++q) {
          const int i = rg + (64 / C) * q;
          if (i < ln[e]) us[base[e] + i * C] = fmaf(-td, vv[e][q], u[e][q]);
        }
      }
    }
  };
  Q2Set<TMAX> fa, fb;
  q2_fetch<TMAX>(fa, M.V2, n - 3, km, n, wv, lane);
  __syncthreads();
  for (int s = n - 3; s >= 0; s -= 2) {
    q2_fetch<TMAX>(fb, M.V2, s - 1, km, n, wv, lane);
    apply(fa, s);
    lds_barrier();
    if (s == 0) break;
    q2_fetch<TMAX>(fa, M.V2, s - 2, km, n, wv, lane);
    apply(fb, s - 1);
    lds_barrier();
  }
  __syncthreads();
  float *Um = U + (int64_t)mat * u_stride;
  for (int q = tid; q < n * C; q += Q2_NT) {
    const int r = q / C, c = q % C;
    if (c0 + c < kc) Um[(int64_t)r * ldu + c0 + c] = us[q];
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
                            int m1) {
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
  if (n <= 4096) {
    const size_t shm = (size_t)n * 8 * sizeof(float);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_sb_q2<8, 16>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_sb_q2<8, 16>), dim3((kmax + 7) / 8, nm), dim3(Q2_NT), shm, st, a, 0, w.Z, w.ldz, w.k, U,
                       ldu, u_stride);
  } else {
    const size_t shm = (size_t)n * 4 * sizeof(float);
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_sb_q2<4, 32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_sb_q2<4, 32>), dim3((kmax + 3) / 4, nm), dim3(Q2_NT), shm, st, a, 0, w.Z, w.ldz, w.k, U,
                       ldu, u_stride);
  }
  return hipGetLastError();
}

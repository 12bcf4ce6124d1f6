// Feature-mode Gram matrix F = sum_s X_s^T X_s (d x d) and energy E = ||X||_F^2
// (section 4: the feature-mode spectrum is kept exact in both variants, section 5).
//
// The row set {(s, r)} of a cell is cut into `chunks_per_cell` contiguous runs;
// one 256-thread workgroup reduces a run into a d x d fp32 partial (16 x 16 thread
// grid, each thread an (d/16) x (d/16) block) plus an fp64 partial energy, staging
// 32 rows at a time in LDS.  A second kernel adds the partials of a cell in a fixed
// order in fp64, so results are deterministic.  The same kernel serves the Gram of
// the projected tensor Y (rows (s, r) of Y_s) during ST-HOSVD.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int ROWS = 32;

template <int D, typename TX>
__global__ void __launch_bounds__(256) k_fgram(FGramArgs a) {
  constexpr int B = D / 16;
  __shared__ float xs[ROWS][D + 4];
  const int cell = blockIdx.y, chunk = blockIdx.x;
  const int tid = threadIdx.x, ti = tid / 16, tj = tid % 16;
  const int rps = a.cells[cell].rows_per_seg;
  const int64_t total = (int64_t)a.nseg * rps;
  const int64_t r0 = total * chunk / a.chunks_per_cell, r1 = total * (chunk + 1) / a.chunks_per_cell;
  const TX *base = reinterpret_cast<const TX *>(a.cells[cell].base);
  float acc[B][B];
#pragma unroll
  for (int i = 0; i < B; ++i)
#pragma unroll
    for (int j = 0; j < B; ++j) acc[i][j] = 0.f;
  double e = 0.0;
  int bad = 0;
  constexpr int LPR = D / 8;               // threads per row when loading
  constexpr int RPP = 256 / LPR;           // rows per load pass
  for (int64_t rb = r0; rb < r1; rb += ROWS) {
    __syncthreads();
    for (int rr = tid / LPR; rr < ROWS; rr += RPP) {
      const int64_t row = rb + rr;
      const int c8 = (tid % LPR) * 8;
      float v[8];
      if (row < r1) {
        const int s = (int)(row / rps), r = (int)(row % rps);
        const TX *p = base + (int64_t)(s / a.seg_heads) * a.seg_hi +
                      (int64_t)(s % a.seg_heads) * a.seg_lo + (int64_t)r * a.row_stride + c8;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if constexpr (sizeof(TX) == 2) v[i] = bf16_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
          else v[i] = reinterpret_cast<const float *>(p)[i];
          e += (double)v[i] * (double)v[i];
          bad |= !isfinite(v[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) xs[rr][c8 + i] = v[i];
    }
    __syncthreads();
#pragma unroll 4
    for (int rr = 0; rr < ROWS; ++rr) {
      float xa[B], xb[B];
#pragma unroll
      for (int i = 0; i < B; ++i) { xa[i] = xs[rr][ti * B + i]; xb[i] = xs[rr][tj * B + i]; }
#pragma unroll
      for (int i = 0; i < B; ++i)
#pragma unroll
        for (int j = 0; j < B; ++j) acc[i][j] = fmaf(xa[i], xb[j], acc[i][j]);
    }
  }
  float *pf = a.partial_F + ((int64_t)cell * a.chunks_per_cell + chunk) * D * D;
#pragma unroll
  for (int i = 0; i < B; ++i)
#pragma unroll
    for (int j = 0; j < B; ++j) pf[(ti * B + i) * D + tj * B + j] = acc[i][j];
  __shared__ double es[4];
  __shared__ int bs[4];
  double ew = wave_sum(e);
  int bw = __any(bad) ? 1 : 0;
  if ((tid & 63) == 0) { es[tid >> 6] = ew; bs[tid >> 6] = bw; }
  __syncthreads();
  if (tid == 0) {
    a.partial_E[(int64_t)cell * a.chunks_per_cell + chunk] = es[0] + es[1] + es[2] + es[3];
    if (bs[0] | bs[1] | bs[2] | bs[3]) atomicOr(&a.nonfinite[cell], 1);
  }
}

__global__ void k_fgram_reduce(FGramArgs a, int D, float *F_out, double *E_out) {
  const int cell = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t dd = (int64_t)D * D;
  if (i < dd) {
    double s = 0.0;
    const float *p = a.partial_F + (int64_t)cell * a.chunks_per_cell * dd + i;
    for (int c = 0; c < a.chunks_per_cell; ++c) s += (double)p[c * dd];
    F_out[cell * dd + i] = (float)s;
  }
  if (i == 0) {
    double s = 0.0;
    for (int c = 0; c < a.chunks_per_cell; ++c) s += a.partial_E[(int64_t)cell * a.chunks_per_cell + c];
    E_out[cell] = s;
  }
}

}  // namespace

hipError_t launch_feature_gram(const FGramArgs &a, int d, int dtype, hipStream_t st) {
  dim3 grid(a.chunks_per_cell, a.n_cells);
#define L_(D_) \
  if (d == D_) { \
    if (dtype == 1) hipLaunchKernelGGL((k_fgram<D_, uint16_t>), grid, dim3(256), 0, st, a); \
    else hipLaunchKernelGGL((k_fgram<D_, float>), grid, dim3(256), 0, st, a); \
    return hipGetLastError(); }
  L_(32) L_(64) L_(128)
#undef L_
  return hipErrorInvalidValue;
}

hipError_t launch_feature_gram_reduce(const FGramArgs &a, int d, float *F_out, double *E_out,
                                      hipStream_t st) {
  dim3 grid((d * d + 255) / 256, a.n_cells);
  hipLaunchKernelGGL(k_fgram_reduce, grid, dim3(256), 0, st, a, d, F_out, E_out);
  return hipGetLastError();
}

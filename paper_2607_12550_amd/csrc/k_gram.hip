// Feature-mode Gram matrix F = sum_s X_s^T X_s (d x d) and energy E = ||X||_F^2
// (section 4: the feature-mode spectrum is kept exact in both variants, section 5), and
// the slice-mode Gram of the three-mode diagnostics (section 3, appendix A).
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

// bf16 cells with d = 128: the same partials on the bf16 matrix cores.  Each stage takes 64
// rows; thread (row group g = tid / 16, feature block f = tid % 16) loads rows 4g .. 4g+3,
// features 8f .. 8f+7 (16-byte loads), adds their squares to the fp64 energy, and stores them
// transposed into LDS as xt[feature][row] (four rows of one feature per 8-byte store; the
// features are visited in a lane-dependent order so the stores spread over the banks).
// Wave (wm, wn) then accumulates the 64 x 64 block (wm, wn) of F with 2 x 2
// v_mfma_f32_32x32x16_bf16 per 16 rows.  The products of bf16 values are exact in fp32, so
// only the fp32 accumulation order differs from the vector kernel.
constexpr int FR = 64, FLD = FR + 8;

__global__ void __launch_bounds__(256) k_fgram_mfma128(FGramArgs a) {
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
  typedef float f32x16_t __attribute__((ext_vector_type(16)));
  constexpr int D = 128;
  __shared__ __attribute__((aligned(16))) uint16_t xt[D * FLD];
  const int cell = blockIdx.y, chunk = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, lr = lane & 31, lh = lane >> 5;
  const int fb = tid & 15, rg = tid >> 4;
  const int rps = a.cells[cell].rows_per_seg;
  const int64_t total = (int64_t)a.nseg * rps;
  const int64_t r0 = total * chunk / a.chunks_per_cell, r1 = total * (chunk + 1) / a.chunks_per_cell;
  const uint16_t *base = reinterpret_cast<const uint16_t *>(a.cells[cell].base);
  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  double e = 0.0;
  int bad = 0;
  for (int64_t rb = r0; rb < r1; rb += FR) {
    const int64_t row0 = rb + rg * 4;
    int s = 0, r = 0;
    if (row0 < r1) { s = (int)(row0 / rps); r = (int)(row0 - (int64_t)s * rps); }
    ju4 u[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (row0 + k < r1) {
        const uint16_t *p = base + (int64_t)(s / a.seg_heads) * a.seg_hi + (int64_t)(s % a.seg_heads) * a.seg_lo +
                            (int64_t)r * a.row_stride + fb * 8;
        u[k] = gload_u4(p);
      } else {
        u[k] = ju4{0u, 0u, 0u, 0u};
      }
      if (++r == rps) { r = 0; ++s; }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float lo = bf16_to_f32((bf16_t)(u[k][w] & 0xffffu)), hi = bf16_to_f32((bf16_t)(u[k][w] >> 16));
        e += (double)lo * (double)lo;
        e += (double)hi * (double)hi;
        bad |= (int)!isfinite(lo) | (int)!isfinite(hi);
      }
    __syncthreads();                      // the previous stage's fragments have been read
#pragma unroll
    for (int ii = 0; ii < 8; ++ii) {
      const int i = (ii + fb) & 7, w = i >> 1, sh = 16 * (i & 1);
      const uint32_t h0 = (u[0][w] >> sh) & 0xffffu, h1 = (u[1][w] >> sh) & 0xffffu;
      const uint32_t h2 = (u[2][w] >> sh) & 0xffffu, h3 = (u[3][w] >> sh) & 0xffffu;
      *reinterpret_cast<uint2 *>(xt + (fb * 8 + i) * FLD + rg * 4) = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < FR / 16; ++ks) {
      const int ko = ks * 16 + 8 * lh;
      bf16x8_t fa[2], fbv[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        fa[t] = *reinterpret_cast<const bf16x8_t *>(xt + (wm * 64 + t * 32 + lr) * FLD + ko);
        fbv[t] = *reinterpret_cast<const bf16x8_t *>(xt + (wn * 64 + t * 32 + lr) * FLD + ko);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fbv[j], acc[i][j], 0, 0, 0);
    }
  }
  // acc[i][j][q] is F at row wm*64 + i*32 + 8*(q/4) + 4*lh + q%4, column wn*64 + j*32 + lr
  float *pf = a.partial_F + ((int64_t)cell * a.chunks_per_cell + chunk) * D * D;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q)
        pf[(wm * 64 + i * 32 + 8 * (q >> 2) + 4 * lh + (q & 3)) * D + wn * 64 + j * 32 + lr] = acc[i][j][q];
  __shared__ double es[4];
  __shared__ int bs[4];
  double ew = wave_sum(e);
  int bw = __any(bad) ? 1 : 0;
  if (lane == 0) { es[wave] = ew; bs[wave] = bw; }
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

// Slice-mode Gram: thread (a, b) of the 16 x 16 grid owns entry (I*16 + a, J*16 + b) of the
// tile pair (I >= J).  TOK tokens of the 32 slices' feature rows are staged in LDS as fp32
// per step; each token's d-term dot product is summed in fp32 and added to an fp64
// accumulator.
template <int D, typename TX>
__global__ void __launch_bounds__(256) k_slice_gram(SliceGramArgs a) {
  constexpr int TOK = 2, LD = D + 4;
  __shared__ __attribute__((aligned(16))) float xs[2][TOK][16][LD];
  const int cell = blockIdx.z, chunk = blockIdx.y;
  int I = 0, J = 0;
  {
    int t = blockIdx.x, i = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
    while ((i + 1) * (i + 2) / 2 <= t) ++i;
    while (i * (i + 1) / 2 > t) --i;
    I = i; J = t - i * (i + 1) / 2;
  }
  const int tid = threadIdx.x, ta = tid / 16, tb = tid % 16;
  const int t0 = (int)((int64_t)a.T * chunk / a.chunks), t1 = (int)((int64_t)a.T * (chunk + 1) / a.chunks);
  const TX *base = reinterpret_cast<const TX *>(a.cells[cell].base);
  double acc = 0.0;
  constexpr int LPR = D / 8;                       // threads per feature row when loading
  for (int tt = t0; tt < t1; tt += TOK) {
    __syncthreads();
    // 2 tiles x TOK tokens x 16 slices rows of D features, 8 features per thread and pass
    for (int q = tid; q < 2 * TOK * 16 * LPR; q += 256) {
      const int c8 = (q % LPR) * 8, row = q / LPR;
      const int sl = row % 16, k = (row / 16) % TOK, which = row / (16 * TOK);
      const int s = (which ? J : I) * 16 + sl, t = tt + k;
      float v[8];
      if (s < a.m && t < t1) {
        const TX *p = base + (int64_t)(s / a.heads) * a.s_layer + (int64_t)(s % a.heads) * a.s_head +
                      (int64_t)t * a.s_tok + c8;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if constexpr (sizeof(TX) == 2) v[i] = bf16_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
          else v[i] = reinterpret_cast<const float *>(p)[i];
        }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) xs[which][k][sl][c8 + i] = v[i];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TOK; ++k) {
      float sum = 0.f;
#pragma unroll 8
      for (int f = 0; f < D; f += 4) {
        const float4 x = *reinterpret_cast<const float4 *>(&xs[0][k][ta][f]);
        const float4 y = *reinterpret_cast<const float4 *>(&xs[1][k][tb][f]);
        sum = fmaf(x.x, y.x, sum); sum = fmaf(x.y, y.y, sum);
        sum = fmaf(x.z, y.z, sum); sum = fmaf(x.w, y.w, sum);
      }
      acc += (double)sum;
    }
  }
  const int si = I * 16 + ta, sj = J * 16 + tb;
  if (si < a.m && sj < a.m)
    a.partial[(((int64_t)cell * a.chunks + chunk) * a.m + si) * a.m + sj] = acc;
}

// S[cell][i][j] = sum over chunks of the partial at (max(i, j), min(i, j)) (tile-pair
// blocks cover rows in the higher tile; both orders are written inside a diagonal tile)
__global__ void k_slice_gram_reduce(SliceGramArgs a, float *S_out) {
  const int cell = blockIdx.y;
  const int64_t mm = (int64_t)a.m * a.m;
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= mm) return;
  const int i = (int)(q / a.m), j = (int)(q % a.m);
  const int hi = (i / 16 > j / 16) || (i / 16 == j / 16) ? i : j, lo = hi == i ? j : i;
  double s = 0.0;
  const double *p = a.partial + (int64_t)cell * a.chunks * mm + (int64_t)hi * a.m + lo;
  for (int c = 0; c < a.chunks; ++c) s += p[c * mm];
  S_out[cell * mm + q] = (float)s;
}

// One thread per matrix element of a cell; the n_k loads of a run are independent of
// the running sum, so eight are issued ahead of their adds.
__global__ void __launch_bounds__(256) k_prefix_sum_mats(float *M, int n_k, int64_t elems) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= elems) return;
  float *p = M + (int64_t)blockIdx.y * n_k * elems + e;
  double acc = 0.0;
  int k = 0;
  for (; k + 8 <= n_k; k += 8) {
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = p[(int64_t)(k + j) * elems];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      acc += (double)v[j];
      p[(int64_t)(k + j) * elems] = (float)acc;
    }
  }
  for (; k < n_k; ++k) {
    acc += (double)p[(int64_t)k * elems];
    p[(int64_t)k * elems] = (float)acc;
  }
}

}  // namespace

hipError_t launch_prefix_sum_mats(float *M, int n_cells, int n_k, int64_t elems, hipStream_t st) {
  if (n_cells < 1 || n_k < 1 || elems < 1) return hipErrorInvalidValue;
  dim3 grid((unsigned)((elems + 255) / 256), n_cells);
  hipLaunchKernelGGL(k_prefix_sum_mats, grid, dim3(256), 0, st, M, n_k, elems);
  return hipGetLastError();
}

hipError_t launch_slice_gram(const SliceGramArgs &a, int d, int dtype, hipStream_t st) {
  dim3 grid(a.tiles * (a.tiles + 1) / 2, a.chunks, a.n_cells);
#define L_(D_) \
  if (d == D_) { \
    if (dtype == 1) hipLaunchKernelGGL((k_slice_gram<D_, uint16_t>), grid, dim3(256), 0, st, a); \
    else hipLaunchKernelGGL((k_slice_gram<D_, float>), grid, dim3(256), 0, st, a); \
    return hipGetLastError(); }
  L_(32) L_(64) L_(128)
#undef L_
  return hipErrorInvalidValue;
}

hipError_t launch_slice_gram_reduce(const SliceGramArgs &a, float *S_out, hipStream_t st) {
  const int64_t mm = (int64_t)a.m * a.m;
  dim3 grid((unsigned)((mm + 255) / 256), a.n_cells);
  hipLaunchKernelGGL(k_slice_gram_reduce, grid, dim3(256), 0, st, a, S_out);
  return hipGetLastError();
}

hipError_t launch_feature_gram(const FGramArgs &a, int d, int dtype, hipStream_t st) {
  dim3 grid(a.chunks_per_cell, a.n_cells);
  if (d == 128 && dtype == 1 && a.vec16) {
    hipLaunchKernelGGL(k_fgram_mfma128, grid, dim3(256), 0, st, a);
    return hipGetLastError();
  }
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

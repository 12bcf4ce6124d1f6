// FlashJoLT randomized token-mode SVD helpers (section 5): the seeded Gaussian test
// matrix and the CholeskyQR2 orthonormalisation used by the range finder.
//
// Sketch: Omega[c][j] = bf16(sqrt(-2 ln u0) cos(2 pi u1)) with (u0, u1) from Philox4x32-10 at
// counter (c, j, 0, 2) and key = seed; Box-Muller runs in fp64 and is rounded once to bf16.
// CholeskyQR2: G = Y^T Y accumulated in fp64 (split over row chunks, partials summed in a
// fixed order), G = L L^T, Q = Y L^-T, applied twice.  fp64 keeps the Gram usable for
// condition numbers up to ~1e7, which a power-iterated sketch of a decaying spectrum
// reaches.  Directions whose Cholesky pivot falls below 1e-14 of the largest diagonal
// are treated as numerically absent (pivot clamped), so rank-deficient sketches stay finite.
#include "common.h"
#include "kernels.h"

namespace {

__global__ void k_sketch(SketchArgs a) {
  const int cell = blockIdx.y;
  const uint64_t sd = a.seeds[cell];
  const int64_t total = (int64_t)a.N * a.ld;
  uint16_t *om = a.out + (int64_t)cell * a.cell_stride;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(q / a.ld), j = (int)(q % a.ld);
    uint16_t v = 0;
    if (j < a.l) {
      u32x4 w = philox4x32_10(u32x4{(uint32_t)c, (uint32_t)j, 0u, (uint32_t)STREAM_SKETCH},
                              (uint32_t)sd, (uint32_t)(sd >> 32));
      v = f64_to_bf16(box_muller_f64(w.x, w.y));
    }
    om[q] = v;
  }
}

// partial fp64 Gram of a row chunk: Gp[cell][chunk] += Y[rows]^T Y[rows] for the 64 x 64
// output tile (ti, tj), ti >= tj (lower tiles only; the Cholesky reads the lower triangle)
constexpr int GT = 64, GR = 32;
__global__ void __launch_bounds__(256) k_gram64(Gram64Args a) {
  const int cell = blockIdx.z, chunk = blockIdx.y;
  int t = blockIdx.x, ti = 0;
  while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
  const int tj = t - ti * (ti + 1) / 2;
  const int l = a.l;
  const float *Y = a.Y + (int64_t)cell * a.y_cell_stride;
  const int64_t r0 = (int64_t)chunk * a.chunk_rows, r1 = min((int64_t)a.rows, r0 + a.chunk_rows);
  __shared__ float ya[GR][GT + 1], yb[GR][GT + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int64_t rb = r0; rb < r1; rb += GR) {
    __syncthreads();
    for (int q = tid; q < GR * GT; q += 256) {
      const int rr = q / GT, cc = q % GT;
      const int64_t r = rb + rr;
      const int ca = ti * GT + cc, cb = tj * GT + cc;
      ya[rr][cc] = (r < r1 && ca < l) ? Y[r * a.ld + ca] : 0.f;
      yb[rr][cc] = (r < r1 && cb < l) ? Y[r * a.ld + cb] : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int rr = 0; rr < GR; ++rr) {
      double va[4], vb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { va[i] = ya[rr][ty * 4 + i]; vb[i] = yb[rr][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(va[i], vb[j], acc[i][j]);
    }
  }
  double *G = a.partial + ((int64_t)cell * a.chunks + chunk) * (int64_t)l * l;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = ti * GT + ty * 4 + i, c = tj * GT + tx * 4 + j;
      if (r < l && c < l) G[(int64_t)r * l + c] = acc[i][j];
    }
}

__global__ void k_gram64_reduce(Gram64Args a) {
  const int cell = blockIdx.y;
  const int64_t ll = (int64_t)a.l * a.l;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < ll; q += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(q / a.l), c = (int)(q % a.l);
    if (c / GT > r / GT) continue;                 // upper tiles were not computed
    double s = 0.0;
    const double *p = a.partial + (int64_t)cell * a.chunks * ll + q;
    for (int k = 0; k < a.chunks; ++k) s += p[(int64_t)k * ll];
    a.G[(int64_t)cell * ll + q] = s;
  }
}

// one workgroup per cell: G = L L^T (lower, in place), M = L^-1, Rinv = M^T (fp32, l x ldr)
constexpr int CT = 1024;
__global__ void __launch_bounds__(CT) k_chol_inv(CholArgs a) {
  const int cell = blockIdx.x, l = a.l, tid = threadIdx.x;
  const int64_t ll = (int64_t)l * l;
  double *G = a.G + (int64_t)cell * ll;
  double *M = a.M + (int64_t)cell * ll;
  float *R = a.Rinv + (int64_t)cell * l * a.ldr;
  __shared__ double smax;
  __shared__ double red[CT / 64];
  double mx = 0.0;
  for (int i = tid; i < l; i += CT) mx = fmax(mx, G[(int64_t)i * l + i]);
  for (int o = 32; o >= 1; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  if (tid == 0) {
    double m = 0.0;
    for (int w = 0; w < CT / 64; ++w) m = fmax(m, red[w]);
    smax = m;
  }
  __syncthreads();
  const double floor_piv = fmax(1e-14 * smax, 1e-300);
  for (int k = 0; k < l; ++k) {
    double piv = G[(int64_t)k * l + k];
    piv = sqrt(fmax(piv, floor_piv));
    __syncthreads();
    for (int i = k + 1 + tid; i < l; i += CT) G[(int64_t)i * l + k] /= piv;
    if (tid == 0) G[(int64_t)k * l + k] = piv;
    __syncthreads();
    // trailing update of the lower triangle, one row per thread: G[i][j] -= L[i][k] L[j][k]
    for (int gi = k + 1 + tid; gi < l; gi += CT) {
      const double lik = G[(int64_t)gi * l + k];
      double *row = G + (int64_t)gi * l;
      for (int gj = k + 1; gj <= gi; ++gj) row[gj] = fma(-lik, G[(int64_t)gj * l + k], row[gj]);
    }
    __syncthreads();
  }
  // M = L^-1 column by column (thread per column, forward substitution down the column)
  for (int j = tid; j < l; j += CT) {
    for (int i = 0; i < j; ++i) M[(int64_t)i * l + j] = 0.0;
    M[(int64_t)j * l + j] = 1.0 / G[(int64_t)j * l + j];
    for (int i = j + 1; i < l; ++i) {
      double s = 0.0;
      for (int k = j; k < i; ++k) s = fma(G[(int64_t)i * l + k], M[(int64_t)k * l + j], s);
      M[(int64_t)i * l + j] = -s / G[(int64_t)i * l + i];
    }
  }
  __syncthreads();
  for (int64_t q = tid; q < (int64_t)l * a.ldr; q += CT) {
    const int r = (int)(q / a.ldr), c = (int)(q % a.ldr);
    R[q] = (c < l) ? (float)M[(int64_t)c * l + r] : 0.f;   // Rinv[r][c] = M[c][r]
  }
}

}  // namespace

hipError_t launch_sketch(const SketchArgs &a, int n_cells, hipStream_t st) {
  int64_t total = (int64_t)a.N * a.ld;
  int64_t blocks = std::min<int64_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(k_sketch, dim3((unsigned)blocks, n_cells), dim3(256), 0, st, a);
  return hipGetLastError();
}

int gram64_tile() { return GT; }

hipError_t launch_gram64(const Gram64Args &a, int n_cells, hipStream_t st) {
  const int nt = (a.l + GT - 1) / GT;
  hipLaunchKernelGGL(k_gram64, dim3(nt * (nt + 1) / 2, a.chunks, n_cells), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t ll = (int64_t)a.l * a.l;
  hipLaunchKernelGGL(k_gram64_reduce, dim3((unsigned)std::min<int64_t>((ll + 255) / 256, 2048), n_cells),
                     dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_chol_inv(const CholArgs &a, int n_cells, hipStream_t st) {
  hipLaunchKernelGGL(k_chol_inv, dim3(n_cells), dim3(CT), 0, st, a);
  return hipGetLastError();
}

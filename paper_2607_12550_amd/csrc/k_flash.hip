// FlashJoLT randomized token-mode SVD helpers (section 5): the seeded Gaussian test
// matrix and the CholeskyQR2 orthonormalisation used by the range finder.
//
// Sketch: Omega[c][j] = bf16(sqrt(-2 ln u0) cos(2 pi u1)) with (u0, u1) from Philox4x32-10 at
// counter (c, j, 0, 2) and key = seed; Box-Muller runs in fp64 and is rounded once to bf16.
// CholeskyQR2: G = Y^T Y accumulated in fp64 (split over row chunks, partials summed in a
// fixed order), G = L L^T, Q = Y L^-T, applied twice.  fp64 keeps the Gram usable for
// condition numbers up to ~1e7.  Directions whose Cholesky pivot falls below 1e-14 of
// the largest diagonal are treated as numerically absent (pivot clamped), so
// rank-deficient sketches stay finite.
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
// output tile (ti, tj), ti >= tj (lower tiles only; the Cholesky reads the lower triangle).
// Each thread loads two 4-column runs of both 32 x 64 operand blocks; the next block's loads
// are issued before the current block is multiplied, so their latency overlaps the fp64
// multiply-adds.
constexpr int GT = 64, GR = 32;

// four consecutive entries of row r from column c (zero at and beyond column l)
JOLT_DEV jf4 gram64_load4(const float *Y, int64_t ld, int64_t r, bool row_ok, int c, int l) {
  if (!row_ok || c >= l) return jf4{0.f, 0.f, 0.f, 0.f};
  const float *p = Y + r * ld + c;
  if (c + 4 <= l && ((reinterpret_cast<uintptr_t>(p) & 15) == 0)) return gload_f4(p);
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = c + e < l ? p[e] : 0.f;
  return jf4{v[0], v[1], v[2], v[3]};
}

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
  // staging: thread (ty, tx) moves rows ty and ty + 16, columns 4 tx .. 4 tx + 3 of each block
  jf4 pa[2], pb[2];
  auto fetch = [&](int64_t rb) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t r = rb + ty + 16 * h;
      pa[h] = gram64_load4(Y, a.ld, r, r < r1, ti * GT + 4 * tx, l);
      pb[h] = gram64_load4(Y, a.ld, r, r < r1, tj * GT + 4 * tx, l);
    }
  };
  if (r0 < r1) fetch(r0);
  for (int64_t rb = r0; rb < r1; rb += GR) {
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ya[ty + 16 * h][4 * tx + e] = pa[h][e];
        yb[ty + 16 * h][4 * tx + e] = pb[h][e];
      }
    __syncthreads();
    if (rb + GR < r1) fetch(rb + GR);
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

// fp32 Gram (from the matrix-core GEMM) widened to the fp64 layout the Cholesky reads
__global__ void k_widen_gram(const float *C, double *G, int l, int n_cells) {
  const int64_t ll = (int64_t)l * l, total = ll * n_cells;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total; q += (int64_t)gridDim.x * blockDim.x)
    G[q] = (double)C[q];
}

// Blocked Cholesky G = L L^T and triangular inverse M = L^-1 in fp64, 64 x 64 tiles.
// Per block column kb: k_chol_diag factors the diagonal tile in LDS and inverts it
// (D_kb = L_kb,kb^-1), k_chol_panel forms L_I,kb = G_I,kb D_kb^T below it and
// k_chol_update subtracts L_I,kb L_J,kb^T from the trailing lower tiles.  The inverse
// is then built one block row at a time: M_IJ = -D_I sum_{J<=K<I} L_IK M_KJ.
// Pivots below 1e-14 of the largest diagonal entry of G are raised to that floor and
// counted per cell (CholArgs::clamped).
constexpr int CB = 64, CLD = CB + 1;

JOLT_DEV void tile_load(double (*t)[CLD], const double *A, int l, int r0, int c0) {
  for (int q = threadIdx.x; q < CB * CB; q += 256) {
    const int i = q / CB, j = q % CB, r = r0 + i, c = c0 + j;
    t[i][j] = (r < l && c < l) ? A[(int64_t)r * l + c] : 0.0;
  }
}

// Diagonal tile of block column kb, one wavefront: lane i keeps row i of the tile in
// registers.  Column j is factored by broadcasting its pivot and its entries l_kj across the
// lanes (shuffles, no barriers), with the same operations in the same order as a
// right-looking factorisation: l_ij = t_ij / sqrt(t_jj), t_ik -= l_ij l_kj (j < k <= i).  The
// factor is then staged in LDS and lane j forms column j of its inverse by forward
// substitution: inv_jj = 1 / l_jj, inv_ij = -(sum_{j<=k<i} l_ik inv_kj) / l_ii.
__global__ void __launch_bounds__(CB) k_chol_diag(CholArgs a, int kb) {
  static_assert(CB == 64, "one lane per tile row");
  const int cell = blockIdx.x, l = a.l, lane = threadIdx.x;
  double *G = a.G + (int64_t)cell * l * l;
  double *D = a.Dinv + ((int64_t)cell * a.nbk + kb) * CB * CB;
  double *M = a.M + (int64_t)cell * l * l;
  __shared__ double ts[CB][CLD];
  double sdmax;
  if (kb == 0) {                       // largest diagonal entry of the untouched Gram
    double mx = 0.0;
    for (int i = lane; i < l; i += CB) mx = fmax(mx, G[(int64_t)i * l + i]);
    for (int o = 32; o >= 1; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
    if (lane == 0) a.dmax[cell] = mx;
    sdmax = mx;
  } else {
    sdmax = a.dmax[cell];              // written by the kb = 0 launch
  }
  const int o = kb * CB, nb = min(CB, l - o);
  double t[CB];
#pragma unroll
  for (int c = 0; c < CB; ++c)        // zeros outside the matrix, identity on the padding
    t[c] = (lane < nb && c < nb) ? G[(int64_t)(o + lane) * l + o + c] : (c == lane && lane >= nb ? 1.0 : 0.0);
  // an all-zero Gram (a zero cell) factors as the identity: Q = Y L^-T stays zero and finite
  const double floor_piv = sdmax > 0.0 ? fmax(1e-14 * sdmax, 1e-300) : 1.0;
  int n_clamped = 0;                   // pivots of this tile raised to the floor
  // column j of the factor is broadcast through LDS (two alternating buffers, so one
  // barrier per column): every lane reads the entries l_kj it needs with independent
  // broadcast loads instead of one cross-lane shuffle pair per entry
  __shared__ double colb[2][CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    const double raw = __shfl(t[j], j, 64);
    n_clamped += (j < nb && !(raw >= floor_piv)) ? 1 : 0;
    const double piv = sqrt(fmax(raw, j < nb ? floor_piv : 1.0));
    if (lane > j) t[j] /= piv;
    else if (lane == j) t[j] = piv;
    const double lij = t[j];
    colb[j & 1][lane] = lij;
    __syncthreads();
#pragma unroll
    for (int k = j + 1; k < CB; ++k) {
      const double lkj = colb[j & 1][k];
      if (lane >= k) t[k] = fma(-lij, lkj, t[k]);
    }
  }
#pragma unroll
  for (int c = 0; c < CB; ++c) ts[lane][c] = t[c];
  // clamp count of the whole factorisation: reset by the first block column's launch
  if (lane == 0 && a.clamped) a.clamped[cell] = (kb == 0 ? 0 : a.clamped[cell]) + n_clamped;
  __syncthreads();
  // column `lane` of the inverse of the lower-triangular factor
  double inv[CB];
#pragma unroll
  for (int i = 0; i < CB; ++i) inv[i] = 0.0;
  const double djj = 1.0 / ts[lane][lane];
#pragma unroll
  for (int i = 0; i < CB; ++i) if (i == lane) inv[i] = djj;
#pragma unroll
  for (int i = 1; i < CB; ++i) {
    double sum = 0.0;
#pragma unroll
    for (int k = 0; k < i; ++k) sum = fma(ts[i][k], inv[k], sum);   // inv[k] = 0 for k < lane
    if (lane < i) inv[i] = -sum / ts[i][i];
  }
#pragma unroll
  for (int r = 0; r < CB; ++r) {
    D[r * CB + lane] = inv[r];
    if (r < nb && lane < nb) {
      if (lane <= r) G[(int64_t)(o + r) * l + o + lane] = ts[r][lane];
      M[(int64_t)(o + r) * l + o + lane] = inv[r];
    }
  }
}

// 4 x 4 outputs per thread of a 64 x 64 tile: acc[r][c] += sum_k A[r][k] B[c][k]
JOLT_DEV void tile_mma_nt(double (&acc)[4][4], const double (*A)[CLD], const double (*B)[CLD], int k0, int k1) {
  const int r0 = (threadIdx.x >> 4) * 4, c0 = (threadIdx.x & 15) * 4;
  for (int k = k0; k < k1; ++k) {
    double av[4], bv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) { av[i] = A[r0 + i][k]; bv[i] = B[c0 + i][k]; }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[i][c] = fma(av[i], bv[c], acc[i][c]);
  }
}

__global__ void __launch_bounds__(256) k_chol_panel(CholArgs a, int kb) {
  const int cell = blockIdx.y, I = kb + 1 + blockIdx.x, l = a.l;
  double *G = a.G + (int64_t)cell * l * l;
  const double *D = a.Dinv + ((int64_t)cell * a.nbk + kb) * CB * CB;
  __shared__ double ta[CB][CLD], td[CB][CLD];
  tile_load(ta, G, l, I * CB, kb * CB);
  for (int q = threadIdx.x; q < CB * CB; q += 256) td[q / CB][q % CB] = D[q];
  __syncthreads();
  double acc[4][4] = {};
  tile_mma_nt(acc, ta, td, 0, CB);             // L_I,kb = G_I,kb D^T
  const int r0 = (threadIdx.x >> 4) * 4, c0 = (threadIdx.x & 15) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = I * CB + r0 + i, cc = kb * CB + c0 + c;
      if (r < l && cc < l) G[(int64_t)r * l + cc] = acc[i][c];
    }
}

__global__ void __launch_bounds__(256) k_chol_update(CholArgs a, int kb) {
  const int cell = blockIdx.y, l = a.l;
  int t = blockIdx.x, ti = 0;
  while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
  const int I = kb + 1 + ti, J = kb + 1 + (t - ti * (ti + 1) / 2);
  double *G = a.G + (int64_t)cell * l * l;
  __shared__ double ta[CB][CLD], tb[CB][CLD];
  tile_load(ta, G, l, I * CB, kb * CB);
  tile_load(tb, G, l, J * CB, kb * CB);
  __syncthreads();
  double acc[4][4] = {};
  tile_mma_nt(acc, ta, tb, 0, CB);
  const int r0 = (threadIdx.x >> 4) * 4, c0 = (threadIdx.x & 15) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = I * CB + r0 + i, cc = J * CB + c0 + c;
      if (r < l && cc < l) G[(int64_t)r * l + cc] -= acc[i][c];
    }
}

// block row I of M = L^-1: M_IJ = -D_I sum_{K=J}^{I-1} L_IK M_KJ for every J < I
__global__ void __launch_bounds__(256) k_chol_inv_row(CholArgs a, int I) {
  const int cell = blockIdx.y, J = blockIdx.x, l = a.l;
  const double *G = a.G + (int64_t)cell * l * l;
  double *M = a.M + (int64_t)cell * l * l;
  const double *D = a.Dinv + ((int64_t)cell * a.nbk + I) * CB * CB;
  __shared__ double ta[CB][CLD], tb[CB][CLD];
  const int r0 = (threadIdx.x >> 4) * 4, c0 = (threadIdx.x & 15) * 4;
  double acc[4][4] = {};
  // the tiles of step K + 1 (L_I,K+1 and M_K+1,J) are loaded into registers while step K
  // is multiplied; thread element h is entry (q / CB, q % CB), q = tid + 256 h, of each tile
  constexpr int PE = CB * CB / 256;
  double pa[PE], pb[PE];
  auto fetch = [&](int K) {
#pragma unroll
    for (int h = 0; h < PE; ++h) {
      const int q = threadIdx.x + 256 * h, i = q / CB, j = q % CB;
      const int ra = I * CB + i, ca = K * CB + j, rb = K * CB + i, cb = J * CB + j;
      pa[h] = (ra < l && ca < l) ? G[(int64_t)ra * l + ca] : 0.0;          // L_IK[i][j]
      pb[h] = (rb < l && cb < l) ? M[(int64_t)rb * l + cb] : 0.0;          // M_KJ[i][j]
    }
  };
  if (J < I) fetch(J);
  for (int K = J; K < I; ++K) {
    __syncthreads();
#pragma unroll
    for (int h = 0; h < PE; ++h) {
      const int q = threadIdx.x + 256 * h, i = q / CB, j = q % CB;
      ta[i][j] = pa[h];
      tb[j][i] = pb[h];                                   // transposed: tb[c][k] = M_KJ[k][c]
    }
    __syncthreads();
    if (K + 1 < I) fetch(K + 1);
    tile_mma_nt(acc, ta, tb, 0, CB);
  }
  __syncthreads();
  // S = acc -> tb (transposed, tb[c][k] = S[k][c]); D_I -> ta
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) tb[c0 + c][r0 + i] = acc[i][c];
  for (int q = threadIdx.x; q < CB * CB; q += 256) ta[q / CB][q % CB] = D[q];
  __syncthreads();
  double out[4][4] = {};
  tile_mma_nt(out, ta, tb, 0, CB);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = I * CB + r0 + i, cc = J * CB + c0 + c;
      if (r < l && cc < l) M[(int64_t)r * l + cc] = -out[i][c];
    }
}

// Rinv = M^T in fp32 (l x ldr), zero above the diagonal of M and in the padding columns
__global__ void k_chol_rinv(CholArgs a) {
  const int cell = blockIdx.y, l = a.l;
  const double *M = a.M + (int64_t)cell * l * l;
  float *R = a.Rinv + (int64_t)cell * l * a.ldr;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < (int64_t)l * a.ldr;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(q / a.ldr), c = (int)(q % a.ldr);
    R[q] = (c < l && c >= r) ? (float)M[(int64_t)c * l + r] : 0.f;
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

// Split-K partial Grams (lower-triangle tiles of each row chunk's product, chunk t of cell c
// at part[(c * n_split + t) * l * l]) summed in chunk order in fp64 into the full symmetric
// fp64 Gram the Cholesky reads
__global__ void k_sum_gram_parts(const float *part, double *G, int l, int n_split, int n_cells) {
  const int64_t ll = (int64_t)l * l, total = ll * n_cells;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total; q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = q / ll, e = q - c * ll;
    const int i = (int)(e / l), j = (int)(e - (int64_t)i * l);
    const float *p = part + c * n_split * ll + (int64_t)max(i, j) * l + min(i, j);
    double s = 0.0;
    for (int t = 0; t < n_split; ++t) s += (double)p[(int64_t)t * ll];
    G[q] = s;
  }
}

hipError_t launch_sum_gram_parts(const float *part, double *G, int l, int n_split, int n_cells, hipStream_t st) {
  const int64_t total = (int64_t)l * l * n_cells;
  hipLaunchKernelGGL(k_sum_gram_parts, dim3((unsigned)std::min<int64_t>((total + 255) / 256, 4096)), dim3(256), 0,
                     st, part, G, l, n_split, n_cells);
  return hipGetLastError();
}

hipError_t launch_widen_gram(const float *C, double *G, int l, int n_cells, hipStream_t st) {
  const int64_t total = (int64_t)l * l * n_cells;
  hipLaunchKernelGGL(k_widen_gram, dim3((unsigned)std::min<int64_t>((total + 255) / 256, 4096)), dim3(256), 0, st,
                     C, G, l, n_cells);
  return hipGetLastError();
}

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

int chol_blocks(int l) { return (l + CB - 1) / CB; }

hipError_t launch_chol_inv(const CholArgs &a, int n_cells, hipStream_t st) {
  const int nbk = a.nbk;
  if (nbk != chol_blocks(a.l)) return hipErrorInvalidValue;
  for (int kb = 0; kb < nbk; ++kb) {
    hipLaunchKernelGGL(k_chol_diag, dim3(n_cells), dim3(CB), 0, st, a, kb);
    const int below = nbk - kb - 1;
    if (below > 0) {
      hipLaunchKernelGGL(k_chol_panel, dim3(below, n_cells), dim3(256), 0, st, a, kb);
      hipLaunchKernelGGL(k_chol_update, dim3(below * (below + 1) / 2, n_cells), dim3(256), 0, st, a, kb);
    }
  }
  for (int I = 1; I < nbk; ++I)
    hipLaunchKernelGGL(k_chol_inv_row, dim3(I, n_cells), dim3(256), 0, st, a, I);
  const int64_t tot = (int64_t)a.l * a.ldr;
  hipLaunchKernelGGL(k_chol_rinv, dim3((unsigned)std::min<int64_t>((tot + 255) / 256, 1024), n_cells),
                     dim3(256), 0, st, a);
  return hipGetLastError();
}

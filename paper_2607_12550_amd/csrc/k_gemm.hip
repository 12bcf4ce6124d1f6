// Batched fp32 MFMA GEMM for gfx950 (v_mfma_f32_32x32x2_f32): the products that need
// fp32 operands in full, i.e. the reconstruction U_T W_s from the stored factors, the
// ST-HOSVD core products, the eigensolver's blocked updates and back-transforms, the
// FlashJoLT B B^T and fp32 cells, and the fallback for any table the bf16 kernel's layout
// conditions reject.  Inputs (bf16 / fp16 / fp32) are widened exactly to fp32.
//
// Tile: 128 x 128 outputs per 256-thread workgroup, 4 wavefronts in a 2 x 2 grid,
// each wave owning 64 x 64 = 2 x 2 MFMA 32x32 blocks.  K advances in steps of 32;
// the next K tile is fetched into registers while the current one is multiplied
// out of LDS.  LDS keeps both operands k-contiguous; within a K tile the k index is
// permuted identically for A and B (a sum over k does not depend on its order) so
// that each lane reads its fragment with 16-byte LDS loads.
// Operands are addressed through GemmOperand so the cache cell (slices at two-level
// strides) is read in place, never repacked.
#include "common.h"
#include "kernels.h"

typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace {

constexpr int BM = 128, BN = 128, BK = 32, NT = 256;

JOLT_DEV int64_t op_offset(const GemmOperand &op, int row, int col) {
  return (int64_t)row * op.ld + operand_col(op, col);
}

template <int TY>
JOLT_DEV float load_elem(const void *p, int64_t off) {
  if constexpr (TY == GT_BF16) return bf16_to_f32(gptr(reinterpret_cast<const uint16_t *>(p))[off]);
  else if constexpr (TY == GT_F16) return (float)gptr(reinterpret_cast<const _Float16 *>(p))[off];
  else return gptr(reinterpret_cast<const float *>(p))[off];
}

// 8 consecutive elements along the operand's contiguous dimension, widened to fp32
template <int TY>
JOLT_DEV void load8_f32(const GemmOperand &op, int row, int col, int nrows, int ncols,
                        float (&v)[8]) {
  const int64_t off0 = (row < nrows && col + 8 <= ncols) ? op_offset(op, row, col) : 0;
  const size_t esz = TY == GT_F32 ? 4 : 2;
  if (row < nrows && col + 8 <= ncols &&
      ((reinterpret_cast<uintptr_t>(op.ptr) + (uintptr_t)off0 * esz) & 15) == 0) {
    const int64_t off = off0;
    if constexpr (TY == GT_F32) {
      const float *q = reinterpret_cast<const float *>(op.ptr) + off;
      const jf4 a = gload_f4(q), b = gload_f4(q + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
      const ju4 u = gload_u4(reinterpret_cast<const uint16_t *>(op.ptr) + off);
      uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint16_t lo = (uint16_t)(w[i] & 0xffff), hi = (uint16_t)(w[i] >> 16);
        if constexpr (TY == GT_BF16) {
          v[2 * i] = bf16_to_f32(lo); v[2 * i + 1] = bf16_to_f32(hi);
        } else {
          _Float16 a, b;
          __builtin_memcpy(&a, &lo, 2); __builtin_memcpy(&b, &hi, 2);
          v[2 * i] = (float)a; v[2 * i + 1] = (float)b;
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      v[i] = (row < nrows && col + i < ncols) ? load_elem<TY>(op.ptr, op_offset(op, row, col + i)) : 0.f;
  }
}

// Each thread moves two 8-element chunks of a 128 x 32 (k-contiguous) or
// 32 x 128 (mn-contiguous) operand tile per K step.
template <bool KCONTIG>
JOLT_DEV void chunk_coords(int chunk, int &r, int &c) {
  if (KCONTIG) { r = chunk >> 2; c = (chunk & 3) * 8; }   // 128 rows x 4 chunks
  else { r = chunk >> 4; c = (chunk & 15) * 8; }          // 32 rows x 16 chunks
}

struct Smem {
  static constexpr int LD = BK + 4;                       // fp32 elements
  float a[BM * LD], b[BN * LD];
};

template <int TA, int TB, bool AK, bool BK_>
__global__ void __launch_bounds__(NT) k_gemm(const GemmProblem *__restrict__ probs) {
  const GemmProblem &P = probs[blockIdx.z];
  const int tm = blockIdx.y, tn = blockIdx.x;
  if (tm * BM >= P.M || tn * BN >= P.N) return;
  if (P.lower_only && tm < tn) return;
  __shared__ Smem sm;
  constexpr int LD = Smem::LD;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = tm * BM, n0 = tn * BN;

  // memory-order dims of the operands
  const int a_rows = AK ? P.M : P.K, a_cols = AK ? P.K : P.M;
  const int b_rows = BK_ ? P.N : P.K, b_cols = BK_ ? P.K : P.N;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  // register staging of the next tile
  float ra[2][8], rb[2][8];

  auto fetch = [&](int k0) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      int r, c;
      const int chunk = tid + h * NT;
      chunk_coords<AK>(chunk, r, c);
      const int ar = AK ? m0 + r : k0 + r, ac = AK ? k0 + c : m0 + c;
      chunk_coords<BK_>(chunk, r, c);
      const int br = BK_ ? n0 + r : k0 + r, bc = BK_ ? k0 + c : n0 + c;
      load8_f32<TA>(P.A, ar, ac, a_rows, a_cols, ra[h]);
      load8_f32<TB>(P.B, br, bc, b_rows, b_cols, rb[h]);
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      int r, c;
      const int chunk = tid + h * NT;
      chunk_coords<AK>(chunk, r, c);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int idx = AK ? r * LD + c + i : (c + i) * LD + r;
        sm.a[idx] = ra[h][i];
      }
      chunk_coords<BK_>(chunk, r, c);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int idx = BK_ ? r * LD + c + i : (c + i) * LD + r;
        sm.b[idx] = rb[h][i];
      }
    }
  };

  const int lr = lane & 31, lh = lane >> 5;
  fetch(0);
  for (int k0 = 0; k0 < P.K; k0 += BK) {
    __syncthreads();
    stash();
    __syncthreads();
    if (k0 + BK < P.K) fetch(k0 + BK);
    // lane group lh covers k in [16 lh, 16 lh + 16): sixteen MFMA steps of 2
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float4 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = *reinterpret_cast<const float4 *>(&sm.a[(wm * 64 + i * 32 + lr) * LD + lh * 16 + q * 4]);
        fb[i] = *reinterpret_cast<const float4 *>(&sm.b[(wn * 64 + i * 32 + lr) * LD + lh * 16 + q * 4]);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][s], fb[j][s], acc[i][j], 0, 0, 0);
    }
  }

  // alpha 2^e is applied as ldexp(alpha * acc, e): 2^e alone may lie outside fp32's range
  const float alpha = P.alpha;
  const int aexp = P.alpha_exp2 ? (int)*gptr(P.alpha_exp2) : 0;
  // Epilogue through LDS, 32 rows at a time (one MFMA row block of one wave row per round),
  // so that C is read (beta != 0) and written as float4 rows: acc[i][j][q] is the output at
  // row wm*64 + i*32 + 8*(q/4) + 4*lh + q%4, column wn*64 + j*32 + lr of the tile.
  float *cs = reinterpret_cast<float *>(&sm);
  constexpr int CLD = BN + 4;
  static_assert(32 * CLD * sizeof(float) <= sizeof(Smem), "epilogue tile exceeds LDS");
  const bool use_beta = P.beta != 0.f;
  const bool vec = ((reinterpret_cast<uintptr_t>(P.C) & 15) == 0) && (P.ldc % 4 == 0);
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    __syncthreads();
    if (wm == (h >> 1)) {
      const int i = h & 1;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q)
          cs[(8 * (q >> 2) + 4 * lh + (q & 3)) * CLD + wn * 64 + j * 32 + lr] = acc[i][j][q];
    }
    __syncthreads();
    // 32 rows x 32 float4 chunks, 4 per thread
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + u * NT, rr = idx >> 5, cc = (idx & 31) * 4;
      const int row = m0 + h * 32 + rr, col = n0 + cc;
      if (row >= P.M || col >= P.N) continue;
      const float4 a4 = *reinterpret_cast<const float4 *>(&cs[rr * CLD + cc]);
      float v[4] = {ldexpf(alpha * a4.x, aexp), ldexpf(alpha * a4.y, aexp), ldexpf(alpha * a4.z, aexp),
                     ldexpf(alpha * a4.w, aexp)};
      JOLT_GLOBAL float *dst = gptr(P.C + (int64_t)row * P.ldc + col);
      if (vec && col + 4 <= P.N) {
        if (use_beta) {
          const jf4 o4 = *reinterpret_cast<const JOLT_GLOBAL jf4 *>(dst);
          v[0] = fmaf(P.beta, o4.x, v[0]); v[1] = fmaf(P.beta, o4.y, v[1]);
          v[2] = fmaf(P.beta, o4.z, v[2]); v[3] = fmaf(P.beta, o4.w, v[3]);
        }
        *reinterpret_cast<JOLT_GLOBAL jf4 *>(dst) = jf4{v[0], v[1], v[2], v[3]};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < P.N) dst[e] = use_beta ? fmaf(P.beta, dst[e], v[e]) : v[e];
      }
    }
  }
}

template <int TA, int TB>
hipError_t launch_t(const GemmProblem *probs, int n, dim3 grid, bool ak, bool bk, hipStream_t st) {
  if (ak && bk) hipLaunchKernelGGL((k_gemm<TA, TB, true, true>), grid, dim3(NT), 0, st, probs);
  else if (ak) hipLaunchKernelGGL((k_gemm<TA, TB, true, false>), grid, dim3(NT), 0, st, probs);
  else if (bk) hipLaunchKernelGGL((k_gemm<TA, TB, false, true>), grid, dim3(NT), 0, st, probs);
  else hipLaunchKernelGGL((k_gemm<TA, TB, false, false>), grid, dim3(NT), 0, st, probs);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmProblem *probs_dev, int n_probs, int max_M, int max_N, int mode,
                       int ta, int tb, bool a_kcontig, bool b_kcontig, hipStream_t st) {
  if (n_probs <= 0 || max_M <= 0 || max_N <= 0) return hipSuccess;
  dim3 grid((max_N + BN - 1) / BN, (max_M + BM - 1) / BM, n_probs);
  if (mode != 1) return hipErrorInvalidValue;
#define TT(A_, B_) if (ta == A_ && tb == B_) return launch_t<A_, B_>(probs_dev, n_probs, grid, a_kcontig, b_kcontig, st)
  TT(GT_F32, GT_F32);
  TT(GT_BF16, GT_F32);
  TT(GT_F32, GT_BF16);
  TT(GT_F16, GT_F32);
  TT(GT_F32, GT_F16);
  TT(GT_F16, GT_F16);
  TT(GT_BF16, GT_BF16);
#undef TT
  return hipErrorInvalidValue;
}

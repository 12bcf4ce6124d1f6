// Batched GEMM on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16, fp32 accumulate) for
// the contractions that read the cache: the token Gram, the FlashJoLT sketch products
// X Omega, X^T Q, X Q' and Q^T X, and the ST-HOSVD projection U_T^T X.
//
// Operands are bf16 (used as they are) or fp32, in which case each element is split on
// the fly into x = hi + lo with hi = bf16(x), lo = bf16(x - hi) (both round to nearest
// even) and the product takes two MFMA passes (A hi * B + A lo * B, or the same for B):
// |x - hi - lo| <= 2^-17 |x|, so the products carry about 16 significant bits where the
// other operand is exact bf16 data.
//
// Tile 128 x 128 per 256-thread workgroup (4 waves, each 64 x 64 = 2 x 2 MFMA blocks),
// K tiles of 64 staged through LDS with the next tile held in registers while the current
// one is multiplied.  LDS keeps both operands k-contiguous (rows of 64 + 8 bf16); an
// operand whose memory layout is contiguous along M/N is transposed in registers (each
// thread moves a 4 (k) x 8 (m) block and writes 8-byte k-runs), never element by element.
#include "common.h"
#include "kernels.h"

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace {

constexpr int BM = 128, BN = 128, BK = 64, NT = 256, LDK = BK + 8;

JOLT_DEV int64_t opoff(const GemmOperand &op, int row, int col) {
  return (int64_t)row * op.ld + operand_col(op, col);
}

JOLT_DEV void split_bf16(float x, uint16_t &h, uint16_t &l) {
  h = f32_to_bf16(x);
  l = f32_to_bf16(x - bf16_to_f32(h));
}

// 8 consecutive elements along the operand's contiguous axis at (row, col): raw bf16 bits,
// or fp32 values; out-of-range elements read as zero
template <bool F32>
struct Vec8 {
  uint16_t h[8];
};
template <>
struct Vec8<true> {
  float f[8];
};

template <bool F32>
JOLT_DEV void load8(const GemmOperand &op, int row, int col, int nrows, int ncols, Vec8<F32> &v) {
  const bool in = row < nrows && col + 8 <= ncols;
  const int64_t o = in ? opoff(op, row, col) : 0;
  if constexpr (F32) {
    const float *p = reinterpret_cast<const float *>(op.ptr) + o;
    if (in && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      const jf4 a = gload_f4(p), b = gload_f4(p + 4);
      v.f[0] = a.x; v.f[1] = a.y; v.f[2] = a.z; v.f[3] = a.w;
      v.f[4] = b.x; v.f[5] = b.y; v.f[6] = b.z; v.f[7] = b.w;
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v.f[i] = (row < nrows && col + i < ncols)
                     ? gptr(reinterpret_cast<const float *>(op.ptr))[opoff(op, row, col + i)] : 0.f;
    }
  } else {
    const uint16_t *p = reinterpret_cast<const uint16_t *>(op.ptr) + o;
    if (in && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      const ju4 u = gload_u4(p);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) { v.h[2 * i] = (uint16_t)(w[i] & 0xffff); v.h[2 * i + 1] = (uint16_t)(w[i] >> 16); }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        v.h[i] = (row < nrows && col + i < ncols)
                     ? gptr(reinterpret_cast<const uint16_t *>(op.ptr))[opoff(op, row, col + i)] : (uint16_t)0;
    }
  }
}

JOLT_DEV uint32_t pk(uint16_t a, uint16_t b) { return (uint32_t)a | ((uint32_t)b << 16); }

// Staging of one 128 (m or n) x 64 (k) operand tile.
//   k-contiguous: thread t moves units u = t + 256 q (q < 4): row u / 8, k run (u % 8) * 8;
//   mn-contiguous: thread t moves the 4 (k) x 8 (mn) block at k (t / 16) * 4, mn (t % 16) * 8.
template <bool KC, bool F32>
struct Stager {
  static constexpr int NV = KC ? 4 : 4;   // vectors held per thread
  Vec8<F32> v[NV];

  JOLT_DEV void fetch(const GemmOperand &op, int mn0, int k0, int MN, int K, int tid) {
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      if constexpr (KC) {
        const int u = tid + NT * q, r = u >> 3, kc = (u & 7) * 8;
        load8<F32>(op, mn0 + r, k0 + kc, MN, K, v[q]);
      } else {
        const int kb = (tid >> 4) * 4, mb = (tid & 15) * 8;
        load8<F32>(op, k0 + kb + q, mn0 + mb, K, MN, v[q]);
      }
    }
  }

  // hi (and lo for fp32) tiles: [128][LDK] bf16 each
  JOLT_DEV void stash(uint16_t *hi, uint16_t *lo, int tid) const {
    if constexpr (KC) {
#pragma unroll
      for (int q = 0; q < NV; ++q) {
        const int u = tid + NT * q, r = u >> 3, kc = (u & 7) * 8;
        uint16_t h[8], l[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if constexpr (F32) split_bf16(v[q].f[i], h[i], l[i]);
          else h[i] = v[q].h[i];
        }
        *reinterpret_cast<uint4 *>(hi + r * LDK + kc) = make_uint4(pk(h[0], h[1]), pk(h[2], h[3]), pk(h[4], h[5]), pk(h[6], h[7]));
        if constexpr (F32)
          *reinterpret_cast<uint4 *>(lo + r * LDK + kc) = make_uint4(pk(l[0], l[1]), pk(l[2], l[3]), pk(l[4], l[5]), pk(l[6], l[7]));
      }
    } else {
      const int kb = (tid >> 4) * 4, mb = (tid & 15) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        uint16_t h[4], l[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if constexpr (F32) split_bf16(v[q].f[e], h[q], l[q]);
          else h[q] = v[q].h[e];
        }
        *reinterpret_cast<uint2 *>(hi + (mb + e) * LDK + kb) = make_uint2(pk(h[0], h[1]), pk(h[2], h[3]));
        if constexpr (F32)
          *reinterpret_cast<uint2 *>(lo + (mb + e) * LDK + kb) = make_uint2(pk(l[0], l[1]), pk(l[2], l[3]));
      }
    }
  }
};

template <bool AS, bool BS>
struct Lds16 {
  static constexpr int TILE = 128 * LDK;
  uint16_t a[TILE * (AS ? 2 : 1)];
  uint16_t b[TILE * (BS ? 2 : 1)];
};

// AK/BK_: operand k-contiguous in memory; AS/BS: operand is fp32 (split into hi + lo)
template <bool AK, bool BK_, bool AS, bool BS>
__global__ void __launch_bounds__(NT) k_gemm16(const GemmProblem *__restrict__ probs) {
  const GemmProblem &P = probs[blockIdx.z];
  const int tm = blockIdx.y, tn = blockIdx.x;
  if (tm * BM >= P.M || tn * BN >= P.N) return;
  if (P.lower_only && tm < tn) return;
  __shared__ __attribute__((aligned(16))) Lds16<AS, BS> sm;
  constexpr int TILE = Lds16<AS, BS>::TILE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, lr = lane & 31, lh = lane >> 5;
  const int m0 = tm * BM, n0 = tn * BN;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  Stager<AK, AS> sa;
  Stager<BK_, BS> sb;
  sa.fetch(P.A, m0, 0, P.M, P.K, tid);
  sb.fetch(P.B, n0, 0, P.N, P.K, tid);
  for (int k0 = 0; k0 < P.K; k0 += BK) {
    __syncthreads();
    sa.stash(sm.a, sm.a + TILE, tid);
    sb.stash(sm.b, sm.b + TILE, tid);
    __syncthreads();
    if (k0 + BK < P.K) {
      sa.fetch(P.A, m0, k0 + BK, P.M, P.K, tid);
      sb.fetch(P.B, n0, k0 + BK, P.N, P.K, tid);
    }
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int ko = s * 16 + 8 * lh;
      bf16x8_t fa[2], fb[2], la[2], lb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int ra = (wm * 64 + i * 32 + lr) * LDK + ko, rb = (wn * 64 + i * 32 + lr) * LDK + ko;
        fa[i] = *reinterpret_cast<const bf16x8_t *>(sm.a + ra);
        fb[i] = *reinterpret_cast<const bf16x8_t *>(sm.b + rb);
        if constexpr (AS) la[i] = *reinterpret_cast<const bf16x8_t *>(sm.a + TILE + ra);
        if constexpr (BS) lb[i] = *reinterpret_cast<const bf16x8_t *>(sm.b + TILE + rb);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
          if constexpr (AS) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(la[i], fb[j], acc[i][j], 0, 0, 0);
          if constexpr (BS) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], lb[j], acc[i][j], 0, 0, 0);
        }
    }
  }

  float alpha = P.alpha;
  if (P.alpha_exp2) alpha = ldexpf(alpha, (int)*gptr(P.alpha_exp2));
  // epilogue through LDS, 32 rows per round: acc[i][j][q] is the output at row
  // wm*64 + i*32 + 8*(q/4) + 4*lh + q%4, column wn*64 + j*32 + lr of the tile
  float *cs = reinterpret_cast<float *>(&sm);
  constexpr int CLD = BN + 4;
  static_assert(32 * CLD * sizeof(float) <= sizeof(Lds16<AS, BS>), "epilogue tile exceeds LDS");
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
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + u * NT, rr = idx >> 5, cc = (idx & 31) * 4;
      const int row = m0 + h * 32 + rr, col = n0 + cc;
      if (row >= P.M || col >= P.N) continue;
      const float4 a4 = *reinterpret_cast<const float4 *>(&cs[rr * CLD + cc]);
      float v[4] = {alpha * a4.x, alpha * a4.y, alpha * a4.z, alpha * a4.w};
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

template <bool AS, bool BS>
hipError_t launch16(const GemmProblem *probs, dim3 grid, bool ak, bool bk, hipStream_t st) {
  if (ak && bk) hipLaunchKernelGGL((k_gemm16<true, true, AS, BS>), grid, dim3(NT), 0, st, probs);
  else if (ak) hipLaunchKernelGGL((k_gemm16<true, false, AS, BS>), grid, dim3(NT), 0, st, probs);
  else if (bk) hipLaunchKernelGGL((k_gemm16<false, true, AS, BS>), grid, dim3(NT), 0, st, probs);
  else hipLaunchKernelGGL((k_gemm16<false, false, AS, BS>), grid, dim3(NT), 0, st, probs);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm16(const GemmProblem *probs_dev, int n_probs, int max_M, int max_N, int ta,
                         int tb, bool a_kcontig, bool b_kcontig, hipStream_t st) {
  if (n_probs <= 0 || max_M <= 0 || max_N <= 0) return hipSuccess;
  const dim3 grid((max_N + BN - 1) / BN, (max_M + BM - 1) / BM, n_probs);
  const bool as = ta == GT_F32, bs = tb == GT_F32;
  if ((ta != GT_BF16 && !as) || (tb != GT_BF16 && !bs) || (as && bs)) return hipErrorInvalidValue;
  if (as) return launch16<true, false>(probs_dev, grid, a_kcontig, b_kcontig, st);
  if (bs) return launch16<false, true>(probs_dev, grid, a_kcontig, b_kcontig, st);
  return launch16<false, false>(probs_dev, grid, a_kcontig, b_kcontig, st);
}

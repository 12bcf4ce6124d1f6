// Batched GEMM on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16, fp32 accumulate) for
// the contractions that read the cache: the token Gram, the FlashJoLT sketch products
// X Omega, X^T Q, X Q' and Q^T X, the ST-HOSVD projection U_T^T X, and the products of
// the FlashJoLT orthonormaliser.
//
// Operands are bf16 (used as they are) or fp32, in which case each element is split on
// the fly into x = hi + lo with hi = bf16(x), lo = bf16(x - hi) (both round to nearest
// even): |x - hi - lo| <= 2^-17 |x|.  One fp32 operand takes two MFMA passes
// (A hi * B + A lo * B, or the same for B); two fp32 operands take three
// (hi*hi + lo*hi + hi*lo, dropping lo*lo, which is below 2^-16 of the product).
//
// Tile BM x BN (128 x 128, 256 x 128, or 256 x 256 for the token Gram of long rows) per
// 256-thread workgroup, 4 waves in a 2 x 2 grid, each (BM/2) x (BN/2) = (BM/64) x (BN/64)
// MFMA blocks; K tiles of 64.  Operands go global -> registers ->
// LDS; the next K tile's loads are issued before the current tile is multiplied and their
// registers are only read when they are stored to LDS, so the loads stay in flight during
// the MFMAs.  With two LDS buffers (see Lds for when) the next tile is stored into the
// second buffer while the first is multiplied, with one barrier per step.  LDS keeps both
// operands k-contiguous (rows of 64 + 8 bf16: conflict-free 16-byte fragment reads); an
// operand whose memory layout is contiguous along M/N is transposed in registers (each
// thread moves a 4 (k) x 8 (m) block; 16 lanes write one LDS row as 8-byte runs).
//
// Work decomposition: a 1-D grid over all tiles of all problems.  The hardware deals
// workgroups to the 8 XCDs round-robin; the kernel remaps its block index so that each XCD
// takes a contiguous run of tiles (ordered in groups of 8 tile rows), so tiles that share
// operand panels run on the same XCD and share its L2.
//
// Full K tiles load through per-thread 32-bit offsets fixed at the start, without bounds
// checks: rows (or column runs) beyond the operand's extent read a clamped in-range address
// and only feed outputs the epilogue does not store.  A ragged last K tile is loaded with
// every element checked (zeros beyond K).  gemm16_prepare() checks on the host that a
// table meets the layout conditions this needs; otherwise the caller uses the fp32 kernel.
#include "common.h"
#include "kernels.h"
#include <algorithm>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace {

constexpr int BK = 64, NT = 256, LDK = BK + 8;
constexpr int LDS_BYTES = 160 * 1024;

struct Grid {
  int tiles_m, tiles_n, per_prob, lower_only;
  int total, per_xcd;
  int wide;                 // lower-triangle tables with 256-row tiles (two tile columns per row)
};

JOLT_DEV int64_t opoff(const GemmOperand &op, int row, int col) {
  return (int64_t)row * op.ld + operand_col(op, col);
}

JOLT_DEV void split_bf16(float x, uint16_t &h, uint16_t &l) {
  h = f32_to_bf16(x);
  l = f32_to_bf16(x - bf16_to_f32(h));
}

// 8 elements as loaded: bf16 bits in four 32-bit words, or two float4
template <bool F32> struct Vec8 { ju4 w; };
template <> struct Vec8<true> { jf4 a, b; };

template <bool F32>
JOLT_DEV void load8(const GemmOperand &op, int row, int col, int nrows, int ncols, Vec8<F32> &v) {
  const bool in = row < nrows && col + 8 <= ncols;
  const int64_t o = in ? opoff(op, row, col) : 0;
  if constexpr (F32) {
    const float *p = reinterpret_cast<const float *>(op.ptr) + o;
    if (in && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      v.a = gload_f4(p); v.b = gload_f4(p + 4);
    } else {
      float f[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        f[i] = (row < nrows && col + i < ncols)
                   ? gptr(reinterpret_cast<const float *>(op.ptr))[opoff(op, row, col + i)] : 0.f;
      v.a = jf4{f[0], f[1], f[2], f[3]}; v.b = jf4{f[4], f[5], f[6], f[7]};
    }
  } else {
    const uint16_t *p = reinterpret_cast<const uint16_t *>(op.ptr) + o;
    if (in && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      v.w = gload_u4(p);
    } else {
      uint32_t h[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        h[i] = (row < nrows && col + i < ncols)
                   ? gptr(reinterpret_cast<const uint16_t *>(op.ptr))[opoff(op, row, col + i)] : 0u;
      v.w = ju4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
    }
  }
}

JOLT_DEV uint32_t pk(uint16_t a, uint16_t b) { return (uint32_t)a | ((uint32_t)b << 16); }

// Staging of one R (m or n) x 64 (k) operand tile through registers.
//   k-contiguous: unit u = tid + 256 q: row u / 8, k run (u % 8) * 8 (8 lanes per 128-byte row);
//   mn-contiguous: 4 (k) x 8 (mn) blocks b = tid + 256 p: k block b % 16, mn block b / 16, so
//   16 lanes write one LDS row's 64 k values as consecutive 8-byte runs.
// Full K tiles use precomputed per-thread offsets and branch-free loads (rows or columns
// beyond the operand's extent are read at a clamped in-range address and zeroed); a ragged
// last K tile goes through the bounds-checked load8.
template <int R, bool KC, bool F32>
struct Stage {
  static constexpr int NV = R * BK / 8 / NT;   // 8-element vectors per thread
  Vec8<F32> v[NV];
};

template <int R, bool KC, bool F32>
struct Addr {
  static constexpr int NV = R * BK / 8 / NT;
  uint32_t off[NV];     // element offset at k0 = 0 (KC: without the k column part)

  // Rows (KC) or column runs (mn-contiguous) beyond the operand's extent are read at a
  // clamped in-range address and not zeroed: they only feed output rows / columns that the
  // epilogue does not store.
  JOLT_DEV void init(const GemmOperand &op, int mn0, int MN, int tid) {
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      if constexpr (KC) {
        const int u = tid + NT * q, r = mn0 + (u >> 3), kc = (u & 7) * 8;
        off[q] = (uint32_t)((r < MN ? r : 0) * op.ld + kc);
      } else {
        const int b = tid + NT * (q >> 2), kb = (b & 15) * 4 + (q & 3), mb = mn0 + (b >> 4) * 8;
        off[q] = (uint32_t)(kb * op.ld + operand_col(op, mb < MN ? mb : 0));
      }
    }
  }

  // full K tile at k0 (k0 + 64 <= K); the raw registers are only read by stash, so the
  // loads stay in flight while earlier tiles are multiplied
  JOLT_DEV void fetch_full(const GemmOperand &op, int k0, Stage<R, KC, F32> &s) const {
    int64_t step;
    if constexpr (KC) step = operand_col(op, k0);      // a 64-wide k run stays in one segment
    else step = (int64_t)k0 * op.ld;
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      const int64_t o = (int64_t)off[q] + step;
      if constexpr (F32) {
        const float *p = reinterpret_cast<const float *>(op.ptr) + o;
        s.v[q].a = gload_f4(p); s.v[q].b = gload_f4(p + 4);
      } else {
        s.v[q].w = gload_u4(reinterpret_cast<const uint16_t *>(op.ptr) + o);
      }
    }
  }

  // ragged K tile: every element bounds-checked
  JOLT_DEV void fetch_tail(const GemmOperand &op, int mn0, int k0, int MN, int K, int tid,
                           Stage<R, KC, F32> &s) const {
#pragma unroll
    for (int q = 0; q < NV; ++q) {
      if constexpr (KC) {
        const int u = tid + NT * q, r = u >> 3, kc = (u & 7) * 8;
        load8<F32>(op, mn0 + r, k0 + kc, MN, K, s.v[q]);
      } else {
        const int b = tid + NT * (q >> 2), kb = (b & 15) * 4 + (q & 3), mb = (b >> 4) * 8;
        load8<F32>(op, k0 + kb, mn0 + mb, K, MN, s.v[q]);
      }
    }
  }

  JOLT_DEV float elem_f(const Stage<R, KC, F32> &s, int q, int e) const {
    return e < 4 ? s.v[q].a[e] : s.v[q].b[e - 4];
  }
  JOLT_DEV uint16_t elem_h(const Stage<R, KC, F32> &s, int q, int e) const {
    return (uint16_t)(s.v[q].w[e >> 1] >> (16 * (e & 1)));
  }

  JOLT_DEV void stash(const Stage<R, KC, F32> &s, uint16_t *hi, uint16_t *lo, int tid) const {
    if constexpr (KC) {
#pragma unroll
      for (int q = 0; q < NV; ++q) {
        const int u = tid + NT * q, r = u >> 3, kc = (u & 7) * 8;
        uint16_t h[8], l[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if constexpr (F32) split_bf16(elem_f(s, q, i), h[i], l[i]);
          else h[i] = elem_h(s, q, i);
        }
        *reinterpret_cast<uint4 *>(hi + r * LDK + kc) = make_uint4(pk(h[0], h[1]), pk(h[2], h[3]), pk(h[4], h[5]), pk(h[6], h[7]));
        if constexpr (F32)
          *reinterpret_cast<uint4 *>(lo + r * LDK + kc) = make_uint4(pk(l[0], l[1]), pk(l[2], l[3]), pk(l[4], l[5]), pk(l[6], l[7]));
      }
    } else {
#pragma unroll
      for (int p = 0; p < NV / 4; ++p) {
        const int b = tid + NT * p, kb = (b & 15) * 4, mb = (b >> 4) * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint16_t h[4], l[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if constexpr (F32) split_bf16(elem_f(s, 4 * p + q, e), h[q], l[q]);
            else h[q] = elem_h(s, 4 * p + q, e);
          }
          *reinterpret_cast<uint2 *>(hi + (mb + e) * LDK + kb) = make_uint2(pk(h[0], h[1]), pk(h[2], h[3]));
          if constexpr (F32)
            *reinterpret_cast<uint2 *>(lo + (mb + e) * LDK + kb) = make_uint2(pk(l[0], l[1]), pk(l[2], l[3]));
        }
      }
    }
  }
};

// Two LDS buffers are used when they fit in half the LDS (two workgroups per CU), or, for
// the 256-row tiles, in all of it: one workgroup per CU with double buffering measured
// faster than two single-buffered ones there, slower for the 128-row split-operand tiles.
template <int BM, int BN, bool AS, bool BS>
struct Lds {
  static constexpr int LA = BM * LDK * (AS ? 2 : 1), LB = BN * LDK * (BS ? 2 : 1);
  static constexpr bool DB = 2 * 2 * (LA + LB) <= (BM == 256 ? LDS_BYTES : LDS_BYTES / 2);
  uint16_t a[LA * (DB ? 2 : 1)];
  uint16_t b[LB * (DB ? 2 : 1)];
};

// tile of work item j (after the XCD remap): problem, tile row, tile column
JOLT_DEV bool decode(const Grid &g, int j, int &z, int &tm, int &tn) {
  if (j >= g.total) return false;
  z = j / g.per_prob;
  int r = j - z * g.per_prob;
  if (g.lower_only && g.wide) {
    // 256 x 128 tiles: row tm holds the 2 tm + 2 tiles tn <= 2 tm + 1 (the last row may
    // hold fewer), so the r-th lower tile has tm (tm + 1) <= r
    int t = (int)((sqrtf(4.f * (float)r + 1.f) - 1.f) * 0.5f);
    while ((t + 1) * (t + 2) <= r) ++t;
    while (t * (t + 1) > r) --t;
    tm = t; tn = r - t * (t + 1);
  } else if (g.lower_only) {
    // r-th lower tile in row-major order: tm (tm + 1) / 2 <= r
    int t = (int)((sqrtf(8.f * (float)r + 1.f) - 1.f) * 0.5f);
    while ((t + 1) * (t + 2) / 2 <= r) ++t;
    while (t * (t + 1) / 2 > r) --t;
    tm = t; tn = r - t * (t + 1) / 2;
  } else {
    // groups of 8 tile rows, column-major inside a group
    constexpr int GR = 8;
    const int gsz = GR * g.tiles_n, grp = r / gsz, in = r - grp * gsz;
    const int rows = min(GR, g.tiles_m - grp * GR);
    tm = grp * GR + in % rows; tn = in / rows;
  }
  return true;
}

// Epilogue of a BM x BN tile through LDS (cs, at least 32 (BN + 4) floats; every wave has
// finished with the operand buffers when it is called), 32 rows per round:
// acc[a][b][q] is the output at row wm*(BM/2) + a*32 + 8*(q/4) + 4*lh + q%4, column
// wn*(BN/2) + b*32 + lr of the tile.
template <int BM, int BN>
JOLT_DEV void store_tile(const GemmProblem &P, f32x16_t (&acc)[BM / 64][BN / 64], float *cs, int m0, int n0) {
  constexpr int MI = BM / 64, NI = BN / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, lr = lane & 31, lh = lane >> 5;
  // alpha 2^e is applied as ldexp(alpha * acc, e): 2^e alone may lie outside fp32's range
  const float alpha = P.alpha;
  const int aexp = P.alpha_exp2 ? (int)*gptr(P.alpha_exp2) : 0;
  constexpr int CLD = BN + 4;
  const bool use_beta = P.beta != 0.f;
  const bool ct = P.c_trans != 0;   // store the transpose: C[col * ldc + row]
  const bool vec = ((reinterpret_cast<uintptr_t>(P.C) & 15) == 0) && (P.ldc % 4 == 0);
#pragma unroll
  for (int h = 0; h < BM / 32; ++h) {
    __syncthreads();
    if (wm == h / MI) {
      const int a = h % MI;
#pragma unroll
      for (int b = 0; b < NI; ++b)
#pragma unroll
        for (int q = 0; q < 16; ++q)
          cs[(8 * (q >> 2) + 4 * lh + (q & 3)) * CLD + wn * (BN / 2) + b * 32 + lr] = acc[a][b][q];
    }
    __syncthreads();
    // 32 rows x BN columns in runs of 4 (along the row, or along the column for C^T)
#pragma unroll
    for (int u = 0; u < 8 * BN / NT; ++u) {
      const int idx = tid + u * NT;
      int rr, cc;
      if (ct) { cc = idx >> 3; rr = (idx & 7) * 4; }
      else { rr = idx / (BN / 4); cc = (idx % (BN / 4)) * 4; }
      const int row = m0 + h * 32 + rr, col = n0 + cc;
      if (ct) {
        if (col >= P.N || row >= P.M) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = ldexpf(alpha * cs[(rr + e) * CLD + cc], aexp);
        JOLT_GLOBAL float *dst = gptr(P.C + (int64_t)col * P.ldc + row);
        if (vec && row + 4 <= P.M) {
          if (use_beta) {
            const jf4 o4 = *reinterpret_cast<const JOLT_GLOBAL jf4 *>(dst);
            v[0] = fmaf(P.beta, o4.x, v[0]); v[1] = fmaf(P.beta, o4.y, v[1]);
            v[2] = fmaf(P.beta, o4.z, v[2]); v[3] = fmaf(P.beta, o4.w, v[3]);
          }
          *reinterpret_cast<JOLT_GLOBAL jf4 *>(dst) = jf4{v[0], v[1], v[2], v[3]};
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (row + e < P.M) dst[e] = use_beta ? fmaf(P.beta, dst[e], v[e]) : v[e];
        }
      } else {
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
}

// BM x BN tile per 256-thread workgroup; waves in a 2 x 2 grid, each (BM/2) x (BN/2).
template <int BM, int BN, bool AK, bool BK_, bool AS, bool BS>
__global__ void __launch_bounds__(NT) k_gemm16(const GemmProblem *__restrict__ probs, Grid g) {
  // blocks are dealt to the 8 XCDs round-robin; give each XCD a contiguous run of tiles
  const int i = blockIdx.x, j = (i & 7) * g.per_xcd + (i >> 3);
  int z, tm, tn;
  if (!decode(g, j, z, tm, tn)) return;
  const GemmProblem P = probs[z];
  if (tm * BM >= P.M || tn * BN >= P.N) return;
  constexpr int MI = BM / 64, NI = BN / 64;      // 32-row / 32-column MFMA blocks per wave
  __shared__ __attribute__((aligned(16))) Lds<BM, BN, AS, BS> sm;
  constexpr int TA = BM * LDK, TB = BN * LDK;
  constexpr int LA = Lds<BM, BN, AS, BS>::LA, LB = Lds<BM, BN, AS, BS>::LB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, lr = lane & 31, lh = lane >> 5;
  const int m0 = tm * BM, n0 = tn * BN;

  f32x16_t acc[MI][NI];
#pragma unroll
  for (int a = 0; a < MI; ++a)
#pragma unroll
    for (int b = 0; b < NI; ++b)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[a][b][q] = 0.f;

  constexpr int NS = 1;   // register stages (a deeper prefetch measured no faster)
  Addr<BM, AK, AS> ad_a;
  Addr<BN, BK_, BS> ad_b;
  Stage<BM, AK, AS> sa[NS];
  Stage<BN, BK_, BS> sb[NS];
  ad_a.init(P.A, m0, P.M, tid);
  ad_b.init(P.B, n0, P.N, tid);
  const int kfull = P.K & ~(BK - 1);
#define MM_FETCH(s, k) do { const int k_ = (k); \
    if (k_ < kfull) { ad_a.fetch_full(P.A, k_, sa[s]); ad_b.fetch_full(P.B, k_, sb[s]); } } while (0)
  auto compute_at = [&](int buf) {
    const uint16_t *la_ = sm.a + buf * LA, *lb_ = sm.b + buf * LB;
    // 16-wide k steps; with 256 x 256 tiles they are not unrolled, so that the fragments of
    // one step only are live beside the 256 accumulator registers
#pragma unroll (BN == 256 ? 1 : BK / 16)
    for (int s = 0; s < BK / 16; ++s) {
      const int ko = s * 16 + 8 * lh;
      bf16x8_t fa[MI], fb[NI], la[MI], lb[NI];
#pragma unroll
      for (int a = 0; a < MI; ++a) {
        const int ra = (wm * (BM / 2) + a * 32 + lr) * LDK + ko;
        fa[a] = *reinterpret_cast<const bf16x8_t *>(la_ + ra);
        if constexpr (AS) la[a] = *reinterpret_cast<const bf16x8_t *>(la_ + TA + ra);
      }
#pragma unroll
      for (int b = 0; b < NI; ++b) {
        const int rb = (wn * (BN / 2) + b * 32 + lr) * LDK + ko;
        fb[b] = *reinterpret_cast<const bf16x8_t *>(lb_ + rb);
        if constexpr (BS) lb[b] = *reinterpret_cast<const bf16x8_t *>(lb_ + TB + rb);
      }
#pragma unroll
      for (int a = 0; a < MI; ++a)
#pragma unroll
        for (int b = 0; b < NI; ++b) {
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b], acc[a][b], 0, 0, 0);
          if constexpr (AS) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(la[a], fb[b], acc[a][b], 0, 0, 0);
          if constexpr (BS) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], lb[b], acc[a][b], 0, 0, 0);
        }
    }
  };
  if constexpr (Lds<BM, BN, AS, BS>::DB) {
  // two LDS buffers: tile k+1 is stored into one while tile k is multiplied out of the
  // other; one barrier per step
  
  int cur = 0;
  if (kfull > 0) {
    MM_FETCH(0, 0);
    ad_a.stash(sa[0], sm.a, sm.a + TA, tid);
    ad_b.stash(sb[0], sm.b, sm.b + TB, tid);
    MM_FETCH(0, BK);
    __syncthreads();
  }
  for (int k0 = 0; k0 < kfull; k0 += BK) {
    compute_at(cur);
    if (k0 + BK < kfull) {
      ad_a.stash(sa[0], sm.a + (cur ^ 1) * LA, sm.a + (cur ^ 1) * LA + TA, tid);
      ad_b.stash(sb[0], sm.b + (cur ^ 1) * LB, sm.b + (cur ^ 1) * LB + TB, tid);
      MM_FETCH(0, k0 + 2 * BK);
    }
    __syncthreads();
    cur ^= 1;
  }
  } else {
#pragma unroll
  for (int s = 0; s < NS; ++s) MM_FETCH(s, s * BK);
  for (int k0 = 0; k0 < kfull; k0 += NS * BK) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (k0 + s * BK >= kfull) break;
      __syncthreads();
      ad_a.stash(sa[s], sm.a, sm.a + TA, tid);
      ad_b.stash(sb[s], sm.b, sm.b + TB, tid);
      __syncthreads();
      MM_FETCH(s, k0 + (s + NS) * BK);
      compute_at(0);
    }
  }
  }
#undef MM_FETCH
  if (kfull < P.K) {            // ragged last K tile, every element bounds-checked
    ad_a.fetch_tail(P.A, m0, kfull, P.M, P.K, tid, sa[0]);
    ad_b.fetch_tail(P.B, n0, kfull, P.N, P.K, tid, sb[0]);
    __syncthreads();
    ad_a.stash(sa[0], sm.a, sm.a + TA, tid);
    ad_b.stash(sb[0], sm.b, sm.b + TB, tid);
    __syncthreads();
    compute_at(0);
  }

  static_assert(32 * (BN + 4) * sizeof(float) <= sizeof(Lds<BM, BN, AS, BS>), "epilogue tile exceeds LDS");
  store_tile<BM, BN>(P, acc, reinterpret_cast<float *>(&sm), m0, n0);
}

// 256 x 256 tiles for bf16 x bf16 products whose operands are both k-contiguous and whose
// K is a multiple of 64 (the token Gram of wide cells).  Operand tiles go from global
// memory straight into LDS (global_load_lds_dwordx4: the 16 bytes of lane L land at the
// instruction's LDS base + 16 L), so no registers hold them on the way and no vector work
// repacks them.  An LDS row is one tile row's 64 k (128 bytes, unpadded) with its 16-byte
// chunks permuted by row (chunk c of row r at position c ^ f(r), f(r) = (r & 7) ^ ((r >> 3)
// & 1)), so that the fragment reads of any 8 consecutive rows, and of the even and of the odd
// rows among 16, fall in distinct banks; lane L of a load instruction therefore fetches chunk
// (L % 8) ^ f(r) of row r = (its 8-row group) + L / 8.  Two buffers: tile
// k + 1 streams in while tile k is multiplied; the fragments of the next 16-wide k step
// are read while the current one is multiplied.
constexpr int SQ = 256, SQ_ROWB = BK * 2;             // tile rows, bytes per LDS row
struct SqLds {
  uint8_t a[2][SQ * SQ_ROWB], b[2][SQ * SQ_ROWB];     // 128 KB
};

JOLT_DEV void lds_dma16(const void *src, uint8_t *lds_row_base) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src,
                                   (__attribute__((address_space(3))) void *)lds_row_base, 16, 0, 0);
}

__global__ void __launch_bounds__(NT) k_gemm16_sq(const GemmProblem *__restrict__ probs, Grid g) {
  const int i = blockIdx.x, j = (i & 7) * g.per_xcd + (i >> 3);
  int z, tm, tn;
  if (!decode(g, j, z, tm, tn)) return;
  const GemmProblem P = probs[z];
  if (tm * SQ >= P.M || tn * SQ >= P.N) return;
  constexpr int MI = 4, NI = 4, NQ = SQ / 8 / 4;      // load instructions per wave and operand
  __shared__ __attribute__((aligned(16))) SqLds sm;
  static_assert(32 * (SQ + 4) * sizeof(float) <= sizeof(SqLds), "epilogue tile exceeds LDS");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, lr = lane & 31, lh = lane >> 5;
  const int m0 = tm * SQ, n0 = tn * SQ;

  f32x16_t acc[MI][NI];
#pragma unroll
  for (int a = 0; a < MI; ++a)
#pragma unroll
    for (int b = 0; b < NI; ++b)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[a][b][q] = 0.f;

  // byte offsets of this lane's chunk in instruction q (rows past the extent read row 0 of
  // the operand and only feed outputs the epilogue does not store)
  uint32_t offa[NQ], offb[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int r = 8 * (NQ * wave + q) + (lane >> 3), c = (lane & 7) ^ (r & 7) ^ ((r >> 3) & 1);
    const int ra = m0 + r, rb = n0 + r;
    offa[q] = 2u * (uint32_t)((ra < P.M ? ra : 0) * P.A.ld + 8 * c);
    offb[q] = 2u * (uint32_t)((rb < P.N ? rb : 0) * P.B.ld + 8 * c);
  }
  auto dma = [&](int buf, int k0) {
    const char *pa = reinterpret_cast<const char *>(P.A.ptr) + 2 * operand_col(P.A, k0);
    const char *pb = reinterpret_cast<const char *>(P.B.ptr) + 2 * operand_col(P.B, k0);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      lds_dma16(pa + offa[q], sm.a[buf] + 8 * (NQ * wave + q) * SQ_ROWB);
      lds_dma16(pb + offb[q], sm.b[buf] + 8 * (NQ * wave + q) * SQ_ROWB);
    }
  };
  const int nk = P.K / BK, x = (lr & 7) ^ ((lr >> 3) & 1);
  bf16x8_t fa[2][MI], fb[2][NI];
  const uint8_t *la = sm.a[0], *lb = sm.b[0];
  auto frag = [&](int s, int set) {
    const int ch = ((2 * s + lh) ^ x) * 16;
#pragma unroll
    for (int a = 0; a < MI; ++a) fa[set][a] = *reinterpret_cast<const bf16x8_t *>(la + a * 32 * SQ_ROWB + ch);
#pragma unroll
    for (int b = 0; b < NI; ++b) fb[set][b] = *reinterpret_cast<const bf16x8_t *>(lb + b * 32 * SQ_ROWB + ch);
  };
  auto frag0 = [&](int buf) {
    la = sm.a[buf] + (wm * (SQ / 2) + lr) * SQ_ROWB;
    lb = sm.b[buf] + (wn * (SQ / 2) + lr) * SQ_ROWB;
    frag(0, 0);
  };
  auto compute = [&](int buf) {
    (void)buf;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      // the next step's 8 fragment reads go out between this step's 16 products, one after
      // every second product (scheduling groups; the barriers keep each step's region apart)
      if (s + 1 < BK / 16) frag(s + 1, (s + 1) & 1);
#pragma unroll
      for (int a = 0; a < MI; ++a)
#pragma unroll
        for (int b = 0; b < NI; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s & 1][a], fb[s & 1][b], acc[a][b], 0, 0, 0);
      if (s + 1 < BK / 16) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  if (nk > 0) dma(0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    // this wave's loads of tile kt have landed; the barrier then covers every wave's, and
    // every wave has finished reading the other buffer (tile kt - 1)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    // the first step's fragment reads go out before the next tile's loads are issued
    frag0(cur);
    __builtin_amdgcn_sched_barrier(0);
    if (kt + 1 < nk) dma(cur ^ 1, (kt + 1) * BK);
    __builtin_amdgcn_sched_barrier(0);
    compute(cur);
  }
  __syncthreads();
  store_tile<SQ, SQ>(P, acc, reinterpret_cast<float *>(&sm), m0, n0);
}

// C = C + alpha A B for fp32 A (M x K) and B (K x N) stored mn-contiguous (the operands'
// rows run along M and N), K <= 64, lower tiles only: the rank-2k update of the blocked
// tridiagonalisation (A = [V W]^T, B = [W V]).  It runs on the bf16 matrix cores with each
// operand element split into three bf16 terms, x = h + m + l (h = bf16(x), m = bf16(x - h),
// l = bf16(x - h - m), so |x - h - m - l| <= 2^-27 |x|), keeping the six products of order
// at most 2^-18 (hh, hm, mh, hl, mm, lh): what is dropped stays below 2^-25 of each product,
// under fp32's own rounding of it.  128 x 128 tiles; K in halves of 32 through LDS (three
// planes per operand, k-contiguous rows of 32 + 8: 61 KB, two workgroups per CU), all
// operand loads issued at once; the epilogue requests the whole C tile before its first
// round.
constexpr int U3_BM = 128, U3_KH = 32, U3_LDK = U3_KH + 8;
struct U3Lds {
  uint16_t a[3][U3_BM * U3_LDK], b[3][U3_BM * U3_LDK];   // 61.4 KB
};

JOLT_DEV void split3_bf16(float x, uint16_t &h, uint16_t &m, uint16_t &l) {
  h = f32_to_bf16(x);
  const float r1 = x - bf16_to_f32(h);                   // exact
  m = f32_to_bf16(r1);
  l = f32_to_bf16(r1 - bf16_to_f32(m));                  // exact difference, rounded once
}

// the thread's 4 (k) x 8 (mn) block of an mn-contiguous operand, zero outside K x MN
JOLT_DEV void load_block_mn(const GemmOperand &op, int k0, int mn0, int K, int MN, bool vec, float (&v)[4][8]) {
  const float *base = reinterpret_cast<const float *>(op.ptr);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int k = k0 + kk;
    if (vec && k < K && mn0 + 8 <= MN) {
      const float *p = base + (int64_t)k * op.ld + mn0;
      const jf4 x0 = gload_f4(p), x1 = gload_f4(p + 4);
      v[kk][0] = x0.x; v[kk][1] = x0.y; v[kk][2] = x0.z; v[kk][3] = x0.w;
      v[kk][4] = x1.x; v[kk][5] = x1.y; v[kk][6] = x1.z; v[kk][7] = x1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        v[kk][e] = (k < K && mn0 + e < MN) ? gptr(base)[(int64_t)k * op.ld + mn0 + e] : 0.f;
    }
  }
}

JOLT_DEV void stash3(const float (&v)[4][8], uint16_t *p0, uint16_t *p1, uint16_t *p2, int mn, int kb) {
  // kb: the block's first k within the LDS half
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint16_t h[4], m[4], l[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) split3_bf16(v[kk][e], h[kk], m[kk], l[kk]);
    const int o = (mn + e) * U3_LDK + kb;
    *reinterpret_cast<uint2 *>(p0 + o) = make_uint2(pk(h[0], h[1]), pk(h[2], h[3]));
    *reinterpret_cast<uint2 *>(p1 + o) = make_uint2(pk(m[0], m[1]), pk(m[2], m[3]));
    *reinterpret_cast<uint2 *>(p2 + o) = make_uint2(pk(l[0], l[1]), pk(l[2], l[3]));
  }
}

__global__ void __launch_bounds__(NT, 2) k_update3(const GemmProblem *__restrict__ probs, Grid g) {
  const int i = blockIdx.x, j = (i & 7) * g.per_xcd + (i >> 3);
  int z, tm, tn;
  if (!decode(g, j, z, tm, tn)) return;
  const GemmProblem P = probs[z];
  if (tm * U3_BM >= P.M || tn * U3_BM >= P.N) return;
  __shared__ __attribute__((aligned(16))) U3Lds sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, lr = lane & 31, lh = lane >> 5;
  const int m0 = tm * U3_BM, n0 = tn * U3_BM, K = P.K;

  // operands: 4 (k) x 8 (mn) per thread, k = 4 (tid % 16) .., mn = 8 (tid / 16) ..
  const int kb = 4 * (tid & 15), mb = 8 * (tid >> 4);
  const bool avec = ((reinterpret_cast<uintptr_t>(P.A.ptr) & 15) == 0) && (P.A.ld % 4 == 0);
  const bool bvec = ((reinterpret_cast<uintptr_t>(P.B.ptr) & 15) == 0) && (P.B.ld % 4 == 0);
  float va[4][8], vb[4][8];
  load_block_mn(P.A, kb, m0 + mb, K, P.M, avec, va);
  load_block_mn(P.B, kb, n0 + mb, K, P.N, bvec, vb);

  f32x16_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[a][b][q] = 0.f;
  const int ks = (K + 15) / 16;
#pragma unroll
  for (int s = 0; s < BK / 16; ++s) {
    if (s >= ks) break;
    if ((s & 1) == 0) {
      // k half s / 2 to LDS (the threads whose block lies in it)
      if (s) __syncthreads();
      if ((kb >= U3_KH) == (s >= 2)) {
        stash3(va, sm.a[0], sm.a[1], sm.a[2], mb, kb % U3_KH);
        stash3(vb, sm.b[0], sm.b[1], sm.b[2], mb, kb % U3_KH);
      }
      __syncthreads();
    }
    const int ko = (s & 1) * 16 + 8 * lh;
    bf16x8_t fa[3][2], fb[3][2];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        fa[t][a] = *reinterpret_cast<const bf16x8_t *>(sm.a[t] + (wm * 64 + a * 32 + lr) * U3_LDK + ko);
        fb[t][a] = *reinterpret_cast<const bf16x8_t *>(sm.b[t] + (wn * 64 + a * 32 + lr) * U3_LDK + ko);
      }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        f32x16_t c = acc[a][b];
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[2][a], fb[0][b], c, 0, 0, 0);   // l h
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][a], fb[1][b], c, 0, 0, 0);   // m m
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][a], fb[2][b], c, 0, 0, 0);   // h l
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][a], fb[0][b], c, 0, 0, 0);   // m h
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][a], fb[1][b], c, 0, 0, 0);   // h m
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][a], fb[0][b], c, 0, 0, 0);   // h h
        acc[a][b] = c;
      }
  }

  // epilogue through LDS, 32 rows per round (acc[a][b][q] is the output at row
  // wm*64 + a*32 + 8*(q/4) + 4*lh + q%4, column wn*64 + b*32 + lr of the tile)
  // the C tile, all of it requested before the first round: round h, piece u covers row
  // h * 32 + idx / 32, columns 4 (idx % 32) .. + 3, idx = tid + 256 u
  const bool cvec = ((reinterpret_cast<uintptr_t>(P.C) & 15) == 0) && (P.ldc % 4 == 0);
  jf4 cin[4][4];
#pragma unroll
  for (int h = 0; h < 4; ++h)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + u * NT, row = m0 + h * 32 + (idx >> 5), col = n0 + (idx & 31) * 4;
      const JOLT_GLOBAL float *src = gptr(P.C + (int64_t)row * P.ldc + col);
      if (row < P.M && cvec && col + 4 <= P.N) {
        cin[h][u] = *reinterpret_cast<const JOLT_GLOBAL jf4 *>(src);
      } else {
        float t[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) t[e] = (row < P.M && col + e < P.N) ? src[e] : 0.f;
        cin[h][u] = jf4{t[0], t[1], t[2], t[3]};
      }
    }
  float *cs = reinterpret_cast<float *>(&sm);
  constexpr int CLD = U3_BM + 4;
  static_assert(32 * CLD * sizeof(float) <= sizeof(U3Lds), "epilogue tile exceeds LDS");
  const float alpha = P.alpha;
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    __syncthreads();
    if (wm == (h >> 1)) {
      const int a = h & 1;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int q = 0; q < 16; ++q)
          cs[(8 * (q >> 2) + 4 * lh + (q & 3)) * CLD + wn * 64 + b * 32 + lr] = acc[a][b][q];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + u * NT, rr = idx >> 5, cc = (idx & 31) * 4;
      const int row = m0 + h * 32 + rr, col = n0 + cc;
      if (row >= P.M || col >= P.N) continue;
      const float4 a4 = *reinterpret_cast<const float4 *>(&cs[rr * CLD + cc]);
      const jf4 o4 = cin[h][u];
      const float v[4] = {fmaf(alpha, a4.x, P.beta * o4.x), fmaf(alpha, a4.y, P.beta * o4.y),
                          fmaf(alpha, a4.z, P.beta * o4.z), fmaf(alpha, a4.w, P.beta * o4.w)};
      JOLT_GLOBAL float *dst = gptr(P.C + (int64_t)row * P.ldc + col);
      if (cvec && col + 4 <= P.N) {
        *reinterpret_cast<JOLT_GLOBAL jf4 *>(dst) = jf4{v[0], v[1], v[2], v[3]};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < P.N) dst[e] = v[e];
      }
    }
  }
}

template <int BM, bool AS, bool BS>
hipError_t launch_bm(const GemmProblem *probs, const Grid &g, bool ak, bool bk, hipStream_t st) {
  const dim3 grid(g.per_xcd * 8);
  if (ak && bk) hipLaunchKernelGGL((k_gemm16<BM, 128, true, true, AS, BS>), grid, dim3(NT), 0, st, probs, g);
  else if (ak) hipLaunchKernelGGL((k_gemm16<BM, 128, true, false, AS, BS>), grid, dim3(NT), 0, st, probs, g);
  else if (bk) hipLaunchKernelGGL((k_gemm16<BM, 128, false, true, AS, BS>), grid, dim3(NT), 0, st, probs, g);
  else hipLaunchKernelGGL((k_gemm16<BM, 128, false, false, AS, BS>), grid, dim3(NT), 0, st, probs, g);
  return hipGetLastError();
}

// largest element offset of an operand view of rows x cols (row-major over ld with segments)
int64_t max_offset(const GemmOperand &o, int64_t rows, int64_t cols) {
  if (rows <= 0 || cols <= 0) return 0;
  int64_t colmax = cols - 1;
  if (o.seg_len > 0) {
    const int64_t segs = (cols + o.seg_len - 1) / o.seg_len;
    int64_t best = 0;
    // the segment offset grows with both its quotient and remainder by seg_heads
    const int64_t hq = (segs - 1) / o.seg_heads, hr = std::min<int64_t>(segs - 1, o.seg_heads - 1);
    best = hq * o.seg_hi + hr * o.seg_lo + (o.seg_len - 1);
    colmax = best;
  }
  return (rows - 1) * o.ld + colmax;
}

// Layout conditions of the fast loads for one operand: 16-byte aligned vectors at every
// (row, 8-aligned column), 64-wide k runs inside one segment (k-contiguous), 8-wide
// column runs inside one segment and inside the row (mn-contiguous), 32-bit offsets.
bool operand_ok(const GemmOperand &o, bool kc, bool f32, int MN, int K) {
  const int esz = f32 ? 4 : 2, vec = 16 / esz;
  if (reinterpret_cast<uintptr_t>(o.ptr) % 16) return false;
  if (o.ld % vec) return false;
  if (o.seg_len > 0) {
    if (o.seg_hi % vec || o.seg_lo % vec) return false;
    if (kc ? (o.seg_len % BK) : (o.seg_len % 8)) return false;
  }
  const int64_t lim = (int64_t)1 << 31;
  if (kc) {
    // per-thread part: row * ld + (k run within the tile); the k column part is added
    // in 64 bits per step
    if ((int64_t)(MN - 1) * o.ld + BK >= lim) return false;
    if (o.seg_len == 0 && o.ld < K) return false;
  } else {
    // column runs may overhang MN by up to 7 elements inside the row's ld
    if (MN % 8 && o.seg_len == 0 && o.ld < ((MN + 7) / 8) * 8) return false;
    if ((int64_t)BK * o.ld + max_offset(o, 1, MN) >= lim) return false;
  }
  return true;
}

}  // namespace

bool gemm16_prepare(GemmProblem *probs, int n, int &ta, int &tb, bool &ak, bool &bk, int &bm) {
  if (n <= 0) return false;
  if ((ta != GT_BF16 && ta != GT_F32) || (tb != GT_BF16 && tb != GT_F32)) return false;
  // one fp32 operand is taken on the B side (its 128-wide tile keeps the split registers
  // small): swap the roles of A and B and store C^T
  const bool swap = ta == GT_F32 && tb == GT_BF16;
  for (int i = 0; i < n; ++i) {
    GemmProblem p = probs[i];
    if (p.c_trans) return false;
    if (swap) { std::swap(p.A, p.B); std::swap(p.M, p.N); p.c_trans = 1; }
    const bool a32 = (swap ? tb : ta) == GT_F32, b32 = (swap ? ta : tb) == GT_F32;
    const bool akc = swap ? bk : ak, bkc = swap ? ak : bk;
    if (!operand_ok(p.A, akc, a32, p.M, p.K) || !operand_ok(p.B, bkc, b32, p.N, p.K)) return false;
    if (p.c_trans && p.lower_only) return false;
  }
  for (int i = 1; i < n; ++i)
    if ((probs[i].lower_only != 0) != (probs[0].lower_only != 0)) return false;
  int maxM = 0, minK = 1 << 30;
  bool lower = false;
  for (int i = 0; i < n; ++i) {
    GemmProblem &p = probs[i];
    if (swap) { std::swap(p.A, p.B); std::swap(p.M, p.N); p.c_trans = 1; }
    maxM = std::max(maxM, p.M);
    minK = std::min(minK, p.K);
    lower = lower || p.lower_only;
  }
  if (swap) { std::swap(ta, tb); std::swap(ak, bk); }
  // 256-row tiles for split-operand products over long M whose bf16 operand is k-contiguous
  // (two LDS buffers still fit); 256 x 256 tiles for large lower-triangle bf16 tables with a
  // long K (the token Gram of wide cells: each K step moves 512 operand rows for 256 x 256
  // outputs, and each wave's 128 x 128 block reads 8 fragments per 16 MFMAs, where the
  // 128 x 128 tiles read 4 per 4 and leave the K loop bound by LDS bandwidth); 128 otherwise
  // (an m-contiguous bf16 operand is transposed on its way to LDS, and the 128-row tile
  // then runs two workgroups per CU; at K = 4096 the 128-row tiles also keep two
  // workgroups per CU busy and measured faster)
  const bool bf_both = ta == GT_BF16 && tb == GT_BF16 && ak && bk;
  bool k64 = true;
  for (int i = 0; i < n; ++i) k64 = k64 && probs[i].K % BK == 0;
  if (lower && bf_both && k64 && maxM >= 2048 && minK >= 16384) bm = GEMM16_SQUARE256;
  else bm = (tb == GT_F32 && ta == GT_BF16 && maxM >= 2048 && !lower && ak) ? 256 : 128;
  return true;
}

hipError_t launch_gemm16(const GemmProblem *probs_dev, int n_probs, int max_M, int max_N, int ta,
                         int tb, bool a_kcontig, bool b_kcontig, int bm, bool lower_only,
                         hipStream_t st) {
  if (n_probs <= 0 || max_M <= 0 || max_N <= 0) return hipSuccess;
  const bool as = ta == GT_F32, bs = tb == GT_F32;
  if ((ta != GT_BF16 && !as) || (tb != GT_BF16 && !bs)) return hipErrorInvalidValue;
  if (bm != 128 && bm != 256 && bm != GEMM16_SQUARE256) return hipErrorInvalidValue;
  if (lower_only && bm != 128 && (as || bs)) return hipErrorInvalidValue;
  const bool square = bm == GEMM16_SQUARE256;
  const int tm_rows = square ? 256 : bm, tn_cols = square ? 256 : 128;
  Grid g;
  g.tiles_m = (max_M + tm_rows - 1) / tm_rows;
  g.tiles_n = (max_N + tn_cols - 1) / tn_cols;
  g.lower_only = lower_only ? 1 : 0;
  g.wide = lower_only && bm == 256 ? 1 : 0;
  if (g.wide) {
    // rows of 2 tm + 2 tiles; the last row is cut to the tile columns that exist
    g.per_prob = g.tiles_m * (g.tiles_m + 1) - std::max(0, 2 * g.tiles_m - g.tiles_n);
  } else {
    g.per_prob = lower_only ? g.tiles_m * (g.tiles_m + 1) / 2 : g.tiles_m * g.tiles_n;
  }
  g.total = g.per_prob * n_probs;
  g.per_xcd = (g.total + 7) / 8;
  if (square) {
    // 256 x 256 tiles, bf16 x bf16 with both operands k-contiguous only
    if (as || bs || !a_kcontig || !b_kcontig) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_gemm16_sq, dim3(g.per_xcd * 8), dim3(NT), 0, st, probs_dev, g);
    return hipGetLastError();
  }
  if (bm == 256) {
    if (as && bs) return hipErrorInvalidValue;
    if (as) return launch_bm<256, true, false>(probs_dev, g, a_kcontig, b_kcontig, st);
    if (bs) return launch_bm<256, false, true>(probs_dev, g, a_kcontig, b_kcontig, st);
    return launch_bm<256, false, false>(probs_dev, g, a_kcontig, b_kcontig, st);
  }
  if (as && bs) return launch_bm<128, true, true>(probs_dev, g, a_kcontig, b_kcontig, st);
  if (as) return launch_bm<128, true, false>(probs_dev, g, a_kcontig, b_kcontig, st);
  if (bs) return launch_bm<128, false, true>(probs_dev, g, a_kcontig, b_kcontig, st);
  return launch_bm<128, false, false>(probs_dev, g, a_kcontig, b_kcontig, st);
}

hipError_t launch_update3(const GemmProblem *probs_dev, int n_probs, int max_MN, hipStream_t st) {
  if (n_probs <= 0 || max_MN <= 0) return hipSuccess;
  Grid g;
  g.tiles_m = g.tiles_n = (max_MN + U3_BM - 1) / U3_BM;
  g.lower_only = 1;
  g.wide = 0;
  g.per_prob = g.tiles_m * (g.tiles_m + 1) / 2;
  g.total = g.per_prob * n_probs;
  g.per_xcd = (g.total + 7) / 8;
  hipLaunchKernelGGL(k_update3, dim3(g.per_xcd * 8), dim3(NT), 0, st, probs_dev, g);
  return hipGetLastError();
}

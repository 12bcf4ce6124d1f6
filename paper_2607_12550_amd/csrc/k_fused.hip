// Reconstruction fused into the residual and decode passes (section 4: R = X - X~ with X~
// rebuilt from the stored factors; decoding adds the dequantised, unrotated residual back).
//
// For slice s of a cell, X~_s = U^_T W_s with W_s = 2^e_s G^_s U^_d^T (r_T x d).  A small
// GEMM forms W_s^T (d x r_T, fp32) in the workspace; k_w_prepare picks a power of two
// 2^k_s with max |W_s| 2^-k_s <= 2^14 and rewrites each entry in place as its fp16 hi and
// lo terms, so tiles only separate them.  The fused kernel then multiplies, per tile of
// 128 tokens x d features of one slice, on the fp16 matrix cores (v_mfma_f32_32x32x16_f16,
// fp32 accumulation):
//   * U^_T is an exact fp16 operand when the factors are stored in fp16; fp32 factors are
//     scaled by 2^6 and split into hi + lo fp16 terms;
//   * W_s 2^-k_s is split into hi + lo fp16 terms (hi = fp16(w), lo = fp16(w - hi)), so
//     |w - hi - lo| <= 2^-22 |w| for entries in the fp16 normal range;
//   * X~ = 2^(k_s - u) (U_hi (W_hi + W_lo) [+ U_lo W_hi]), u = 6 for split factors, else 0:
//     two MFMA passes per K step (three for fp32 factors), products exact in fp32.
// The accumulator tile goes through LDS, 64 rows at a time, to the row layout of the
// residual kernels (a feature row over d/8 lanes) and the epilogue finishes the row in
// registers:
//   residual: r = X - X~, rotate (FWHT), group max, fp16 scale, codes, pack;
//   decode:   dequantise, inverse rotation, + X~, optional RoPE, cast, store;
//   export:   X~ itself (fp32; the test hook of the closed loop).
// X~ never reaches HBM: per cache entry the residual pass reads the cache once and writes
// the codes and scales, the decode pass reads codes and scales and writes the output.
//
// Tiles: 128 tokens x d features of one slice per 256-thread workgroup, 4 waves in a
// WM x WN grid (2 x 2 for d >= 64), K = r_T in steps of 32 (zero-padded).  The 1-D grid
// is remapped so that each XCD takes a contiguous run of tiles, ordered cell, slice, token
// block: the token blocks of a slice share W_s, the slices of a cell share U^_T.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "rowops.h"

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace {
using namespace rowops;

constexpr int BT = 128, BK = 32, LDK = BK + 8, NT = 256;

constexpr int EH = 64;                                         // epilogue rows per half

template <int D, bool USPLIT>
struct FusedLds {
  static constexpr int A = BT * LDK, B = D * LDK;              // halves per operand term
  static constexpr int OPER = (USPLIT ? 2 : 1) * A + 2 * B;     // A hi [A lo] B hi B lo
  static constexpr int EPI = EH * (D + 4) * 2;                  // fp32 epilogue half, in halves
  static constexpr int HALVES = OPER > EPI ? OPER : EPI;
};

JOLT_DEV uint16_t h_bits(float x) {
  _Float16 h = (_Float16)x;
  uint16_t b;
  __builtin_memcpy(&b, &h, 2);
  return b;
}
JOLT_DEV float h_val(uint16_t b) {
  _Float16 h;
  __builtin_memcpy(&h, &b, 2);
  return (float)h;
}
// x = hi + lo, hi = fp16(x), lo = fp16(x - hi)
JOLT_DEV void split_f16(float x, uint16_t &hi, uint16_t &lo) {
  hi = h_bits(x);
  lo = h_bits(x - h_val(hi));
}
JOLT_DEV uint32_t pk2(uint16_t a, uint16_t b) { return (uint32_t)a | ((uint32_t)b << 16); }

// 8 consecutive operand values along k (k0 .. k0 + 7 of row `row`), fp32; zeros beyond
// the row count or beyond K.  Aligned full runs use 16-byte loads.
template <bool F32>
JOLT_DEV void load_run(const void *base, int64_t ld, int row, int rows, int k0, int K, float (&v)[8]) {
  if (row >= rows || k0 >= K) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
    return;
  }
  if constexpr (F32) {
    const float *p = reinterpret_cast<const float *>(base) + (int64_t)row * ld + k0;
    if (k0 + 8 <= K && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      const jf4 a = gload_f4(p), b = gload_f4(p + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = k0 + i < K ? gptr(p)[i] : 0.f;
    }
  } else {
    const uint16_t *p = reinterpret_cast<const uint16_t *>(base) + (int64_t)row * ld + k0;
    if (k0 + 8 <= K && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      const ju4 u = gload_u4(p);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[2 * i] = h_val((uint16_t)(w[i] & 0xffffu));
        v[2 * i + 1] = h_val((uint16_t)(w[i] >> 16));
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = k0 + i < K ? h_val(gptr(p)[i]) : 0.f;
    }
  }
}

// 8 cache entries of one row as loaded (converted to fp32 only when used)
template <typename T> struct Raw8;
template <> struct Raw8<bf16_t> { ju4 w; };
template <> struct Raw8<float> { jf4 a, b; };
JOLT_DEV void raw_load(const bf16_t *p, Raw8<bf16_t> &r) { r.w = gload_u4(p); }
JOLT_DEV void raw_load(const float *p, Raw8<float> &r) { r.a = gload_f4(p); r.b = gload_f4(p + 4); }
JOLT_DEV void raw_f32(const Raw8<bf16_t> &r, float (&v)[8]) {
  const uint32_t w[4] = {r.w.x, r.w.y, r.w.z, r.w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_to_f32((bf16_t)(w[i] & 0xffffu));
    v[2 * i + 1] = bf16_to_f32((bf16_t)(w[i] >> 16));
  }
}
JOLT_DEV void raw_f32(const Raw8<float> &r, float (&v)[8]) {
  v[0] = r.a.x; v[1] = r.a.y; v[2] = r.a.z; v[3] = r.a.w; v[4] = r.b.x; v[5] = r.b.y; v[6] = r.b.z; v[7] = r.b.w;
}
// the b-bit codes of 8 entries (LSB first) as loaded: b = 2, 4 or 8 bytes
typedef uint32_t ju2 __attribute__((ext_vector_type(2)));
JOLT_DEV ju2 codes_load(const uint8_t *codes, int64_t elem, int bits) {
  if (bits == 2) return ju2{(uint32_t)*gptr(reinterpret_cast<const uint16_t *>(codes + elem / 4)), 0u};
  if (bits == 4) return ju2{*gptr(reinterpret_cast<const uint32_t *>(codes + elem / 2)), 0u};
  return *gptr(reinterpret_cast<const ju2 *>(codes + elem));
}
JOLT_DEV void codes_unpack(ju2 w, int bits, uint32_t (&c)[8]) {
  if (bits == 8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c[i] = (w.x >> (8 * i)) & 255u;
      c[i + 4] = (w.y >> (8 * i)) & 255u;
    }
  } else {
    const uint32_t mask = (1u << bits) - 1u;
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = (w.x >> (bits * i)) & mask;
  }
}

// 8 fp16 values of a run (k0 .. k0 + 7 of row `row`) as raw bits; zeros past the row count
// or K (and for a partial run past K; `full` runs lie inside K)
JOLT_DEV ju4 load_run_h(const uint16_t *base, int64_t ld, int row, int rows, int k0, int K) {
  if (row >= rows || k0 >= K) return ju4{0u, 0u, 0u, 0u};
  const uint16_t *p = base + (int64_t)row * ld + k0;
  if (k0 + 8 <= K && (reinterpret_cast<uintptr_t>(p) & 15) == 0) return gload_u4(p);
  uint16_t h[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) h[i] = k0 + i < K ? gptr(p)[i] : (uint16_t)0;
  return ju4{pk2(h[0], h[1]), pk2(h[2], h[3]), pk2(h[4], h[5]), pk2(h[6], h[7])};
}

template <int D, int MODE, typename TIO, bool USPLIT, bool ROPE>
__global__ void __launch_bounds__(NT, 2) k_fused(FusedArgs a) {
  constexpr int WN = D >= 64 ? 2 : 1, WM = 4 / WN;
  constexpr int WR = BT / WM, WC = D / WN;          // wave tile
  constexpr int MI = WR / 32, NI = WC / 32;         // 32 x 32 MFMA blocks per wave
  constexpr int L = RowLayout<D>::L, R = RowLayout<D>::R;
  using Lds = FusedLds<D, USPLIT>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[Lds::HALVES];
  uint16_t *sa = lds, *sa_lo = lds + Lds::A, *sb = lds + (USPLIT ? 2 : 1) * Lds::A, *sb_lo = sb + Lds::B;

  // tile: XCD-contiguous order (cell, slice, token block)
  const int i = blockIdx.x, j = (i & 7) * a.per_xcd + (i >> 3);
  if (j >= a.total) return;
  const int per_cell = a.m * a.tiles_t;
  const int cell = j / per_cell, rem = j - cell * per_cell;
  const int s = rem / a.tiles_t, t0 = (rem - s * a.tiles_t) * BT;
  const FusedCell c = a.cells[cell];
  if (MODE == FUSED_RESIDUAL && c.bits == 0) return;
  const int rT = c.rT, T = a.T;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN, lr = lane & 31, lh = lane >> 5;

  // the epilogue's HBM operands (cache rows or codes and scales of the rows this lane
  // finishes) are requested first, so that their latency overlaps the reconstruction; those
  // of the second half after the first half is done.  Wave w finishes rows
  // h 64 + 16 w .. h 64 + 16 w + 15 of each half h, R at a time.
  constexpr int NPH = (EH / 4) / R;                 // epilogue passes per half
  const int row_in_wave = lane / L, lane_in_row = lane % L;
  const int64_t srow = (int64_t)(s / a.heads) * a.s_layer + (int64_t)(s % a.heads) * a.s_head;
  Raw8<TIO> px[MODE == FUSED_RESIDUAL ? NPH : 1];
  ju2 pcode[MODE == FUSED_DECODE ? NPH : 1];
  uint16_t pscale[MODE == FUSED_DECODE ? NPH : 1];
  auto prefetch = [&](int h) {
#pragma unroll
    for (int pp = 0; pp < NPH; ++pp) {
      const int t = t0 + h * EH + wave * (EH / 4) + pp * R + row_in_wave;
      if (t >= T) continue;
      const int64_t elem = ((int64_t)s * T + t) * D + lane_in_row * 8;
      if constexpr (MODE == FUSED_RESIDUAL)
        raw_load(reinterpret_cast<const TIO *>(c.x) + srow + (int64_t)t * a.s_tok + lane_in_row * 8, px[pp]);
      if constexpr (MODE == FUSED_DECODE) {
        if (c.bits) {
          pcode[pp] = codes_load(c.codes, elem, c.bits);
          pscale[pp] = *gptr(c.scales + elem / a.group);
        }
      }
    }
  };
  prefetch(0);
  float sgv[8];
  {
    const float *sg = a.signs + (int64_t)cell * D + lane_in_row * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) sgv[e] = sg[e];
  }

  f32x16_t acc[MI][NI];
#pragma unroll
  for (int x = 0; x < MI; ++x)
#pragma unroll
    for (int y = 0; y < NI; ++y)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[x][y][q] = 0.f;

  int ks = 0;                              // X~ = 2^(ks - u) acc, applied per value
  if (rT > 0) {
    ks = c.wexp[s];
    // W_s^T as prepared: per entry the fp16 pair (hi, lo), zeros past r_T
    const uint32_t *Wp = reinterpret_cast<const uint32_t *>(c.Wt + (int64_t)s * D * c.ldw);
    // operand units of 8 k values: A has BT rows x 4 units, B has D rows x 4 units
    constexpr int AU = BT * (BK / 8) / NT, BU = D * (BK / 8) / NT > 0 ? D * (BK / 8) / NT : 1;
    float ra[USPLIT ? AU : 1][8];
    ju4 rah[AU], rbh[BU], rbl[BU];
    auto fetch = [&](int k0) {
#pragma unroll
      for (int q = 0; q < AU; ++q) {
        const int u = tid + NT * q, r = u >> 2, kc = (u & 3) * 8;
        if constexpr (USPLIT) load_run<true>(c.UT, rT, t0 + r, T, k0 + kc, rT, ra[q]);
        else rah[q] = load_run_h(reinterpret_cast<const uint16_t *>(c.UT), rT, t0 + r, T, k0 + kc, rT);
      }
#pragma unroll
      for (int q = 0; q < BU; ++q) {
        const int u = tid + NT * q, r = u >> 2, kc = (u & 3) * 8;
        const bool in = u < D * (BK / 8) && k0 + kc < rT;   // runs past r_T are zero
        rbh[q] = in ? gload_u4(Wp + (int64_t)r * c.ldw + k0 + kc) : ju4{0u, 0u, 0u, 0u};
        rbl[q] = in ? gload_u4(Wp + (int64_t)r * c.ldw + k0 + kc + 4) : ju4{0u, 0u, 0u, 0u};
      }
    };
    auto stash = [&]() {
#pragma unroll
      for (int q = 0; q < AU; ++q) {
        const int u = tid + NT * q, r = u >> 2, kc = (u & 3) * 8;
        if constexpr (USPLIT) {
          uint16_t h[8], l[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) split_f16(ra[q][e] * 64.f, h[e], l[e]);
          *reinterpret_cast<uint4 *>(sa + r * LDK + kc) = make_uint4(pk2(h[0], h[1]), pk2(h[2], h[3]), pk2(h[4], h[5]), pk2(h[6], h[7]));
          *reinterpret_cast<uint4 *>(sa_lo + r * LDK + kc) = make_uint4(pk2(l[0], l[1]), pk2(l[2], l[3]), pk2(l[4], l[5]), pk2(l[6], l[7]));
        } else {
          *reinterpret_cast<ju4 *>(sa + r * LDK + kc) = rah[q];
        }
      }
#pragma unroll
      for (int q = 0; q < BU; ++q) {
        const int u = tid + NT * q, r = u >> 2, kc = (u & 3) * 8;
        if (u >= D * (BK / 8)) continue;
        // 8 (hi, lo) pairs -> 8 hi terms and 8 lo terms
        const uint32_t w[8] = {rbh[q].x, rbh[q].y, rbh[q].z, rbh[q].w, rbl[q].x, rbl[q].y, rbl[q].z, rbl[q].w};
        ju4 hv, lv;
        hv.x = __builtin_amdgcn_perm(w[1], w[0], 0x05040100u); lv.x = __builtin_amdgcn_perm(w[1], w[0], 0x07060302u);
        hv.y = __builtin_amdgcn_perm(w[3], w[2], 0x05040100u); lv.y = __builtin_amdgcn_perm(w[3], w[2], 0x07060302u);
        hv.z = __builtin_amdgcn_perm(w[5], w[4], 0x05040100u); lv.z = __builtin_amdgcn_perm(w[5], w[4], 0x07060302u);
        hv.w = __builtin_amdgcn_perm(w[7], w[6], 0x05040100u); lv.w = __builtin_amdgcn_perm(w[7], w[6], 0x07060302u);
        *reinterpret_cast<ju4 *>(sb + r * LDK + kc) = hv;
        *reinterpret_cast<ju4 *>(sb_lo + r * LDK + kc) = lv;
      }
    };
    fetch(0);
    for (int k0 = 0; k0 < rT; k0 += BK) {
      __syncthreads();                     // the previous step's fragments have been read
      stash();
      __syncthreads();
      if (k0 + BK < rT) fetch(k0 + BK);    // in flight during the MFMAs below
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ko = ks * 16 + 8 * lh;
        f16x8_t fa[MI], fl[MI], fb[NI], fbl[NI];
#pragma unroll
        for (int x = 0; x < MI; ++x) {
          const int ra_ = (wm * WR + x * 32 + lr) * LDK + ko;
          fa[x] = *reinterpret_cast<const f16x8_t *>(sa + ra_);
          if constexpr (USPLIT) fl[x] = *reinterpret_cast<const f16x8_t *>(sa_lo + ra_);
        }
#pragma unroll
        for (int y = 0; y < NI; ++y) {
          const int rb_ = (wn * WC + y * 32 + lr) * LDK + ko;
          fb[y] = *reinterpret_cast<const f16x8_t *>(sb + rb_);
          fbl[y] = *reinterpret_cast<const f16x8_t *>(sb_lo + rb_);
        }
#pragma unroll
        for (int x = 0; x < MI; ++x)
#pragma unroll
          for (int y = 0; y < NI; ++y) {
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[x], fb[y], acc[x][y], 0, 0, 0);
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[x], fbl[y], acc[x][y], 0, 0, 0);
            if constexpr (USPLIT)
              acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fl[x], fb[y], acc[x][y], 0, 0, 0);
          }
      }
    }
  }
  const int gl = a.group / 8;
  // accumulators -> LDS half tile [EH][D + 4] (fp32), half h holding tile rows h EH ..:
  // acc[x][y][q] is row wm WR + x 32 + 8 (q / 4) + 4 lh + q % 4, column wn WC + y 32 + lr
  constexpr int ELD = D + 4;
  float *E = reinterpret_cast<float *>(lds);
#pragma unroll
  for (int h = 0; h < BT / EH; ++h) {
    if (h > 0) prefetch(h);
    __syncthreads();                       // operand tiles, or the previous half, are read
#pragma unroll
    for (int x = 0; x < MI; ++x) {
#pragma unroll
      for (int y = 0; y < NI; ++y) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int row = wm * WR + x * 32 + 8 * (q >> 2) + 4 * lh + (q & 3) - h * EH;
          if (row >= 0 && row < EH) E[row * ELD + wn * WC + y * 32 + lr] = acc[x][y][q];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int pp = 0; pp < NPH; ++pp) {
      const int rr = wave * (EH / 4) + pp * R + row_in_wave, t = t0 + h * EH + rr;
      if (t >= T) continue;                // whole rows (L lanes) drop out together
      float xt[8];
      {
        const jf4 u0 = *reinterpret_cast<const jf4 *>(E + rr * ELD + lane_in_row * 8);
        const jf4 u1 = *reinterpret_cast<const jf4 *>(E + rr * ELD + lane_in_row * 8 + 4);
        xt[0] = u0.x; xt[1] = u0.y; xt[2] = u0.z; xt[3] = u0.w; xt[4] = u1.x; xt[5] = u1.y; xt[6] = u1.z; xt[7] = u1.w;
        const int xe = ks - (USPLIT ? 6 : 0);
#pragma unroll
        for (int e = 0; e < 8; ++e) xt[e] = rT > 0 ? ldexpf(xt[e], xe) : 0.f;   // exact
      }
      const int64_t elem = ((int64_t)s * T + t) * D + lane_in_row * 8;
      if constexpr (MODE == FUSED_XTILDE) {
        store8(c.xt_out + elem, xt);
      } else if constexpr (MODE == FUSED_RESIDUAL) {
        float v[8];
        raw_f32(px[pp], v);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (v[e] - xt[e]) * sgv[e];
        fwht_row<D>(v, lane_in_row);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] *= a.inv_sqrt_d;
        uint32_t code[8];
        float delta;
        quantize8(v, c.bits, gl, lane_in_row, code, delta);
        store_codes(c.codes, elem, c.bits, code);
        if ((lane_in_row % gl) == 0) c.scales[elem / a.group] = h_bits(delta);
      } else {
        float v[8];
        if (c.bits) {
          uint32_t code[8];
          codes_unpack(pcode[pp], c.bits, code);
          const float delta = h_val(pscale[pp]);
          const float mid = 0.5f * (float)((1 << c.bits) - 1);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = ((float)code[e] - mid) * delta;
          fwht_row<D>(v, lane_in_row);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = xt[e] + sgv[e] * (v[e] * a.inv_sqrt_d);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = xt[e];
        }
        if constexpr (ROPE) {
          double theta[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int jj = (lane_in_row * 8 + e) % (D / 2);
            theta[e] = exp2(-(2.0 * jj / D) * a.rope_log2_base);
          }
          rope_row<D>(v, lane_in_row, (double)(t + a.rope_offset), theta);
        }
        store8(reinterpret_cast<TIO *>(c.out) + srow + (int64_t)t * a.s_tok + lane_in_row * 8, v);
      }
    }
  }
}

// k_s of every (cell, slice): the smallest power of two with max |W_s| 2^-k_s <= 2^14
// (0 for an all-zero slice or a cell without backbone), then every entry of W_s^T up to
// column round8(r_T) rewritten in place as the pair (hi, lo) of fp16 terms of W 2^-k_s, hi in
// the low half-word (zeros from r_T on).  One workgroup per (slice, cell).
__global__ void __launch_bounds__(256) k_w_prepare(const FusedCell *cells, int m, int d) {
  const int s = blockIdx.x, cell = blockIdx.y;
  const FusedCell &c = cells[cell];
  if (s >= m || c.rT <= 0) return;
  float *W = c.Wt + (int64_t)s * d * c.ldw;
  // the columns the fused passes read, 0 .. round8(r_T) - 1 of each row (ldw may be far
  // wider), as d * n4 chunks of 4 entries, four chunks in flight per thread; chunk q is
  // row q / n4, entries 4 (q % n4) .. + 3
  const int n4 = ((c.rT + 7) / 8) * 2, nq = d * n4;
  const float inv_n4 = 1.f / (float)n4;
  auto row_of = [&](int q) {                      // exact q / n4 for q < 2^24
    int r = (int)((float)q * inv_n4);
    if (r * n4 > q) --r;
    if ((r + 1) * n4 <= q) ++r;
    return r;
  };
  auto addr = [&](int q) {                        // float offset of chunk q in the slice
    const int r = row_of(q);
    return (int64_t)r * c.ldw + 4 * (q - r * n4);
  };
  constexpr int U4 = 4;
  float mx = 0.f;
  for (int q0 = threadIdx.x; q0 < nq; q0 += 256 * U4) {
    jf4 v[U4];
#pragma unroll
    for (int u = 0; u < U4; ++u) {
      const int q = q0 + 256 * u;
      v[u] = q < nq ? gload_f4(W + addr(q)) : jf4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < U4; ++u) {
      const int q = q0 + 256 * u;
      const int k = 4 * (q - row_of(q) * n4);
      if (q < nq) {
        mx = fmaxf(mx, fmaxf(fmaxf(k < c.rT ? fabsf(v[u].x) : 0.f, k + 1 < c.rT ? fabsf(v[u].y) : 0.f),
                             fmaxf(k + 2 < c.rT ? fabsf(v[u].z) : 0.f, k + 3 < c.rT ? fabsf(v[u].w) : 0.f)));
      }
    }
  }
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  __shared__ float red[4];
  __shared__ int ks_s;
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    int e = 0;
    if (mx > 0.f) {
      int ex;
      const float f = frexpf(mx, &ex);            // mx = f 2^ex, 0.5 <= f < 1
      e = (f == 0.5f ? ex - 1 : ex) - 14;          // ceil(log2 mx) - 14
    }
    c.wexp[s] = e;
    ks_s = e;
  }
  __syncthreads();
  const int ks = ks_s;
  for (int q0 = threadIdx.x; q0 < nq; q0 += 256 * U4) {
    jf4 v[U4];
#pragma unroll
    for (int u = 0; u < U4; ++u) {
      const int q = q0 + 256 * u;
      v[u] = q < nq ? gload_f4(W + addr(q)) : jf4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < U4; ++u) {
      const int q = q0 + 256 * u;
      if (q >= nq) continue;
      const int k = 4 * (q - row_of(q) * n4);
      const float x[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint16_t hi = 0, lo = 0;
        if (k + e < c.rT) split_f16(ldexpf(x[e], -ks), hi, lo);
        o[e] = pk2(hi, lo);
      }
      *reinterpret_cast<ju4 *>(W + addr(q)) = ju4{o[0], o[1], o[2], o[3]};
    }
  }
}

// ------------------------------------------------------------------------- core path
// Factors stored in fp16 (the default) take the reconstruction in the other order,
// X~_s = 2^e_s (U^_T G^_s) U^_d^T, which costs 2 r_T r_d + 4 r_d d flops per token and slice
// instead of the 4 r_T d of U^_T W_s:
//   stage 1  Y_s^T = G^_s^T U^_T^T (r_d x tokens): fp16 operands as stored, products exact in
//            fp32, fp32 accumulation;
//   stage 2  X~_s^T 2^-(e_s + ky_s) = U^_d (Y_s^T 2^-ky_s): Y scaled by the power of two
//            2^-ky_s that bounds it by 2^15 (|Y| <= |U^_T row| |G^_s column| <=
//            1.01 sqrt(r_T) max|G^_s|) and split into fp16 hi + lo, two MFMA passes;
//            U^_d is an exact fp16 operand.
// k_core_prepare writes, per slice, G^_s^T zero-padded to RD = round32(r_d) rows of
// K16 = round16(r_T) entries (in the slice's W area) and ky_s (in the exponent array), and
// per cell U^_d with its columns permuted into the order of stage 2's k slots (below).
//
// Each wave owns 32 tokens of one slice (a workgroup 128 tokens, tiles ordered as in
// k_fused).  Stage 1's accumulator block b holds Y^T rows 32 b + 8 (q / 4) + 4 h + q % 4 for
// the lane's token (lane % 32) in its entry q, h = lane / 32; stage 2 takes entries
// q = 8 c .. 8 c + 7 of block b as the B operand of k chunk kc = 2 b + c, so U^_d's columns are
// permuted to match (slot s of lane half h is column 16 kc + 4 h + s % 4 + 8 (s / 4)).  Stage
// 2's accumulator leaves token t's row split over the lane pair (t, t + 32): lane half h
// holds features f = 8 u + 4 h + i for units u < d/8 and i < 4, value index 4 u + i.  The
// epilogue works in that layout: the Walsh-Hadamard transform runs log2(d) - 1 butterfly
// stages inside the lane and the stage of feature bit 2 across the pair (v_permlane32_swap);
// a quantiser group of g features is g/8 units of one lane plus the same units of the other.
constexpr int CORE_UDP_PAD = 8;                                 // halves per LDS row of U^_d

// Across the lane pair (l, l + 32): v_permlane32_swap of two copies of v leaves the lower
// lane's value in the first result and the upper lane's in the second, in both lanes.
// Butterfly: the lower lane gets v_lo + v_hi, the upper v_lo - v_hi (sgn = +1 / -1).
JOLT_DEV float pair_butterfly(float v, float sgn) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaf(sgn, __uint_as_float(r[1]), __uint_as_float(r[0]));
}
JOLT_DEV float pair_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__global__ void __launch_bounds__(256) k_core_prepare(const FusedCell *cells, const float *signs, int m, int d) {
  const int s = blockIdx.x, cell = blockIdx.y;
  const FusedCell &c = cells[cell];
  if (s >= m || c.rT <= 0) return;
  const int rT = c.rT, rd = c.rd, RD = (rd + 31) & ~31, K16 = (rT + 15) & ~15;
  const uint16_t *G = c.G + (int64_t)s * rT * rd;
  uint16_t *Gt = reinterpret_cast<uint16_t *>(c.Wt + (int64_t)s * d * c.ldw);
  __shared__ uint16_t tile[64][130];
  float mx = 0.f;
  for (int i0 = 0; i0 < K16; i0 += 64) {
    for (int q = threadIdx.x; q < 64 * RD; q += 256) {
      const int r = q / RD, j = q - r * RD, i = i0 + r;
      uint16_t v = 0;
      if (i < rT && j < rd) {
        v = G[(int64_t)i * rd + j];
        mx = fmaxf(mx, fabsf(h_val(v)));
      }
      tile[r][j] = v;
    }
    __syncthreads();
    for (int q = threadIdx.x; q < 64 * RD; q += 256) {
      const int j = q / 64, r = q - j * 64;
      if (i0 + r < K16) Gt[(int64_t)j * K16 + i0 + r] = tile[r][j];
    }
    __syncthreads();
  }
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    int e = 0;
    if (mx > 0.f) {
      const double bound = 1.01 * sqrt((double)rT) * (double)mx;
      int ex;
      const double f = frexp(bound, &ex);         // bound = f 2^ex, 0.5 <= f < 1
      e = (f == 0.5 ? ex - 1 : ex) - 15;          // ceil(log2 bound) - 15
    }
    c.wexp[s] = e;
  }
  if (s == 0) {
    // s_f U^_d[f, :] (d x r_d, fp16, rotation sign s_f folded in: an exact sign flip) with
    // columns in stage 2's slot order, zeros past r_d
    for (int q = threadIdx.x; q < d * RD; q += 256) {
      const int f = q / RD, p = q - f * RD;
      const int kc = p >> 4, hh = (p >> 3) & 1, sl = p & 7;
      const int jsrc = 16 * kc + 4 * hh + (sl & 3) + 8 * (sl >> 2);
      const uint16_t flip = signs[(int64_t)cell * d + f] < 0.f ? 0x8000u : 0u;
      c.udp[q] = jsrc < rd ? (uint16_t)(c.Ud[(int64_t)f * rd + jsrc] ^ flip) : (uint16_t)0;
    }
  }
}

JOLT_DEV f16x8_t as_f16x8(ju4 u) {
  f16x8_t r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}

// LDS of k_core: U^_d (permuted, rows padded), then one area shared in turn by the staged
// cache rows of the tile (residual input), the staged codes and scales (decode input), the
// K chunks of stage 1 (U^_T rows of the tile and G^_s^T rows, 32 k each, rows padded), and
// the staged output (codes, or decoded rows).  All global traffic of the tile is in
// 16-byte (cache rows, operands) or 4-byte (codes) pieces along contiguous memory.
template <int D, typename TIO>
struct CoreLds {
  static constexpr int LDU = D + CORE_UDP_PAD;                  // halves per U^_d row
  static constexpr int UD_BYTES = D * LDU * 2;
  static constexpr int LDK = 40;                                // halves per K-chunk row
  static constexpr int OPER = 2 * BT * LDK * 2;                 // U^_T chunk + G^T chunk
  static constexpr int IO_ROW = D * (int)sizeof(TIO) + 16;      // bytes per staged cache row
  static constexpr int IO = BT * IO_ROW;
  static constexpr int CODE_ROW = D + 4;                        // bytes per staged code row (max)
  static constexpr int CODES = BT * CODE_ROW + BT * (D / 8) * 2;
  static constexpr int SHARED = OPER > IO ? (OPER > CODES ? OPER : CODES) : (IO > CODES ? IO : CODES);
  static constexpr int BYTES = UD_BYTES + SHARED;
};

template <int D, int MODE, typename TIO, bool ROPE>
__global__ void __launch_bounds__(NT, sizeof(TIO) == 2 ? 2 : 1) k_core(FusedArgs a) {
  constexpr int FB = D / 32, NU = D / 8, NV = D / 2;     // feature blocks, units, values per lane
  using L = CoreLds<D, TIO>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[L::BYTES];
  uint16_t *sud = reinterpret_cast<uint16_t *>(smem);
  uint8_t *sh = smem + L::UD_BYTES;
  uint16_t *sU = reinterpret_cast<uint16_t *>(sh), *sG = sU + BT * L::LDK;

  const int bi = blockIdx.x, jt = (bi & 7) * a.per_xcd + (bi >> 3);
  if (jt >= a.total) return;
  const int per_cell = a.m * a.tiles_t;
  const int cell = jt / per_cell, rem = jt - cell * per_cell;
  const int s = rem / a.tiles_t, t0 = (rem - s * a.tiles_t) * BT;
  const FusedCell c = a.cells[cell];
  if (MODE == FUSED_RESIDUAL && c.bits == 0) return;
  const int T = a.T, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, tl = lane & 31, h = lane >> 5;
  const int trow = wave * 32 + tl;                         // tile row of this lane's token
  const int t = t0 + trow;
  const bool tin = t < T;
  const int tc = tin ? t : T - 1;
  const int nrows = T - t0 < BT ? T - t0 : BT;             // valid rows of the tile
  const int64_t srow = (int64_t)(s / a.heads) * a.s_layer + (int64_t)(s % a.heads) * a.s_head;
  const int64_t ebase = ((int64_t)s * T + tc) * D;         // element of (s, t, feature 0)
  const int bits = c.bits, g = a.group, gw = g / 8;
  const int rT = c.rT;
  const int ky = rT > 0 ? c.wexp[s] : 0;
  const int xe = rT > 0 ? ky + (int)c.gexp[s] : 0;         // X~ = 2^xe (stage-2 accumulator)
  const int RD = rT > 0 ? (c.rd + 31) & ~31 : 0;

  // U^_d in the permuted slot order to its LDS area (read after the next barrier)
  for (int q = tid; q < D * RD / 8; q += NT) {
    const int f = q / (RD / 8), p8 = q - f * (RD / 8);
    *reinterpret_cast<ju4 *>(sud + f * L::LDU + 8 * p8) = gload_u4(c.udp + (int64_t)f * RD + 8 * p8);
  }
  // stage-1 operands: U^_T rows of the tile and G^_s^T rows, K chunks of 32; each thread moves
  // two 16-byte pieces of each operand per chunk (128 rows x 4 pieces).  The first two
  // chunks are requested here, ahead of the epilogue operands.
  const int K16 = (rT + 15) & ~15, NB1 = RD / 32;
  const uint16_t *Gt = reinterpret_cast<const uint16_t *>(c.Wt + (int64_t)s * D * c.ldw);
  const uint16_t *UT = reinterpret_cast<const uint16_t *>(c.UT);
  const bool whole = (rT & 7) == 0;                         // U^_T rows 16-byte aligned
  ju4 pu[2][2], pg[2][2];
  auto fetch = [&](int sl, int k0) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int q = tid + NT * e, r = q >> 2, k = k0 + 8 * (q & 3);
      const int tr = t0 + r < T ? t0 + r : T - 1;
      if (whole) pu[sl][e] = k < rT ? gload_u4(UT + (int64_t)tr * rT + k) : ju4{0u, 0u, 0u, 0u};
      else pu[sl][e] = load_run_h(UT, rT, tr, T, k, rT);
      pg[sl][e] = r < RD && k < K16 ? gload_u4(Gt + (int64_t)r * K16 + k) : ju4{0u, 0u, 0u, 0u};
    }
  };
  if (rT > 0) {
    fetch(0, 0);
    if (32 < K16) fetch(1, 32);
  }
  const float *sgn = a.signs + (int64_t)cell * D;          // rotation signs s_f (+-1)
  const int rows_bytes = D * bits / 8, code_row = rows_bytes + 4;       // codes per row, staged
  const int lg = 31 - __builtin_clz(g), lgw = lg - 3;       // g and g / 8 are powers of two

  // U^_d carries the rotation signs (k_core_prepare), so stage 2 adds s * X~ 2^-xe to the
  // accumulator, which starts from (exact scaling):
  //   residual and export: zero, ending as s * X~ 2^-xe; the residual pass keeps -s * X of
  //             its entries in registers and forms -s * r = -s * X + s * X~ after the
  //             reconstruction, a subtraction of close fp32 values that is exact, so r
  //             carries the rounding of X~ only (the export mode returns the same X~);
  //   decode:   H r^ / sqrt(d) 2^-xe, so that it ends as s * X^ 2^-xe.
  // acc2[fb][q] is value 16 fb + q: unit 4 fb + q / 4, entry q % 4.
  f32x16_t acc2[FB];
#pragma unroll
  for (int fb = 0; fb < FB; ++fb)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc2[fb][q] = 0.f;
  // residual: -s * X of the lane's entries as loaded (bf16 pairs, or fp32 in two words)
  ju2 xw[MODE == FUSED_RESIDUAL ? NU : 1], xw2[MODE == FUSED_RESIDUAL && sizeof(TIO) == 4 ? NU : 1];
  if constexpr (MODE == FUSED_RESIDUAL) {
    // the tile's cache rows to LDS as -s * X: each thread moves the same 16-byte piece p of
    // several rows and flips the sign bits of its entries by a mask (-s_f < 0 sets the bit)
    constexpr int PR = D * (int)sizeof(TIO) / 16;           // 16-byte pieces per cache row
    static_assert(NT % PR == 0, "piece index fixed per thread");
    const int pp = tid % PR;
    ju4 flip;
    {
      uint32_t m4[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (sizeof(TIO) == 2) {
          const int f = 8 * pp + 2 * w;
          m4[w] = (sgn[f] > 0.f ? 0x8000u : 0u) | (sgn[f + 1] > 0.f ? 0x80000000u : 0u);
        } else {
          m4[w] = sgn[4 * pp + w] > 0.f ? 0x80000000u : 0u;
        }
      }
      flip = ju4{m4[0], m4[1], m4[2], m4[3]};
    }
    const uint8_t *xb = reinterpret_cast<const uint8_t *>(c.x);
    for (int r = tid / PR; r < BT; r += NT / PR) {
      const int tr = t0 + r < T ? t0 + r : T - 1;
      *reinterpret_cast<ju4 *>(sh + r * L::IO_ROW + 16 * pp) =
          gload_u4(xb + (srow + (int64_t)tr * a.s_tok) * (int64_t)sizeof(TIO) + 16 * pp) ^ flip;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const uint8_t *src = sh + trow * L::IO_ROW + (8 * u + 4 * h) * (int)sizeof(TIO);
      if constexpr (sizeof(TIO) == 2) {
        const uint2 w = *reinterpret_cast<const uint2 *>(src);
        xw[u] = ju2{w.x, w.y};
      } else {
        const float4 w = *reinterpret_cast<const float4 *>(src);
        xw[u] = ju2{__float_as_uint(w.x), __float_as_uint(w.y)};
        xw2[u] = ju2{__float_as_uint(w.z), __float_as_uint(w.w)};
      }
    }
    __syncthreads();                                        // the staging area is reused
  } else if constexpr (MODE == FUSED_DECODE) {
    if (bits) {
      const int lng = 31 - __builtin_clz(D / g), ng = 1 << lng;              // scales per row
      uint16_t *sS = reinterpret_cast<uint16_t *>(sh + BT * L::CODE_ROW);
      const int lW = 31 - __builtin_clz(rows_bytes / 4), W = 1 << lW;        // code words per row
      const uint8_t *cb = c.codes + ((int64_t)s * T + t0) * rows_bytes;
      for (int q = tid; q < BT * W; q += NT) {
        const int r = q >> lW, wi = q & (W - 1), rr = r < nrows ? r : nrows - 1;
        *reinterpret_cast<uint32_t *>(sh + r * code_row + 4 * wi) =
            *gptr(reinterpret_cast<const uint32_t *>(cb + (int64_t)rr * rows_bytes + 4 * wi));
      }
      const uint16_t *sb = c.scales + ((int64_t)s * T + t0) * ng;
      for (int q = tid; q < BT * ng; q += NT) {
        const int r = q >> lng, k = q & (ng - 1), rr = r < nrows ? r : nrows - 1;
        sS[q] = *gptr(sb + (int64_t)rr * ng + k);
      }
      __syncthreads();
      const int levels = (1 << bits) - 1;
      const float mid = 0.5f * (float)levels;
      float v[NV];
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const uint8_t *src = sh + trow * code_row + (8 * u + 4 * h) * bits / 8;
        uint32_t cw;
        if (bits == 8) cw = *reinterpret_cast<const uint32_t *>(src);
        else if (bits == 4) cw = *reinterpret_cast<const uint16_t *>(src);
        else cw = *src;
        const float dl = h_val(sS[(trow << lng) + ((8 * u) >> lg)]);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[4 * u + i] = ((float)((cw >> (bits * i)) & (uint32_t)levels) - mid) * dl;
      }
      __syncthreads();                                      // the staging area is reused
      // Walsh-Hadamard transform: value bits in the lane, feature bit 2 across the pair
#pragma unroll
      for (int w = 1; w < NV; w <<= 1)
#pragma unroll
        for (int k = 0; k < NV; ++k)
          if ((k & w) == 0) {
            const float p = v[k], q = v[k + w];
            v[k] = p + q;
            v[k + w] = p - q;
          }
#pragma unroll
      for (int k = 0; k < NV; ++k) acc2[k >> 4][k & 15] = ldexpf(pair_butterfly(v[k], h ? -1.f : 1.f) * a.inv_sqrt_d, -xe);
    }
  }

  if (rT > 0) {
    f32x16_t acc1[FB];
#pragma unroll
    for (int b = 0; b < FB; ++b)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc1[b][q] = 0.f;
    // stage 1 over K chunks of 32 staged in LDS, two chunks ahead in registers (slot 0 holds
    // the even chunks, slot 1 the odd ones)
    for (int k0 = 0; k0 < K16; k0 += 64) {
#pragma unroll
      for (int sl = 0; sl < 2; ++sl) {
        const int kc0 = k0 + 32 * sl;
        if (kc0 >= K16) break;
        __syncthreads();                                    // the previous chunk has been read
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int q = tid + NT * e, r = q >> 2, p = q & 3;
          *reinterpret_cast<ju4 *>(sU + r * L::LDK + 8 * p) = pu[sl][e];
          *reinterpret_cast<ju4 *>(sG + r * L::LDK + 8 * p) = pg[sl][e];
        }
        __syncthreads();
        if (kc0 + 64 < K16) fetch(sl, kc0 + 64);            // in flight during two chunks
#pragma unroll
        for (int kk = 0; kk < 32; kk += 16) {
          if (kc0 + kk >= K16) break;
          const f16x8_t ub = *reinterpret_cast<const f16x8_t *>(sU + trow * L::LDK + kk + 8 * h);
#pragma unroll
          for (int b = 0; b < FB; ++b)
            if (b < NB1) {
              const f16x8_t ga = *reinterpret_cast<const f16x8_t *>(sG + (32 * b + tl) * L::LDK + kk + 8 * h);
              acc1[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ga, ub, acc1[b], 0, 0, 0);
            }
        }
      }
    }
    // stage 2: acc2 += U^_d (Y^T 2^-ky), Y split into fp16 hi + lo; chunk kc = 2 b + cc takes
    // entries 8 cc .. 8 cc + 7 of block b
#pragma unroll
    for (int kc = 0; kc < 2 * FB; ++kc) {
      if (kc < RD / 16) {
        const int b = kc >> 1, cc = kc & 1;
        f16x8_t yh, yl;
#pragma unroll
        for (int sl = 0; sl < 8; ++sl) {
          const float yv = ldexpf(acc1[b][8 * cc + sl], -ky);
          const _Float16 hi = (_Float16)yv;
          yh[sl] = hi;
          yl[sl] = (_Float16)(yv - (float)hi);
        }
#pragma unroll
        for (int fb = 0; fb < FB; ++fb) {
          const f16x8_t ua = *reinterpret_cast<const f16x8_t *>(sud + (32 * fb + tl) * L::LDU + 16 * kc + 8 * h);
          acc2[fb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ua, yh, acc2[fb], 0, 0, 0);
          acc2[fb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ua, yl, acc2[fb], 0, 0, 0);
        }
      }
    }
  }
  float v[NV];
#pragma unroll
  for (int fb = 0; fb < FB; ++fb)
#pragma unroll
    for (int q = 0; q < 16; ++q) v[16 * fb + q] = ldexpf(acc2[fb][q], xe);     // exact

  if constexpr (MODE == FUSED_XTILDE) {
    if (tin) {
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const jf4 sq = gload_f4(sgn + 8 * u + 4 * h);
        *reinterpret_cast<jf4 *>(c.xt_out + ebase + 8 * u + 4 * h) =
            jf4{v[4 * u] * sq.x, v[4 * u + 1] * sq.y, v[4 * u + 2] * sq.z, v[4 * u + 3] * sq.w};
      }
    }
  } else if constexpr (MODE == FUSED_RESIDUAL) {
    // v = s * X~ - s * X = -(s * r), exact; r' = H (s * r) / sqrt(d) = -H v / sqrt(d)
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      float x[4];
      if constexpr (sizeof(TIO) == 2) {
        x[0] = bf16_to_f32((bf16_t)(xw[u].x & 0xffffu)); x[1] = bf16_to_f32((bf16_t)(xw[u].x >> 16));
        x[2] = bf16_to_f32((bf16_t)(xw[u].y & 0xffffu)); x[3] = bf16_to_f32((bf16_t)(xw[u].y >> 16));
      } else {
        x[0] = __uint_as_float(xw[u].x); x[1] = __uint_as_float(xw[u].y);
        x[2] = __uint_as_float(xw2[u].x); x[3] = __uint_as_float(xw2[u].y);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * u + i] += x[i];
    }
#pragma unroll
    for (int w = 1; w < NV; w <<= 1)
#pragma unroll
      for (int k = 0; k < NV; ++k)
        if ((k & w) == 0) {
          const float p = v[k], q = v[k + w];
          v[k] = p + q;
          v[k + w] = p - q;
        }
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] = pair_butterfly(v[k], h ? -1.f : 1.f) * -a.inv_sqrt_d;
    // group max: units u / gw of the lane, then the pair
    float am[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u)
      am[u] = fmaxf(fmaxf(fabsf(v[4 * u]), fabsf(v[4 * u + 1])), fmaxf(fabsf(v[4 * u + 2]), fabsf(v[4 * u + 3])));
#pragma unroll
    for (int w = 1; w < NU; w <<= 1)
      if (w < gw) {
#pragma unroll
        for (int u = 0; u < NU; ++u)
          if ((u & w) == 0) {
            const float mm = fmaxf(am[u], am[u + w]);
            am[u] = mm;
            am[u + w] = mm;
          }
      }
    const int levels = (1 << bits) - 1;
    const float mid = 0.5f * (float)levels;
    __syncthreads();                                        // stage 1's chunks have been read
    float delta = 0.f, inv = 0.f;
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      if ((u & (gw - 1)) == 0) {                            // first unit of a group
        const float aa = pair_max(am[u]);
        float dl = 2.f * aa / (float)levels;
        dl = fminf(dl, 65504.f);
        delta = f16_round(dl);
        // r / delta as r * (1 / delta): within 1.5 ulp of the quotient
        inv = delta == 0.f ? 0.f : 1.f / delta;
      }
      uint32_t word = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float cq;
        if (delta == 0.f) {
          cq = (float)(1 << (bits - 1));
        } else {
          cq = __builtin_amdgcn_fmed3f(__builtin_rintf(fmaf(v[4 * u + i], inv, mid)), 0.f, (float)levels);
        }
        word |= (uint32_t)cq << (bits * i);
      }
      uint8_t *dst = sh + trow * code_row + (8 * u + 4 * h) * bits / 8;
      if (bits == 8) *reinterpret_cast<uint32_t *>(dst) = word;
      else if (bits == 4) *reinterpret_cast<uint16_t *>(dst) = (uint16_t)word;
      else *dst = (uint8_t)word;
      if (tin && h == 0 && (u & (gw - 1)) == 0) c.scales[(ebase + 8 * u) >> lg] = h_bits(delta);
    }
    __syncthreads();
    // the tile's codes are one contiguous run of nrows rows
    const int lW = 31 - __builtin_clz(rows_bytes / 4), W = 1 << lW;
    uint8_t *cb = c.codes + ((int64_t)s * T + t0) * rows_bytes;
    for (int q = tid; q < nrows * W; q += NT) {
      const int r = q >> lW, wi = q & (W - 1);
      *gptr(reinterpret_cast<uint32_t *>(cb + (int64_t)r * rows_bytes + 4 * wi)) =
          *reinterpret_cast<const uint32_t *>(sh + r * code_row + 4 * wi);
    }
  } else {
    if constexpr (ROPE) {
      // X^ = s * v first
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const jf4 sq = gload_f4(sgn + 8 * u + 4 * h);
        v[4 * u] *= sq.x; v[4 * u + 1] *= sq.y; v[4 * u + 2] *= sq.z; v[4 * u + 3] *= sq.w;
      }
      // features f and f + D/2 (value indices k and k + NV/2) rotate together by pos theta_j
      const double pos = (double)(t + a.rope_offset);
#pragma unroll
      for (int k = 0; k < NV / 2; ++k) {
        const int f = 8 * (k / 4) + 4 * h + (k % 4);            // < D/2
        const double theta = exp2(-(2.0 * f / D) * a.rope_log2_base);
        double sn, cs;
        sincos(pos * theta, &sn, &cs);
        const float cf = (float)cs, sf = (float)sn;
        const float lo = v[k], hi = v[k + NV / 2];
        v[k] = fmaf(-hi, sf, lo * cf);
        v[k + NV / 2] = fmaf(lo, sf, hi * cf);
      }
    }
    __syncthreads();                                        // stage 1's chunks have been read
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      uint8_t *dst = sh + trow * L::IO_ROW + (8 * u + 4 * h) * (int)sizeof(TIO);
      if constexpr (sizeof(TIO) == 2) {
        const uint32_t w0 = (uint32_t)f32_to_bf16(v[4 * u]) | ((uint32_t)f32_to_bf16(v[4 * u + 1]) << 16);
        const uint32_t w1 = (uint32_t)f32_to_bf16(v[4 * u + 2]) | ((uint32_t)f32_to_bf16(v[4 * u + 3]) << 16);
        *reinterpret_cast<uint2 *>(dst) = make_uint2(w0, w1);
      } else {
        *reinterpret_cast<float4 *>(dst) = make_float4(v[4 * u], v[4 * u + 1], v[4 * u + 2], v[4 * u + 3]);
      }
    }
    __syncthreads();
    // the tile's rows, 8 bytes at a time along each row; each thread moves the same piece p
    // of several rows and applies the rotation signs of its entries (X^ = s * v) by a mask,
    // unless RoPE has applied them already
    constexpr int P8 = D * (int)sizeof(TIO) / 8;
    static_assert(NT % P8 == 0, "piece index fixed per thread");
    const int pp = tid % P8;
    ju2 flip{0u, 0u};
    if constexpr (!ROPE) {
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        if constexpr (sizeof(TIO) == 2) {
          const int f = 4 * pp + 2 * w;
          flip[w] = (sgn[f] < 0.f ? 0x8000u : 0u) | (sgn[f + 1] < 0.f ? 0x80000000u : 0u);
        } else {
          flip[w] = sgn[2 * pp + w] < 0.f ? 0x80000000u : 0u;
        }
      }
    }
    uint8_t *ob = reinterpret_cast<uint8_t *>(c.out);
    for (int r = tid / P8; r < nrows; r += NT / P8) {
      *gptr(reinterpret_cast<ju2 *>(ob + (srow + (int64_t)(t0 + r) * a.s_tok) * (int64_t)sizeof(TIO) + 8 * pp)) =
          *reinterpret_cast<const ju2 *>(sh + r * L::IO_ROW + 8 * pp) ^ flip;
    }
  }
}

template <int D, int MODE, typename TIO, bool USPLIT>
hipError_t launch_mode(const FusedArgs &a, bool rope, hipStream_t st) {
  const dim3 grid((unsigned)(a.per_xcd * 8)), block(NT);
  if constexpr (MODE == FUSED_DECODE) {
    if (rope) {
      hipLaunchKernelGGL((k_fused<D, MODE, TIO, USPLIT, true>), grid, block, 0, st, a);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((k_fused<D, MODE, TIO, USPLIT, false>), grid, block, 0, st, a);
  return hipGetLastError();
}

template <int D, int MODE>
hipError_t launch_d(const FusedArgs &a, int io_dtype, bool split, bool rope, hipStream_t st) {
  if (MODE == FUSED_XTILDE || io_dtype == JOLT_F32)
    return split ? launch_mode<D, MODE, float, true>(a, rope, st) : launch_mode<D, MODE, float, false>(a, rope, st);
  return split ? launch_mode<D, MODE, bf16_t, true>(a, rope, st) : launch_mode<D, MODE, bf16_t, false>(a, rope, st);
}

template <int D, int MODE>
hipError_t launch_core(const FusedArgs &a, int io_dtype, bool rope, hipStream_t st) {
  const dim3 grid((unsigned)(a.per_xcd * 8)), block(NT);
  const bool f32 = MODE == FUSED_XTILDE || io_dtype == JOLT_F32;
  if constexpr (MODE == FUSED_DECODE) {
    if (rope) {
      if (f32) hipLaunchKernelGGL((k_core<D, MODE, float, true>), grid, block, 0, st, a);
      else hipLaunchKernelGGL((k_core<D, MODE, bf16_t, true>), grid, block, 0, st, a);
      return hipGetLastError();
    }
  }
  if (f32) hipLaunchKernelGGL((k_core<D, MODE, float, false>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((k_core<D, MODE, bf16_t, false>), grid, block, 0, st, a);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_m(const FusedArgs &a, int d, int io_dtype, bool split, bool rope, hipStream_t st) {
  if (!split) {
    switch (d) {
      case 32: return launch_core<32, MODE>(a, io_dtype, rope, st);
      case 64: return launch_core<64, MODE>(a, io_dtype, rope, st);
      case 128: return launch_core<128, MODE>(a, io_dtype, rope, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (d) {
    case 32: return launch_d<32, MODE>(a, io_dtype, split, rope, st);
    case 64: return launch_d<64, MODE>(a, io_dtype, split, rope, st);
    case 128: return launch_d<128, MODE>(a, io_dtype, split, rope, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int fused_tile_tokens() { return BT; }

hipError_t launch_w_prepare(const FusedCell *cells_dev, int n_cells, int m, int d, hipStream_t st) {
  if (n_cells <= 0 || m <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_w_prepare, dim3(m, n_cells), dim3(256), 0, st, cells_dev, m, d);
  return hipGetLastError();
}

hipError_t launch_core_prepare(const FusedCell *cells_dev, const float *signs_dev, int n_cells, int m, int d,
                               hipStream_t st) {
  if (n_cells <= 0 || m <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_core_prepare, dim3(m, n_cells), dim3(256), 0, st, cells_dev, signs_dev, m, d);
  return hipGetLastError();
}

hipError_t launch_fused(FusedArgs a, int mode, int d, int io_dtype, bool split_factors, hipStream_t st) {
  a.tiles_t = (a.T + BT - 1) / BT;
  const int64_t total = (int64_t)a.n_cells * a.m * a.tiles_t;
  if (total <= 0) return hipSuccess;
  if (total > (int64_t)1 << 30) return hipErrorInvalidValue;
  a.total = (int32_t)total;
  a.per_xcd = (int32_t)((total + 7) / 8);
  const bool rope = a.rope != 0 && mode == FUSED_DECODE;
  if (mode == FUSED_RESIDUAL) return launch_m<FUSED_RESIDUAL>(a, d, io_dtype, split_factors, false, st);
  if (mode == FUSED_DECODE) return launch_m<FUSED_DECODE>(a, d, io_dtype, split_factors, rope, st);
  if (mode == FUSED_XTILDE) return launch_m<FUSED_XTILDE>(a, d, JOLT_F32, split_factors, false, st);
  return hipErrorInvalidValue;
}

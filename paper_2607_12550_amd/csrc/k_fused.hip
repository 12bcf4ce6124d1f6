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

template <int MODE>
hipError_t launch_m(const FusedArgs &a, int d, int io_dtype, bool split, bool rope, hipStream_t st) {
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

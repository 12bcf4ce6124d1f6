// Decode-time attention evaluated on the compressed factors (the fused path that section 8
// and the conclusion name as the route to decode parity): the decoded cache
// X^_s = U_T (2^e_s G_s) U_d^T + R_s, R_s[t] = signs . H r'_s[t] / sqrt(d), is never formed.
//
//   key side:   q . X^_s[t] = U_T[t] . g + r'_s[t] . q',   g = 2^e_s G_s (U_d^T q),
//               q' = H (signs . q) / sqrt(d)           (H symmetric, entries +-1)
//   value side: sum_t p_t X^_s[t] = ((sum_t p_t U_T[t]) 2^e_s G_s) U_d^T
//                                   + signs . H (sum_t p_t r'_s[t]) / sqrt(d)
//
// Three kernels: k_attend_prep forms g and q' per (item, query head); k_attend_chunk runs
// over 64-token chunks of one key-value head of one item (scores, a chunk-local softmax, and
// the value-side sums of U_T rows and dequantised codes, weighted by the unnormalised
// probabilities, for all query heads of that key-value head at once); k_attend_combine
// merges the chunks with the usual max / rescale rule in a fixed order and applies the
// value factors and the inverse rotation once per query head.  Per token a query head
// reads r_T factor values and d codes instead of d decoded values plus the decompression.
#include <cmath>
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace {

// Blob pointers come from a table in memory, so the compiler cannot tell their address
// space: every load through them goes through gptr() (global_* instructions, which do not
// hold the LDS counter the way flat_* ones do).
JOLT_DEV float factor(const void *p, int64_t i, int f16) {
  return f16 ? (float)gptr(reinterpret_cast<const _Float16 *>(p))[i] : gptr(reinterpret_cast<const float *>(p))[i];
}

// The codes of one slice over a chunk (ATTN_CHUNK rows of D elements), held in registers
// between their global loads and the LDS dequantisation, so that the next slice's loads are
// in flight while the current slice is used.  Thread blocks of 8 elements, consecutive
// threads on consecutive blocks (coalesced); a block lies in one quantiser group (the group
// size is a multiple of 8).
template <int D>
struct CodeRegs {
  static constexpr int NB = ATTN_CHUNK * D / 8;
  static constexpr int BPT = (NB + 255) / 256;
  uint2 w[BPT];
  float sc[BPT];
};

template <int D>
JOLT_DEV void codes_load(CodeRegs<D> &c, const AttnBlob &b, int64_t row0, int nt, int group) {
#pragma unroll
  for (int k = 0; k < CodeRegs<D>::BPT; ++k) {
    const int blk = threadIdx.x + k * 256, t = blk / (D / 8), f = (blk % (D / 8)) * 8;
    c.w[k] = make_uint2(0u, 0u);
    c.sc[k] = 0.f;
    if (blk < CodeRegs<D>::NB && t < nt) {
      const int64_t elem = (row0 + t) * D + f;
      if (b.bits == 8) {
        const uint64_t v = *gptr(reinterpret_cast<const uint64_t *>(b.codes + elem));
        c.w[k].x = (uint32_t)v;
        c.w[k].y = (uint32_t)(v >> 32);
      }
      else if (b.bits == 4) c.w[k].x = *gptr(reinterpret_cast<const uint32_t *>(b.codes + elem / 2));
      else c.w[k].x = *gptr(reinterpret_cast<const uint16_t *>(b.codes + elem / 4));
      c.sc[k] = (float)*gptr(reinterpret_cast<const _Float16 *>(b.scales + elem / group));
    }
  }
}

// code - (2^b - 1)/2 (a half-integer of magnitude <= 127.5: exact in fp16) into ct[t][f .. f+7]
// and the block's scale into csc[t][f / 8]; rows past the chunk's end get scale 0
template <int D>
JOLT_DEV void codes_stash16(const CodeRegs<D> &c, int bits, _Float16 (*ct)[D + 8], float (*csc)[D / 8]) {
  const float mid = 0.5f * (float)((1 << bits) - 1);
  const uint32_t mask = (1u << bits) - 1u;
#pragma unroll
  for (int k = 0; k < CodeRegs<D>::BPT; ++k) {
    const int blk = threadIdx.x + k * 256, t = blk / (D / 8), f = (blk % (D / 8)) * 8;
    if (blk >= CodeRegs<D>::NB) continue;
    _Float16 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int bit = i * bits;
      const uint32_t word = bit < 32 ? c.w[k].x : c.w[k].y;
      v[i] = (_Float16)((float)((word >> (bit & 31)) & mask) - mid);
    }
    uint4 pk;
    __builtin_memcpy(&pk, v, 16);
    *reinterpret_cast<uint4 *>(&ct[t][f]) = pk;
    csc[t][f / 8] = c.sc[k];
  }
}

// dst[q] = src(q) for q < n by all 256 threads: each thread issues eight loads before it
// stores any of them, so a pass costs one memory round trip, not eight
template <int NT = 256, class F>
JOLT_DEV void stage_lds(float *dst, int n, F src) {
  for (int q0 = threadIdx.x; q0 < n; q0 += NT * 8) {
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int q = q0 + k * NT;
      v[k] = q < n ? src(q) : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int q = q0 + k * NT;
      if (q < n) dst[q] = v[k];
    }
  }
}

// a factor matrix of n consecutive values staged as fp32 (the storage type chosen once)
template <int NT = 256>
JOLT_DEV void stage_factor(float *dst, const void *p, int64_t off, int n, int f16) {
  if (f16) {
    const JOLT_GLOBAL _Float16 *h = gptr(reinterpret_cast<const _Float16 *>(p)) + off;
    stage_lds<NT>(dst, n, [&](int q) { return (float)h[q]; });
  } else {
    const JOLT_GLOBAL float *x = gptr(reinterpret_cast<const float *>(p)) + off;
    stage_lds<NT>(dst, n, [&](int q) { return x[q]; });
  }
}

// Sylvester Hadamard entry (-1)^popcount(i & j)
JOLT_DEV float hsign(int i, int j) { return (__popc((unsigned)(i & j)) & 1) ? -1.f : 1.f; }

template <int D>
__global__ void __launch_bounds__(128) k_attend_prep(AttnArgs a) {
  constexpr int ROWS = 32;                          // rows of U_d or G_s per staging pass
  const int item = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
  const AttnItem it = a.items[item];     // by value: one set of scalar loads
  const AttnBlob &kb = it.k;
  const int rep = a.n_q / a.heads, s = it.layer * a.heads + j / rep;
  __shared__ float q[D], qt[D];
  __shared__ float fs[ROWS * D];                    // rows of U_d, then of G_s (r_d <= d)
  const float *qin = a.Q + ((int64_t)item * a.n_q + j) * D;
  const float *sg = a.signs + (int64_t)item * 2 * D;
  for (int f = tid; f < D; f += 128) q[f] = qin[f];
  __syncthreads();
  // q' = H (signs . q) / sqrt(d)
  float *qr = a.qr + ((int64_t)item * a.n_q + j) * D;
  for (int f = tid; f < D; f += 128) {
    float acc = 0.f;
    for (int g = 0; g < D; ++g) acc = fmaf(hsign(f, g), sg[g] * q[g], acc);
    qr[f] = acc * a.inv_sqrt_d;
  }
  // q~ = U_d^T q (rows of U_d staged ROWS at a time), then g = 2^e_s G_s q~
  float qk = 0.f;                                   // thread k < r_d
  for (int f0 = 0; f0 < D; f0 += ROWS) {
    __syncthreads();
    stage_factor<128>(fs, kb.Ud, (int64_t)f0 * kb.rd, ROWS * kb.rd, kb.f16);
    __syncthreads();
    if (tid < kb.rd)
      for (int f = 0; f < ROWS; ++f) qk = fmaf(fs[f * kb.rd + tid], q[f0 + f], qk);
  }
  if (tid < kb.rd) qt[tid] = qk;
  float *gk = a.gk + ((int64_t)item * a.n_q + j) * a.rk_max;
  const int ge = kb.rT ? (int)gptr(kb.gexp)[s] : 0;       // applied per value: 2^ge may not be an fp32
  const int64_t g0 = (int64_t)s * kb.rT * kb.rd;
  for (int i0 = 0; i0 < kb.rT; i0 += ROWS) {
    const int ni = min(ROWS, kb.rT - i0);
    __syncthreads();
    stage_factor<128>(fs, kb.G, g0 + (int64_t)i0 * kb.rd, ni * kb.rd, kb.f16);
    __syncthreads();
    for (int i = tid; i < ni; i += 128) {
      float acc = 0.f;
      for (int k = 0; k < kb.rd; ++k) acc = fmaf(fs[i * kb.rd + k], qt[k], acc);
      gk[i0 + i] = kb.rT ? ldexpf(acc, ge) : 0.f;
    }
  }
}

// eight consecutive factor values of a row (16-byte loads when the row start allows)
JOLT_DEV void factor8(const void *p, int64_t i, int f16, bool vec, float (&v)[8]) {
  if (f16 && vec) {
    const ju4 u = gload_u4(reinterpret_cast<const _Float16 *>(p) + i);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      _Float16 lo, hi;
      const uint16_t l16 = (uint16_t)(w[k] & 0xffff), h16 = (uint16_t)(w[k] >> 16);
      __builtin_memcpy(&lo, &l16, 2); __builtin_memcpy(&hi, &h16, 2);
      v[2 * k] = (float)lo; v[2 * k + 1] = (float)hi;
    }
  } else if (!f16 && vec) {
    const jf4 x = gload_f4(reinterpret_cast<const float *>(p) + i), y = gload_f4(reinterpret_cast<const float *>(p) + i + 4);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w; v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = factor(p, i + k, f16);
  }
}

// One rank block of U_T rows of a chunk: thread (row t = tid / 4, ranks (tid % 4) * 8 + 0..7
// of the block), loaded into registers ahead of its LDS stash.
constexpr int ATTN_RB = 32;

JOLT_DEV void urows_load(float (&u)[8], const AttnBlob &b, int t0, int nt, int i0) {
  const int t = threadIdx.x >> 2, i = i0 + (threadIdx.x & 3) * 8;
#pragma unroll
  for (int k = 0; k < 8; ++k) u[k] = 0.f;
  if (t >= nt || i >= b.rT) return;
  const int64_t e = (int64_t)(t0 + t) * b.rT + i;
  if (i + 8 <= b.rT && (b.f16 ? (e & 7) == 0 : (e & 3) == 0)) {
    factor8(b.UT, e, b.f16, true, u);
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) u[k] = i + k < b.rT ? factor(b.UT, e + k, b.f16) : 0.f;
  }
}

// Chunk pass: one workgroup per (64-token chunk, key-value head, item), so that every
// workgroup issues all of its global loads at once (the slice's key and value codes of the
// chunk, the first rank block of both token factors, the slice's queries) and several
// workgroups share a CU.  For the rep query heads of slice s:
//   1. key scores: residual part from the dequantised codes staged in LDS (fp16 code
//      offsets, one scale per 8 elements) against the rotated queries, plus the low-rank
//      part U_T[t] . g over rank blocks of 32;
//   2. chunk-local softmax: wave r holds head r, lane t token t (scores never leave
//      registers);
//   3. value residual sums b[r][f] = sum_t p[r][t] r'[t][f] and value low-rank sums
//      a[r][i] = sum_t p[r][t] U_T[t][i]: thread (column, token stripe), stripes added in a
//      fixed order.
// REP > 0: the number of query heads per key-value head, fixed at compile time (the head
// loops unroll without predicates); REP = 0 takes it from the call (at most ATTN_REP_MAX).
template <int D, int REP>
__global__ void __launch_bounds__(256) k_attend_chunk(AttnArgs a) {
  constexpr int CH = ATTN_CHUNK, RB = ATTN_RB, RMAX = REP ? REP : ATTN_REP_MAX, P = 256 / D;
  static_assert(CH == 64, "one lane per token of a chunk");
  const int chunk = blockIdx.x, h = blockIdx.y, item = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const AttnItem it = a.items[item];     // by value: one set of scalar loads
  const AttnBlob &kb = it.k, &vb = it.v;
  const int T = a.T, t0 = chunk * CH, nt = min(CH, T - t0);
  const int nq = a.n_q, rep = REP ? REP : nq / a.heads, s = it.layer * a.heads + h, j0 = h * rep;
  __shared__ __attribute__((aligned(16))) _Float16 ct[CH][D + 8];
  __shared__ float csc[CH][D / 8];
  __shared__ float ut[CH][RB + 1];
  __shared__ float gq[RMAX][RB];
  __shared__ __attribute__((aligned(16))) float qv[RMAX][D];
  __shared__ float pp[CH][RMAX];
  __shared__ float red[256 * RMAX];
  // every global load of the workgroup that does not depend on a later result
  CodeRegs<D> kr, vr;
  const int64_t row0 = (int64_t)s * T + t0;
  if (kb.bits) codes_load(kr, kb, row0, nt, a.group);
  if (vb.bits) codes_load(vr, vb, row0, nt, a.group);
  float uk[8], uv[8];
  urows_load(uk, kb, t0, nt, 0);
  urows_load(uv, vb, t0, nt, 0);
  {
    const float *qsrc = a.qr + ((int64_t)item * nq + j0) * D;     // rep consecutive rows
    stage_lds(&qv[0][0], rep * D, [&](int q) { return qsrc[q]; });
    const float *gsrc = a.gk + ((int64_t)item * nq + j0) * a.rk_max;
    const int rk = a.rk_max, rT = kb.rT;
    stage_lds(&gq[0][0], RMAX * RB, [&](int q) {
      const int r = q / RB, i = q % RB;
      return r < rep && i < rT ? gsrc[(int64_t)r * rk + i] : 0.f;
    });
  }
  if (kb.bits) codes_stash16(kr, kb.bits, ct, csc);
  {
    const int t = tid >> 2, c = (tid & 3) * 8;
#pragma unroll
    for (int k = 0; k < 8; ++k) ut[t][c + k] = uk[k];
  }
  __syncthreads();
  // 1. key scores: item k of a thread is head r = wave + 4 k, token t = lane
  float sc[2] = {0.f, 0.f};
  if (kb.bits) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int r = wave + 4 * k;
      if (r >= rep) continue;
      float acc = 0.f;
      for (int b8 = 0; b8 < D / 8; ++b8) {
        const uint4 pk = *reinterpret_cast<const uint4 *>(&ct[lane][b8 * 8]);
        _Float16 cv[8];
        __builtin_memcpy(cv, &pk, 16);
        const float4 x = *reinterpret_cast<const float4 *>(&qv[r][b8 * 8]);
        const float4 y = *reinterpret_cast<const float4 *>(&qv[r][b8 * 8 + 4]);
        float d8 = (float)cv[0] * x.x;
        d8 = fmaf((float)cv[1], x.y, d8); d8 = fmaf((float)cv[2], x.z, d8); d8 = fmaf((float)cv[3], x.w, d8);
        d8 = fmaf((float)cv[4], y.x, d8); d8 = fmaf((float)cv[5], y.y, d8); d8 = fmaf((float)cv[6], y.z, d8);
        d8 = fmaf((float)cv[7], y.w, d8);
        acc = fmaf(csc[lane][b8], d8, acc);
      }
      sc[k] = acc;
    }
  }
  for (int i0 = 0; i0 < kb.rT; i0 += RB) {
    if (i0 > 0) {
      // next rank block: its loads were issued during the previous block
      __syncthreads();
      const int t = tid >> 2, c = (tid & 3) * 8;
#pragma unroll
      for (int k = 0; k < 8; ++k) ut[t][c + k] = uk[k];
      {
        const float *gsrc = a.gk + ((int64_t)item * nq + j0) * a.rk_max + i0;
        const int rk = a.rk_max, nr = kb.rT - i0;
        stage_lds(&gq[0][0], RMAX * RB, [&](int q) {
          const int r = q / RB, i = q % RB;
          return r < rep && i < nr ? gsrc[(int64_t)r * rk + i] : 0.f;
        });
      }
      __syncthreads();
    }
    if (i0 + RB < kb.rT) urows_load(uk, kb, t0, nt, i0 + RB);
    const int ni = min(RB, kb.rT - i0);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int r = wave + 4 * k;
      if (r >= rep) continue;
      float acc = sc[k];
      for (int i = 0; i < ni; ++i) acc = fmaf(ut[lane][i], gq[r][i], acc);
      sc[k] = acc;
    }
  }
  // 2. chunk-local softmax
  const int stride = 2 + a.rv_max + D;
  float *part = a.part + ((int64_t)item * a.chunks + chunk) * nq * stride;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int r = wave + 4 * k;
    if (r >= rep) continue;                       // uniform across the wave
    const float v = lane < nt ? sc[k] * a.scale : -INFINITY;
    float mx = v;
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    const float e = lane < nt ? expf(v - mx) : 0.f;
    float sum = e;
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
    pp[lane][r] = e;
    if (lane == 0) { part[(int64_t)(j0 + r) * stride] = mx; part[(int64_t)(j0 + r) * stride + 1] = sum; }
  }
  __syncthreads();
  // 3a. value residual sums
  if (vb.bits) codes_stash16(vr, vb.bits, ct, csc);
  {
    const int t = tid >> 2, c = (tid & 3) * 8;
#pragma unroll
    for (int k = 0; k < 8; ++k) ut[t][c + k] = uv[k];
  }
  __syncthreads();
  {
    const int f = tid % D, stripe = tid / D;
    float acc[RMAX];
#pragma unroll
    for (int r = 0; r < RMAX; ++r) acc[r] = 0.f;
    if (vb.bits) {
      for (int t = stripe; t < nt; t += P) {
        const float v = csc[t][f / 8] * (float)ct[t][f];
#pragma unroll
        for (int r = 0; r < RMAX; ++r)
          if (r < rep) acc[r] = fmaf(pp[t][r], v, acc[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < RMAX; ++r) red[(stripe * RMAX + r) * D + f] = acc[r];
  }
  __syncthreads();
  for (int q = tid; q < rep * D; q += 256) {
    const int r = q / D, f = q % D;
    float sum = 0.f;
    for (int st = 0; st < P; ++st) sum += red[(st * RMAX + r) * D + f];
    part[(int64_t)(j0 + r) * stride + 2 + a.rv_max + f] = sum;
  }
  // 3b. value low-rank sums, rank block by rank block (stripes of 8 tokens)
  for (int i0 = 0; i0 < vb.rT; i0 += RB) {
    __syncthreads();
    if (i0 > 0) {
      const int t = tid >> 2, c = (tid & 3) * 8;
#pragma unroll
      for (int k = 0; k < 8; ++k) ut[t][c + k] = uv[k];
      __syncthreads();
    }
    if (i0 + RB < vb.rT) urows_load(uv, vb, t0, nt, i0 + RB);
    {
      const int i = tid % RB, stripe = tid / RB;   // 8 stripes
      float acc[RMAX];
#pragma unroll
      for (int r = 0; r < RMAX; ++r) acc[r] = 0.f;
      for (int t = stripe; t < nt; t += 256 / RB) {
        const float u = ut[t][i];
#pragma unroll
        for (int r = 0; r < RMAX; ++r)
          if (r < rep) acc[r] = fmaf(pp[t][r], u, acc[r]);
      }
#pragma unroll
      for (int r = 0; r < RMAX; ++r) red[(stripe * RMAX + r) * RB + i] = acc[r];
    }
    __syncthreads();
    const int ni = min(RB, vb.rT - i0);
    for (int q = tid; q < rep * ni; q += 256) {
      const int r = q / ni, i = q % ni;
      float sum = 0.f;
      for (int st = 0; st < 256 / RB; ++st) sum += red[(st * RMAX + r) * RB + i];
      part[(int64_t)(j0 + r) * stride + 2 + i0 + i] = sum;
    }
  }
}

// Combine: one workgroup per (item, query head).  The chunk partials are summed by column
// with eight chunks' loads in flight per thread; the slice's value core G_s and U_d are
// staged in LDS (eight loads in flight per thread) before the two small products.
template <int D>
__global__ void __launch_bounds__(256) k_attend_combine(AttnArgs a) {
  constexpr int CG = 16;
  const int item = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
  const AttnItem it = a.items[item];     // by value: one set of scalar loads
  const AttnBlob &vb = it.v;
  const int rep = a.n_q / a.heads, s = it.layer * a.heads + j / rep;
  const int stride = 2 + a.rv_max + D, ncol = vb.rT + D;
  const float *part = a.part + ((int64_t)item * a.chunks * a.n_q + j) * stride;
  const int64_t cstride = (int64_t)a.n_q * stride;
  __shared__ float av[ATTN_RT_MAX], w[D], bv[D];
  __shared__ float red[4];
  extern __shared__ float dyn[];          // chunk weights [chunks], then a staging area
  float *cw = dyn;
  float *stage = dyn + (a.chunks + 3) / 4 * 4;
  // M = max over chunks; L = sum_c l_c exp(m_c - M): threads take chunks tid, tid + 256, ...
  // in order, then a fixed butterfly and the four waves in order (deterministic)
  float M = -INFINITY;
  for (int c = tid; c < a.chunks; c += 256) M = fmaxf(M, part[c * cstride]);
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
  if ((tid & 63) == 0) red[tid >> 6] = M;
  __syncthreads();
  M = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float L = 0.f;
  for (int c = tid; c < a.chunks; c += 256) {
    const float wgt = expf(part[c * cstride] - M);
    cw[c] = wgt;
    L += part[c * cstride + 1] * wgt;
  }
  for (int o = 32; o >= 1; o >>= 1) L += __shfl_xor(L, o, 64);
  __syncthreads();
  if ((tid & 63) == 0) red[tid >> 6] = L;
  __syncthreads();
  const float L_s = (red[0] + red[1]) + (red[2] + red[3]);
  // av[i] = sum_c w_c a_c[i], bv[f] = sum_c w_c b_c[f], chunks in order; a thread owns the
  // columns tid, tid + 256, ... and keeps eight chunks' loads of a column in flight
  for (int i = tid; i < ncol; i += 256) {
    const JOLT_GLOBAL float *pc = gptr(part) + 2 + (i < vb.rT ? i : a.rv_max + (i - vb.rT));
    float acc = 0.f;
    for (int c0 = 0; c0 < a.chunks; c0 += 8) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = c0 + k < a.chunks ? pc[(int64_t)(c0 + k) * cstride] : 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (c0 + k < a.chunks) acc = fmaf(cw[c0 + k], v[k], acc);
    }
    if (i < vb.rT) av[i] = acc;
    else bv[i - vb.rT] = acc;
  }
  __syncthreads();
  // w = 2^e_s (a^T G_s): r_d values, G_s staged by row blocks
  const int ge = vb.rT ? (int)gptr(vb.gexp)[s] : 0;       // applied per value: 2^ge may not be an fp32
  const int64_t g0 = (int64_t)s * vb.rT * vb.rd;
  const int gcap = max(1, (CG * ncol) / max(vb.rd, 1));          // rows of G_s per staging pass
  float wk = 0.f;
  for (int i0 = 0; i0 < vb.rT; i0 += gcap) {
    const int ni = min(gcap, vb.rT - i0);
    __syncthreads();
    stage_factor(stage, vb.G, g0 + (int64_t)i0 * vb.rd, ni * vb.rd, vb.f16);
    __syncthreads();
    if (tid < vb.rd)
      for (int i = 0; i < ni; ++i) wk = fmaf(av[i0 + i], stage[i * vb.rd + tid], wk);
  }
  if (tid < vb.rd) w[tid] = ldexpf(wk, ge);
  // U_d staged whole when it fits the staging area, else read directly
  const bool ud_lds = D * vb.rd <= CG * ncol;
  __syncthreads();
  if (ud_lds) stage_factor(stage, vb.Ud, 0, D * vb.rd, vb.f16);
  __syncthreads();
  const float *sg = a.signs + ((int64_t)item * 2 + 1) * D;
  float *o = a.O + ((int64_t)item * a.n_q + j) * D;
  const float invL = 1.f / L_s;
  for (int f = tid; f < D; f += 256) {
    float lr = 0.f;
    for (int k = 0; k < vb.rd; ++k)
      lr = fmaf(ud_lds ? stage[f * vb.rd + k] : factor(vb.Ud, (int64_t)f * vb.rd + k, vb.f16), w[k], lr);
    float res = 0.f;
    if (vb.bits) {
      for (int g = 0; g < D; ++g) res = fmaf(hsign(f, g), bv[g], res);
      res *= sg[f] * a.inv_sqrt_d;
    }
    o[f] = (lr + res) * invL;
  }
}

}  // namespace

hipError_t launch_attend(const AttnArgs &a, int d, hipStream_t st) {
#define L_(D_) \
  if (d == D_) { \
    hipLaunchKernelGGL((k_attend_prep<D_>), dim3(a.n_items, a.n_q), dim3(128), 0, st, a); \
    { const dim3 g(a.chunks, a.heads, a.n_items); const int rep = a.n_q / a.heads; \
      if (rep == 1) hipLaunchKernelGGL((k_attend_chunk<D_, 1>), g, dim3(256), 0, st, a); \
      else if (rep == 2) hipLaunchKernelGGL((k_attend_chunk<D_, 2>), g, dim3(256), 0, st, a); \
      else if (rep == 4) hipLaunchKernelGGL((k_attend_chunk<D_, 4>), g, dim3(256), 0, st, a); \
      else if (rep == 8) hipLaunchKernelGGL((k_attend_chunk<D_, 8>), g, dim3(256), 0, st, a); \
      else hipLaunchKernelGGL((k_attend_chunk<D_, 0>), g, dim3(256), 0, st, a); } \
    hipLaunchKernelGGL((k_attend_combine<D_>), dim3(a.n_items, a.n_q), dim3(256), \
                       ((a.chunks + 3) / 4 * 4 + (size_t)16 * (a.rv_max + D_)) * sizeof(float), st, a); \
    return hipGetLastError(); }
  L_(32) L_(64) L_(128)
#undef L_
  return hipErrorInvalidValue;
}

// Fixed device scratch of jolt_attend_noalloc: the attention workspace of callers that
// cannot allocate device memory.  One array per device that loads the library, held until
// the process ends; every call on a device shares it.
static __device__ __align__(256) uint8_t scratch[ATTN_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void *g_scratch_dev[ATTN_SCRATCH_DEVICES] = {};
}  // namespace

// Device address of this device's scratch array, resolved once per device with
// hipGetSymbolAddress while that device is current (the array's name in host code is not a
// device address).
hipError_t attend_scratch_address(int device, void **ptr) {
  if (!ptr || device < 0 || device >= ATTN_SCRATCH_DEVICES) return hipErrorInvalidValue;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_dev[device] = p;
  }
  *ptr = g_scratch_dev[device];
  return hipSuccess;
}

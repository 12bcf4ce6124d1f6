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
// over 64-token chunks of one item (scores, a chunk-local softmax, and the value-side sums
// of U_T rows and dequantised codes, weighted by the unnormalised probabilities, for all
// query heads of the item at once); k_attend_combine
// merges the chunks with the usual max / rescale rule in a fixed order and applies the
// value factors and the inverse rotation once per query head.  Per token a query head
// reads r_T factor values and d codes instead of d decoded values plus the decompression.
#include <cmath>

#include "common.h"
#include "kernels.h"

namespace {

JOLT_DEV float factor(const void *p, int64_t i, int f16) {
  return f16 ? (float)reinterpret_cast<const _Float16 *>(p)[i] : reinterpret_cast<const float *>(p)[i];
}

// dequantised rotated residual r'[elem] = (code - (2^b - 1)/2) * scale
JOLT_DEV float dequant(const AttnBlob &b, int64_t elem, int group) {
  const int64_t bit = elem * b.bits;
  const uint32_t code = (b.codes[bit >> 3] >> (bit & 7)) & ((1u << b.bits) - 1u);
  const float delta = (float)(*reinterpret_cast<const _Float16 *>(b.scales + elem / group));
  return ((float)code - 0.5f * (float)((1 << b.bits) - 1)) * delta;
}

// eight dequantised values at elem, elem + 1, ... (elem a multiple of 8: one group, and
// the packed codes start on a 2-, 4- or 8-byte boundary for b = 2, 4, 8)
JOLT_DEV void dequant8(const AttnBlob &b, int64_t elem, int group, float (&v)[8]) {
  uint32_t c[8];
  if (b.bits == 2) {
    const uint32_t w = *reinterpret_cast<const uint16_t *>(b.codes + elem / 4);
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = (w >> (2 * i)) & 3u;
  } else if (b.bits == 4) {
    const uint32_t w = *reinterpret_cast<const uint32_t *>(b.codes + elem / 2);
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = (w >> (4 * i)) & 15u;
  } else {
    const uint2 w = *reinterpret_cast<const uint2 *>(b.codes + elem);
#pragma unroll
    for (int i = 0; i < 4; ++i) { c[i] = (w.x >> (8 * i)) & 255u; c[i + 4] = (w.y >> (8 * i)) & 255u; }
  }
  const float delta = (float)(*reinterpret_cast<const _Float16 *>(b.scales + elem / group));
  const float mid = 0.5f * (float)((1 << b.bits) - 1);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = ((float)c[i] - mid) * delta;
}

// Sylvester Hadamard entry (-1)^popcount(i & j)
JOLT_DEV float hsign(int i, int j) { return (__popc((unsigned)(i & j)) & 1) ? -1.f : 1.f; }

template <int D>
__global__ void __launch_bounds__(128) k_attend_prep(AttnArgs a) {
  const int item = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
  const AttnItem &it = a.items[item];
  const AttnBlob &kb = it.k;
  const int rep = a.n_q / a.heads, s = it.layer * a.heads + j / rep;
  __shared__ float q[D], qt[D];
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
  // q~ = U_d^T q, then g = 2^e_s G_s q~
  for (int k = tid; k < kb.rd; k += 128) {
    float acc = 0.f;
    for (int f = 0; f < D; ++f) acc = fmaf(factor(kb.Ud, (int64_t)f * kb.rd + k, kb.f16), q[f], acc);
    qt[k] = acc;
  }
  __syncthreads();
  float *gk = a.gk + ((int64_t)item * a.n_q + j) * a.rk_max;
  const float e = kb.rT ? ldexpf(1.f, (int)kb.gexp[s]) : 0.f;
  const int64_t g0 = (int64_t)s * kb.rT * kb.rd;
  for (int i = tid; i < kb.rT; i += 128) {
    float acc = 0.f;
    for (int k = 0; k < kb.rd; ++k) acc = fmaf(factor(kb.G, g0 + (int64_t)i * kb.rd + k, kb.f16), qt[k], acc);
    gk[i] = e * acc;
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

// Chunk pass.  Every token row of U_T and every (slice, token) row of codes is read once
// per workgroup and applied to all query heads that use it:
//   1. low-rank key scores: thread (token, block of 16 heads), U_T rows against g staged
//      in LDS 128 ranks at a time;
//   2. residual key scores: thread (slice, token) dequantises the row once and dots it
//      with the rotated queries of the slice's heads;
//   3. chunk-local softmax per head (a wave per head, a lane per token);
//   4. value low-rank sums: thread per rank i, all heads at once;
//   5. value residual sums: thread (slice, feature), the slice's heads at once.
template <int D>
__global__ void __launch_bounds__(256) k_attend_chunk(AttnArgs a) {
  constexpr int CH = ATTN_CHUNK, IB = 32, QMAX = ATTN_QMAX, RMAX = ATTN_REP_MAX;
  const int chunk = blockIdx.x, item = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const AttnItem &it = a.items[item];
  const AttnBlob &kb = it.k, &vb = it.v;
  const int T = a.T, t0 = chunk * CH, nt = min(CH, T - t0);
  const int nq = a.n_q, H = a.heads, rep = nq / H;
  // LDS kept small (about 25 KB) so that several workgroups share a CU
  __shared__ float gks[QMAX][IB];
  __shared__ __attribute__((aligned(16))) float pt[CH][QMAX + 4];   // scores, then probabilities
  const float *qrg = a.qr + (int64_t)item * nq * D;   // rotated queries (lanes of a wave share rows)
  // 1. low-rank key scores
  {
    const int t = tid % CH, jb = tid / CH;       // heads jb*16 .. jb*16 + 15
    float acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.f;
    const bool vec = (kb.rT % 8) == 0;
    for (int i0 = 0; i0 < kb.rT; i0 += IB) {
      const int ni = min(IB, kb.rT - i0);
      __syncthreads();
      for (int q = tid; q < nq * ni; q += 256)
        gks[q / ni][q % ni] = a.gk[((int64_t)item * nq + q / ni) * a.rk_max + i0 + q % ni];
      __syncthreads();
      if (t < nt && jb * 16 < nq) {
        const int64_t u0 = (int64_t)(t0 + t) * kb.rT + i0;
        for (int i = 0; i < ni; i += 8) {
          float u[8];
          if (i + 8 <= ni) factor8(kb.UT, u0 + i, kb.f16, vec, u);
          else {
#pragma unroll
            for (int k = 0; k < 8; ++k) u[k] = i + k < ni ? factor(kb.UT, u0 + i + k, kb.f16) : 0.f;
          }
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            if (i + k >= ni) break;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) acc[jj] = fmaf(u[k], gks[min(jb * 16 + jj, QMAX - 1)][i + k], acc[jj]);
          }
        }
      }
    }
    __syncthreads();
    if (jb * 16 < nq) {
#pragma unroll
      for (int jj = 0; jj < 16; ++jj)
        if (jb * 16 + jj < nq) pt[t][jb * 16 + jj] = acc[jj];
    }
  }
  __syncthreads();
  // 2. residual key scores
  if (kb.bits) {
    for (int q = tid; q < H * CH; q += 256) {
      const int h = q / CH, t = q % CH;
      if (t >= nt) continue;
      const int s = it.layer * H + h;
      const int64_t e0 = ((int64_t)s * T + t0 + t) * D;
      float res[RMAX];
#pragma unroll
      for (int r = 0; r < RMAX; ++r) res[r] = 0.f;
      for (int f = 0; f < D; f += 8) {
        float v[8];
        dequant8(kb, e0 + f, a.group, v);
#pragma unroll
        for (int r = 0; r < RMAX; ++r) {
          if (r < rep) {
            const float *qv = qrg + (int64_t)(h * rep + r) * D + f;
            const jf4 x = gload_f4(qv), y = gload_f4(qv + 4);
            float acc = res[r];
            acc = fmaf(v[0], x.x, acc); acc = fmaf(v[1], x.y, acc);
            acc = fmaf(v[2], x.z, acc); acc = fmaf(v[3], x.w, acc);
            acc = fmaf(v[4], y.x, acc); acc = fmaf(v[5], y.y, acc);
            acc = fmaf(v[6], y.z, acc); acc = fmaf(v[7], y.w, acc);
            res[r] = acc;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < RMAX; ++r)
        if (r < rep) pt[t][h * rep + r] += res[r];
    }
  }
  __syncthreads();
  // 3. chunk-local softmax per head
  const int stride = 2 + a.rv_max + D;
  float *part = a.part + ((int64_t)item * a.chunks + chunk) * nq * stride;
  for (int j = wave; j < nq; j += 4) {
    const float v = lane < nt ? pt[lane][j] * a.scale : -INFINITY;
    float mx = v;
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    const float e = lane < nt ? expf(v - mx) : 0.f;
    float sum = e;
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
    pt[lane][j] = e;
    if (lane == 0) { part[(int64_t)j * stride] = mx; part[(int64_t)j * stride + 1] = sum; }
  }
  __syncthreads();
  // 4. value low-rank sums a[j][i] = sum_t p[j][t] U_T^V[t][i], sixteen heads per pass
  for (int q = tid; q < vb.rT * ((nq + 15) / 16); q += 256) {
    const int i = q % vb.rT, j0 = (q / vb.rT) * 16;
    float acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = 0.f;
    // eight tokens' loads are issued before they are consumed
    for (int tb = 0; tb < nt; tb += 8) {
      float u[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        u[k] = tb + k < nt ? factor(vb.UT, (int64_t)(t0 + tb + k) * vb.rT + i, vb.f16) : 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
#pragma unroll
        for (int j4 = 0; j4 < 16; j4 += 4) {
          const float4 w = *reinterpret_cast<const float4 *>(&pt[min(tb + k, CH - 1)][j0 + j4]);
          acc[j4] = fmaf(w.x, u[k], acc[j4]); acc[j4 + 1] = fmaf(w.y, u[k], acc[j4 + 1]);
          acc[j4 + 2] = fmaf(w.z, u[k], acc[j4 + 2]); acc[j4 + 3] = fmaf(w.w, u[k], acc[j4 + 3]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (j0 + j < nq) part[(int64_t)(j0 + j) * stride + 2 + i] = acc[j];
  }
  // 5. value residual sums b[j][f] = sum_t p[j][t] r'_s[t][f]
  for (int q = tid; q < H * D; q += 256) {
    const int h = q / D, f = q % D;
    float acc[RMAX];
#pragma unroll
    for (int r = 0; r < RMAX; ++r) acc[r] = 0.f;
    if (vb.bits) {
      const int s = it.layer * H + h;
      for (int tb = 0; tb < nt; tb += 8) {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
          v[k] = tb + k < nt ? dequant(vb, ((int64_t)s * T + t0 + tb + k) * D + f, a.group) : 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          if (tb + k >= nt) break;
#pragma unroll
          for (int r = 0; r < RMAX; ++r)
            if (r < rep) acc[r] = fmaf(pt[tb + k][h * rep + r], v[k], acc[r]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RMAX; ++r)
      if (r < rep) part[(int64_t)(h * rep + r) * stride + 2 + a.rv_max + f] = acc[r];
  }
}

template <int D>
__global__ void __launch_bounds__(128) k_attend_combine(AttnArgs a) {
  const int item = blockIdx.x, j = blockIdx.y, tid = threadIdx.x;
  const AttnItem &it = a.items[item];
  const AttnBlob &vb = it.v;
  const int rep = a.n_q / a.heads, s = it.layer * a.heads + j / rep;
  const int stride = 2 + a.rv_max + D;
  const float *part = a.part + ((int64_t)item * a.chunks * a.n_q + j) * stride;
  const int64_t cstride = (int64_t)a.n_q * stride;
  __shared__ float av[ATTN_RT_MAX], w[D], bv[D];
  __shared__ float L_s;
  extern __shared__ float cw[];                 // per-chunk weights exp(max_c - M)
  if (tid == 0) {
    float M = -INFINITY;
    for (int c = 0; c < a.chunks; ++c) M = fmaxf(M, part[c * cstride]);
    float L = 0.f;
    for (int c = 0; c < a.chunks; ++c) {
      cw[c] = expf(part[c * cstride] - M);
      L += part[c * cstride + 1] * cw[c];
    }
    L_s = L;
  }
  __syncthreads();
  for (int i = tid; i < vb.rT + D; i += 128) {
    float acc = 0.f;
    const float *pc = part + 2 + (i < vb.rT ? i : a.rv_max + (i - vb.rT));
    for (int c = 0; c < a.chunks; ++c) acc = fmaf(cw[c], pc[c * cstride], acc);
    if (i < vb.rT) av[i] = acc;
    else bv[i - vb.rT] = acc;
  }
  __syncthreads();
  // w = 2^e_s (a^T G_s): r_d values
  const float e = vb.rT ? ldexpf(1.f, (int)vb.gexp[s]) : 0.f;
  const int64_t g0 = (int64_t)s * vb.rT * vb.rd;
  for (int k = tid; k < vb.rd; k += 128) {
    float acc = 0.f;
    for (int i = 0; i < vb.rT; ++i) acc = fmaf(av[i], factor(vb.G, g0 + (int64_t)i * vb.rd + k, vb.f16), acc);
    w[k] = e * acc;
  }
  __syncthreads();
  const float *sg = a.signs + ((int64_t)item * 2 + 1) * D;
  float *o = a.O + ((int64_t)item * a.n_q + j) * D;
  const float invL = 1.f / L_s;
  for (int f = tid; f < D; f += 128) {
    float lr = 0.f;
    for (int k = 0; k < vb.rd; ++k) lr = fmaf(factor(vb.Ud, (int64_t)f * vb.rd + k, vb.f16), w[k], lr);
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
    hipLaunchKernelGGL((k_attend_chunk<D_>), dim3(a.chunks, a.n_items), dim3(256), 0, st, a); \
    hipLaunchKernelGGL((k_attend_combine<D_>), dim3(a.n_items, a.n_q), dim3(128), a.chunks * sizeof(float), st, a); \
    return hipGetLastError(); }
  L_(32) L_(64) L_(128)
#undef L_
  return hipErrorInvalidValue;
}

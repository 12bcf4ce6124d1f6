// Per-row operations of the rotated low-bit residual (section 4, "Rotated residual"),
// shared by the streaming residual / decode kernels and the fused reconstruction kernels.
//
// Layout on the wavefront: a feature row of D entries is held by D/8 consecutive lanes,
// 8 contiguous entries per lane, so one wave64 processes 512/D rows at a time.  The
// Walsh-Hadamard transform runs its first three butterfly stages inside the lane and the
// remaining log2(D/8) stages across lanes (DPP within the 16-lane row).  A quantiser group
// of g entries spans g/8 lanes; its max is a reduction over them.
#pragma once
#include "common.h"

namespace rowops {

template <int D>
struct RowLayout {
  static constexpr int L = D / 8;        // lanes per row
  static constexpr int R = 64 / L;       // rows per wave
};

// Value held by lane `lane ^ M`.  For M < 16 the partner lies in the same row of 16 lanes and
// DPP reads it inside the ALU (quad permutes for M = 1, 2; row shifts left / right by M,
// picked by the lane's bit M, for M = 4, 8); wider distances go through the LDS crossbar.
template <int M>
JOLT_DEV float xor_lane(float v, int lane) {
  const int x = __float_as_int(v);
  if constexpr (M == 1) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0xB1, 0xf, 0xf, false));   // [1,0,3,2]
  } else if constexpr (M == 2) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x4E, 0xf, 0xf, false));   // [2,3,0,1]
  } else if constexpr (M == 4 || M == 8) {
    const int from_hi = __builtin_amdgcn_update_dpp(0, x, 0x100 + M, 0xf, 0xf, false);  // lane + M
    const int from_lo = __builtin_amdgcn_update_dpp(0, x, 0x110 + M, 0xf, 0xf, false);  // lane - M
    return __int_as_float((lane & M) ? from_lo : from_hi);
  } else {
    return __shfl_xor(v, M, 64);
  }
}

// one butterfly stage across lanes at distance M: lower lane a + b, upper lane a' - b'
template <int M>
JOLT_DEV void xstage(float (&v)[8], int lane_in_row) {
  const bool upper = (lane_in_row & M) != 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float p = xor_lane<M>(v[i], lane_in_row);
    v[i] = upper ? (p - v[i]) : (v[i] + p);
  }
}

// max over the gl lanes of a quantiser group (gl a power of two, at most 64)
JOLT_DEV float group_max(float a, int gl, int lane) {
  if (gl > 1) a = fmaxf(a, xor_lane<1>(a, lane));
  if (gl > 2) a = fmaxf(a, xor_lane<2>(a, lane));
  if (gl > 4) a = fmaxf(a, xor_lane<4>(a, lane));
  if (gl > 8) a = fmaxf(a, xor_lane<8>(a, lane));
  if (gl > 16) a = fmaxf(a, xor_lane<16>(a, lane));
  if (gl > 32) a = fmaxf(a, xor_lane<32>(a, lane));
  return a;
}

// Rotary embedding of one decoded row spread over L lanes (8 features each): features j and
// j + D/2 sit in lanes l and l + L/2 and rotate together by the angle pos * theta_j, formed
// and reduced in fp64.
template <int D>
JOLT_DEV void rope_row(float (&v)[8], int lane_in_row, double pos, const double (&theta)[8]) {
  constexpr int L = RowLayout<D>::L;
  const bool upper = lane_in_row >= L / 2;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float partner = xor_lane<L / 2>(v[i], lane_in_row);
    double sn, cs;
    sincos(pos * theta[i], &sn, &cs);
    const float c = (float)cs, s = (float)sn;
    v[i] = upper ? fmaf(partner, s, v[i] * c) : fmaf(-partner, s, v[i] * c);
  }
}

// in-place Walsh-Hadamard transform of the D-entry row spread over L lanes
template <int D>
JOLT_DEV void fwht_row(float (&v)[8], int lane_in_row) {
#pragma unroll
  for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if ((i & h) == 0) {
        float a = v[i], b = v[i + h];
        v[i] = a + b;
        v[i + h] = a - b;
      }
    }
  }
  constexpr int L = RowLayout<D>::L;
  if constexpr (L > 1) xstage<1>(v, lane_in_row);
  if constexpr (L > 2) xstage<2>(v, lane_in_row);
  if constexpr (L > 4) xstage<4>(v, lane_in_row);
  if constexpr (L > 8) xstage<8>(v, lane_in_row);
  if constexpr (L > 16) xstage<16>(v, lane_in_row);
  if constexpr (L > 32) xstage<32>(v, lane_in_row);
}

template <typename T>
JOLT_DEV void load8(const T *p, float (&v)[8]);

template <>
JOLT_DEV void load8<bf16_t>(const bf16_t *p, float (&v)[8]) {
  uint4 u = *reinterpret_cast<const uint4 *>(p);
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_to_f32((bf16_t)(w[i] & 0xffffu));
    v[2 * i + 1] = bf16_to_f32((bf16_t)(w[i] >> 16));
  }
}

template <>
JOLT_DEV void load8<float>(const float *p, float (&v)[8]) {
  float4 a = *reinterpret_cast<const float4 *>(p);
  float4 b = *reinterpret_cast<const float4 *>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

JOLT_DEV void store8(bf16_t *p, const float (&v)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = (uint32_t)f32_to_bf16(v[2 * i]) | ((uint32_t)f32_to_bf16(v[2 * i + 1]) << 16);
  *reinterpret_cast<uint4 *>(p) = uint4{w[0], w[1], w[2], w[3]};
}

JOLT_DEV void store8(float *p, const float (&v)[8]) {
  *reinterpret_cast<float4 *>(p) = float4{v[0], v[1], v[2], v[3]};
  *reinterpret_cast<float4 *>(p + 4) = float4{v[4], v[5], v[6], v[7]};
}

// Quantise 8 rotated entries of one lane; group max over gl = g/8 lanes.
JOLT_DEV void quantize8(const float (&r)[8], int bits, int gl, int lane_in_row, uint32_t (&code)[8],
                        float &delta) {
  float a = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(r[i]));
  a = group_max(a, gl, lane_in_row);
  const int levels = (1 << bits) - 1;
  float dl = 2.f * a / (float)levels;
  dl = fminf(dl, 65504.f);
  delta = f16_round(dl);
  const float mid = 0.5f * (float)levels;
  // r / delta as r * (1 / delta): within 1.5 ulp of the quotient, so a code moves only when
  // the quotient lies that close to a rounding boundary
  const float inv = delta == 0.f ? 0.f : 1.f / delta;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float c;
    if (delta == 0.f) {
      c = (float)(1 << (bits - 1));
    } else {
      c = __builtin_rintf(fmaf(r[i], inv, mid));
      c = fminf(fmaxf(c, 0.f), (float)levels);
    }
    code[i] = (uint32_t)c;
  }
}

JOLT_DEV void store_codes(uint8_t *codes, int64_t elem, int bits, const uint32_t (&c)[8]) {
  if (bits == 2) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) w |= c[i] << (2 * i);
    *reinterpret_cast<uint16_t *>(codes + elem / 4) = (uint16_t)w;
  } else if (bits == 4) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) w |= c[i] << (4 * i);
    *reinterpret_cast<uint32_t *>(codes + elem / 2) = w;
  } else {
    uint32_t lo = c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24);
    uint32_t hi = c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24);
    *reinterpret_cast<uint2 *>(codes + elem) = uint2{lo, hi};
  }
}

JOLT_DEV void load_codes(const uint8_t *codes, int64_t elem, int bits, uint32_t (&c)[8]) {
  if (bits == 2) {
    uint32_t w = *reinterpret_cast<const uint16_t *>(codes + elem / 4);
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = (w >> (2 * i)) & 3u;
  } else if (bits == 4) {
    uint32_t w = *reinterpret_cast<const uint32_t *>(codes + elem / 2);
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = (w >> (4 * i)) & 15u;
  } else {
    uint2 w = *reinterpret_cast<const uint2 *>(codes + elem);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c[i] = (w.x >> (8 * i)) & 255u;
      c[i + 4] = (w.y >> (8 * i)) & 255u;
    }
  }
}

}  // namespace rowops

// Per-row operations of the rotated low-bit residual (section 4, "Rotated residual"),
// shared by the streaming residual / decode kernels and the fused reconstruction kernels.
//
// Layout on the wavefront: a feature row of D entries is held by D/8 consecutive lanes,
// 8 contiguous entries per lane, so one wave64 processes 512/D rows at a time.  The
// Walsh-Hadamard transform runs its first three butterfly stages inside the lane and the
// remaining log2(D/8) stages across lanes with xor shuffles.  A quantiser group of g
// entries spans g/8 lanes; its max is a shuffle reduction.
#pragma once
#include "common.h"

namespace rowops {

template <int D>
struct RowLayout {
  static constexpr int L = D / 8;        // lanes per row
  static constexpr int R = 64 / L;       // rows per wave
};

// Rotary embedding of one decoded row spread over L lanes (8 features each): features j and
// j + D/2 sit in lanes l and l + L/2 and rotate together by the angle pos * theta_j, formed
// and reduced in fp64.
template <int D>
JOLT_DEV void rope_row(float (&v)[8], int lane_in_row, double pos, const double (&theta)[8]) {
  constexpr int L = RowLayout<D>::L;
  const bool upper = lane_in_row >= L / 2;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float partner = shfl_xor(v[i], L / 2);
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
#pragma unroll
  for (int lm = 1; lm < RowLayout<D>::L; lm <<= 1) {
    const bool upper = (lane_in_row & lm) != 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float p = shfl_xor(v[i], lm);
      v[i] = upper ? (p - v[i]) : (v[i] + p);
    }
  }
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
JOLT_DEV void quantize8(const float (&r)[8], int bits, int gl, uint32_t (&code)[8], float &delta) {
  float a = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) a = fmaxf(a, fabsf(r[i]));
  for (int m = 1; m < gl; m <<= 1) a = fmaxf(a, shfl_xor(a, m));
  const int levels = (1 << bits) - 1;
  float dl = 2.f * a / (float)levels;
  dl = fminf(dl, 65504.f);
  delta = f16_round(dl);
  const float mid = 0.5f * (float)levels;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float c;
    if (delta == 0.f) {
      c = (float)(1 << (bits - 1));
    } else {
      c = __builtin_rintf(r[i] / delta + mid);
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

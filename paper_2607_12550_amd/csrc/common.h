// Shared device helpers for the gfx950 kernels: number formats, Philox4x32-10,
// wavefront shuffles and small utilities.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define JOLT_DEV __device__ __forceinline__
#define JOLT_HD __host__ __device__ __forceinline__

typedef uint16_t bf16_t;  // bf16 bit pattern

// Global-memory views of generic pointers: loads and stores through them compile to
// global_* instructions (waited on by vmcnt alone) instead of flat_* ones, which also
// hold lgkmcnt and so serialise against LDS traffic.
#define JOLT_GLOBAL __attribute__((address_space(1)))
template <class T>
JOLT_DEV const JOLT_GLOBAL T *gptr(const T *p) { return (const JOLT_GLOBAL T *)p; }
template <class T>
JOLT_DEV JOLT_GLOBAL T *gptr(T *p) { return (JOLT_GLOBAL T *)p; }
typedef float jf4 __attribute__((ext_vector_type(4)));
typedef uint32_t ju4 __attribute__((ext_vector_type(4)));
JOLT_DEV jf4 gload_f4(const void *p) { return *(const JOLT_GLOBAL jf4 *)p; }
JOLT_DEV ju4 gload_u4(const void *p) { return *(const JOLT_GLOBAL ju4 *)p; }
JOLT_DEV void gstore_f4(void *p, jf4 v) { *(JOLT_GLOBAL jf4 *)p = v; }

// ---------------------------------------------------------------- number formats
JOLT_HD float bf16_to_f32(bf16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

// fp32 -> bf16, round to nearest even (NaN stays NaN)
JOLT_HD bf16_t f32_to_bf16(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// fp64 -> bf16 with a single round to nearest even (no intermediate fp32 rounding).
JOLT_DEV bf16_t f64_to_bf16(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  uint64_t sign = u >> 63;
  int e = (int)((u >> 52) & 0x7ff) - 1023;       // unbiased exponent (finite input)
  if (e < -133 - 1) return (bf16_t)(sign << 15);   // below half the smallest subnormal
  // keep 7 fraction bits for normal bf16 (e >= -126), fewer for subnormals
  int drop = 45 + (e < -126 ? (-126 - e) : 0);
  uint64_t mant = (u & 0xfffffffffffffull) | (1ull << 52);
  uint64_t half = 1ull << (drop - 1);
  uint64_t rem = mant & ((1ull << drop) - 1);
  uint64_t q = mant >> drop;
  if (rem > half || (rem == half && (q & 1))) q += 1;
  // value = q * 2^(e - 52 + drop); rebuild as a float (exact: q < 2^9)
  float v = ldexpf((float)q, e - 52 + drop);
  uint32_t fb;
  __builtin_memcpy(&fb, &v, 4);
  return (bf16_t)((fb >> 16) | (uint32_t)(sign << 15));
}

JOLT_DEV float f16_round(float x) { return (float)(_Float16)x; }

// ---------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC 2011).
struct u32x4 { uint32_t x, y, z, w; };

JOLT_HD u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = u32x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

enum { STREAM_SIGN = 1, STREAM_SKETCH = 2, STREAM_CALIB = 3 };

// Box-Muller (cosine branch) in fp64 from two 32-bit words; u = (w + 1/2) 2^-32.
JOLT_DEV double box_muller_f64(uint32_t w0, uint32_t w1) {
  double u0 = ((double)w0 + 0.5) * 0x1p-32;
  double u1 = ((double)w1 + 0.5) * 0x1p-32;
  return sqrt(-2.0 * log(u0)) * cos((2.0 * 3.141592653589793) * u1);
}

// ---------------------------------------------------------------- wavefront shuffles
JOLT_DEV float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, 64); }
JOLT_DEV double shfl_xor(double v, int mask) { return __shfl_xor(v, mask, 64); }

JOLT_DEV double wave_sum(double v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
JOLT_DEV float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// ---------------------------------------------------------------- cell addressing
// Element (s, t, f) of a cell: base + (s / heads) * s_layer + (s % heads) * s_head + t * s_tok + f
struct CellView {
  const void *base;
  int64_t s_layer, s_head, s_tok;
  int32_t heads;
  JOLT_DEV int64_t row_off(int s, int t) const {
    return (int64_t)(s / heads) * s_layer + (int64_t)(s % heads) * s_head + (int64_t)t * s_tok;
  }
};

// Rotated low-bit residual: streaming kernels (section 4, "Rotated residual").
//
//   compress: R = X - X~, r' = H_d (s * r) / sqrt(d) per feature row, one fp16 scale
//             Delta = fp16(2 max|r'| / (2^b - 1)) per group of g entries,
//             code = clip(rint(r'/Delta + (2^b-1)/2), 0, 2^b-1), packed LSB-first.
//   decode:   X^ = X~ + s * H_d((code - (2^b-1)/2) Delta) / sqrt(d), cast to the output type.
//
// Layout on the wavefront: a feature row of D entries is held by D/8 consecutive
// lanes, 8 contiguous entries per lane (one 16-byte bf16 load or two 16-byte fp32
// loads), so one wave64 processes 512/D rows at a time.  The Walsh-Hadamard
// transform runs its first three butterfly stages inside the lane and the remaining
// log2(D/8) stages across lanes with xor shuffles.  A quantiser group of g entries
// spans g/8 lanes; its max is a shuffle reduction.  Every row is read once and the
// codes and scales are written once: the kernels are HBM-bound.
#include "common.h"
#include "kernels.h"

namespace {

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

// One wave handles R rows of a single cell per iteration; rows of a cell are
// grouped as ceil(m*T / R) row blocks so a wave never straddles two cells.
template <int D, typename TX>
__global__ void __launch_bounds__(256) k_residual_quant(ResidArgs a) {
  constexpr int L = RowLayout<D>::L, R = RowLayout<D>::R;
  const int lane = threadIdx.x & 63;
  const int row_in_wave = lane / L, lane_in_row = lane % L;
  const int64_t rows_per_cell = (int64_t)a.m * a.T;
  const int64_t blocks_per_cell = (rows_per_cell + R - 1) / R;
  const int64_t total = blocks_per_cell * a.n_cells;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const float inv_sqrt_d = a.inv_sqrt_d;
  const int gl = a.group / 8;
  for (int64_t wb = wave0; wb < total; wb += nwaves) {
    const int cell = (int)(wb / blocks_per_cell);
    const int64_t row = (wb % blocks_per_cell) * R + row_in_wave;
    const ResidCell &c = a.cells[cell];
    if (row >= rows_per_cell || c.bits == 0) continue;   // uniform per wave except the tail
    const int s = (int)(row / a.T), t = (int)(row % a.T);
    const TX *x = reinterpret_cast<const TX *>(c.x) +
                  ((int64_t)(s / a.heads) * a.s_layer + (int64_t)(s % a.heads) * a.s_head +
                   (int64_t)t * a.s_tok) + lane_in_row * 8;
    float v[8];
    load8<TX>(x, v);
    if (c.xt) {
      float xt[8];
      load8<float>(c.xt + row * D + lane_in_row * 8, xt);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] -= xt[i];
    }
    const float *sg = a.signs + (int64_t)cell * D + lane_in_row * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] *= sg[i];
    fwht_row<D>(v, lane_in_row);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] *= inv_sqrt_d;
    uint32_t code[8];
    float delta;
    quantize8(v, c.bits, gl, code, delta);
    const int64_t elem = row * D + lane_in_row * 8;
    store_codes(c.codes, elem, c.bits, code);
    if ((lane_in_row % gl) == 0) {
      _Float16 h = (_Float16)delta;
      uint16_t hb;
      __builtin_memcpy(&hb, &h, 2);
      c.scales[elem / a.group] = hb;
    }
  }
}

template <int D, typename TO, bool ROPE>
__global__ void __launch_bounds__(256) k_decode(DecodeArgs a) {
  constexpr int L = RowLayout<D>::L, R = RowLayout<D>::R;
  const int lane = threadIdx.x & 63;
  const int row_in_wave = lane / L, lane_in_row = lane % L;
  // rotary frequencies of this lane's 8 features: base^(-2 j / D), j = feature mod D/2
  double theta[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int j = (lane_in_row * 8 + i) % (D / 2);
    theta[i] = ROPE ? exp2(-(2.0 * j / D) * a.rope_log2_base) : 0.0;
  }
  const int64_t rows_per_cell = (int64_t)a.m * a.T;
  const int64_t blocks_per_cell = (rows_per_cell + R - 1) / R;
  const int64_t total = blocks_per_cell * a.n_cells;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t wb = wave0; wb < total; wb += nwaves) {
    const int cell = (int)(wb / blocks_per_cell);
    const int64_t row = (wb % blocks_per_cell) * R + row_in_wave;
    const DecodeCell &c = a.cells[cell];
    if (row >= rows_per_cell) continue;
    const int s = (int)(row / a.T), t = (int)(row % a.T);
    const int64_t elem = row * D + lane_in_row * 8;
    float v[8];
    if (c.bits) {
      uint32_t code[8];
      load_codes(c.codes, elem, c.bits, code);
      const float delta = (float)(*reinterpret_cast<const _Float16 *>(c.scales + elem / a.group));
      const float mid = 0.5f * (float)((1 << c.bits) - 1);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = ((float)code[i] - mid) * delta;
      fwht_row<D>(v, lane_in_row);
      const float *sg = a.signs + (int64_t)cell * D + lane_in_row * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = sg[i] * (v[i] * a.inv_sqrt_d);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = 0.f;
    }
    if (c.xt) {
      float xt[8];
      load8<float>(c.xt + row * D + lane_in_row * 8, xt);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = xt[i] + v[i];
    }
    if constexpr (ROPE) rope_row<D>(v, lane_in_row, (double)(t + a.rope_offset), theta);
    TO *o = reinterpret_cast<TO *>(c.out) +
            ((int64_t)(s / a.heads) * a.s_layer + (int64_t)(s % a.heads) * a.s_head +
             (int64_t)t * a.s_tok) + lane_in_row * 8;
    store8(o, v);
  }
}

// Rademacher signs of the rotation: s_j = +1 if bit 0 of word 0 of
// philox((j, 0, 0, STREAM_SIGN), seed) is 0, else -1.
__global__ void k_rotation_signs(const uint64_t *seeds, int n_cells, int d, float *signs) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_cells * d) return;
  int cell = i / d, j = i % d;
  uint64_t sd = seeds[cell];
  u32x4 w = philox4x32_10(u32x4{(uint32_t)j, 0u, 0u, (uint32_t)STREAM_SIGN}, (uint32_t)sd,
                          (uint32_t)(sd >> 32));
  signs[i] = (w.x & 1u) ? -1.f : 1.f;
}

// eq. (2) calibration: Gaussian rows (Philox stream 3, fp64 Box-Muller rounded to fp32)
// go through rotate -> quantise -> dequantise -> unrotate for b = 2, 4, 8; each block
// writes fp64 partial sums [sum x^2, sum err_2^2, sum err_4^2, sum err_8^2].
template <int D>
__global__ void __launch_bounds__(256) k_eps2_partial(Eps2Args a) {
  constexpr int L = RowLayout<D>::L, R = RowLayout<D>::R;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row_in_wave = lane / L, lane_in_row = lane % L;
  const int64_t rows = a.n_samples / D;
  const int64_t nblocks_rows = (rows + R - 1) / R;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  double acc[4] = {0, 0, 0, 0};
  float sg[8];
  for (int i = 0; i < 8; ++i) {
    int j = lane_in_row * 8 + i;
    u32x4 w = philox4x32_10(u32x4{(uint32_t)j, 0u, 0u, (uint32_t)STREAM_SIGN},
                            (uint32_t)a.seed, (uint32_t)(a.seed >> 32));
    sg[i] = (w.x & 1u) ? -1.f : 1.f;
  }
  const int gl = a.group / 8;
  for (int64_t wb = wave0; wb < nblocks_rows; wb += nwaves) {
    const int64_t row = wb * R + row_in_wave;
    if (row >= rows) continue;
    float x[8], v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint64_t k = (uint64_t)row * D + lane_in_row * 8 + i;
      u32x4 w = philox4x32_10(u32x4{(uint32_t)k, (uint32_t)(k >> 32), 0u, (uint32_t)STREAM_CALIB},
                              (uint32_t)a.seed, (uint32_t)(a.seed >> 32));
      x[i] = (float)box_muller_f64(w.x, w.y);
      acc[0] += (double)x[i] * (double)x[i];
      v[i] = x[i] * sg[i];
    }
    fwht_row<D>(v, lane_in_row);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] *= a.inv_sqrt_d;
#pragma unroll
    for (int bi = 0; bi < 3; ++bi) {
      const int bits = 2 << bi;
      uint32_t code[8];
      float delta;
      quantize8(v, bits, gl, code, delta);
      const float mid = 0.5f * (float)((1 << bits) - 1);
      float y[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) y[i] = ((float)code[i] - mid) * delta;
      fwht_row<D>(y, lane_in_row);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        double e = (double)(sg[i] * (y[i] * a.inv_sqrt_d)) - (double)x[i];
        acc[1 + bi] += e * e;
      }
    }
  }
  __shared__ double red[4][4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    double v = wave_sum(acc[k]);
    if (lane == 0) red[wave][k] = v;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    double v = red[0][threadIdx.x] + red[1][threadIdx.x] + red[2][threadIdx.x] + red[3][threadIdx.x];
    a.partials[(int64_t)blockIdx.x * 4 + threadIdx.x] = v;
  }
}

int grid_for(int64_t waves_needed) {
  int64_t blocks = (waves_needed + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  return (int)blocks;
}

}  // namespace

#define DISPATCH_D(D, ...)                              \
  switch (D) {                                          \
    case 32: { constexpr int DD = 32; __VA_ARGS__; } break;   \
    case 64: { constexpr int DD = 64; __VA_ARGS__; } break;   \
    case 128: { constexpr int DD = 128; __VA_ARGS__; } break; \
    case 256: { constexpr int DD = 256; __VA_ARGS__; } break; \
    default: return hipErrorInvalidValue;               \
  }

hipError_t launch_residual_quant(const ResidArgs &a, int d, int in_dtype, hipStream_t st) {
  const int R = 64 / (d / 8);
  int64_t waves = ((int64_t)a.m * a.T + R - 1) / R * a.n_cells;
  int grid = grid_for(waves);
  DISPATCH_D(d, {
    if (in_dtype == 1)
      hipLaunchKernelGGL((k_residual_quant<DD, bf16_t>), dim3(grid), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((k_residual_quant<DD, float>), dim3(grid), dim3(256), 0, st, a);
  });
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs &a, int d, int out_dtype, hipStream_t st) {
  const int R = 64 / (d / 8);
  int64_t waves = ((int64_t)a.m * a.T + R - 1) / R * a.n_cells;
  int grid = grid_for(waves);
  DISPATCH_D(d, {
    if (out_dtype == 1 && a.rope)
      hipLaunchKernelGGL((k_decode<DD, bf16_t, true>), dim3(grid), dim3(256), 0, st, a);
    else if (out_dtype == 1)
      hipLaunchKernelGGL((k_decode<DD, bf16_t, false>), dim3(grid), dim3(256), 0, st, a);
    else if (a.rope)
      hipLaunchKernelGGL((k_decode<DD, float, true>), dim3(grid), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((k_decode<DD, float, false>), dim3(grid), dim3(256), 0, st, a);
  });
  return hipGetLastError();
}

hipError_t launch_rotation_signs(const uint64_t *seeds_dev, int n_cells, int d, float *signs,
                                 hipStream_t st) {
  int n = n_cells * d;
  hipLaunchKernelGGL(k_rotation_signs, dim3((n + 255) / 256), dim3(256), 0, st, seeds_dev,
                     n_cells, d, signs);
  return hipGetLastError();
}

int eps2_blocks() { return 1024; }

hipError_t launch_eps2_partial(const Eps2Args &a, int d, hipStream_t st) {
  DISPATCH_D(d, {
    hipLaunchKernelGGL((k_eps2_partial<DD>), dim3(eps2_blocks()), dim3(256), 0, st, a);
  });
  return hipGetLastError();
}

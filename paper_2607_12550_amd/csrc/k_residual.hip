// Rotated low-bit residual (section 4, "Rotated residual"): the rotation signs and the
// eq. (2) calibration of eps^2(b).  The residual and decode passes themselves run fused with
// the reconstruction (k_fused.hip); both use the per-row operations of rowops.h:
//
//   compress: R = X - X~, r' = H_d (s * r) / sqrt(d) per feature row, one fp16 scale
//             Delta = fp16(2 max|r'| / (2^b - 1)) per group of g entries,
//             code = clip(rint(r'/Delta + (2^b-1)/2), 0, 2^b-1), packed LSB-first.
//   decode:   X^ = X~ + s * H_d((code - (2^b-1)/2) Delta) / sqrt(d), cast to the output type.
#include "common.h"
#include "kernels.h"
#include "rowops.h"

namespace {
using namespace rowops;

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
      quantize8(v, bits, gl, lane_in_row, code, delta);
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

}  // namespace

#define DISPATCH_D(D, ...)                              \
  switch (D) {                                          \
    case 32: { constexpr int DD = 32; __VA_ARGS__; } break;   \
    case 64: { constexpr int DD = 64; __VA_ARGS__; } break;   \
    case 128: { constexpr int DD = 128; __VA_ARGS__; } break; \
    case 256: { constexpr int DD = 256; __VA_ARGS__; } break; \
    default: return hipErrorInvalidValue;               \
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

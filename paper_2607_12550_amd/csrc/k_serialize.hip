// Factor serialisation into the blob (eq. (1) prices factors at c bytes per scalar;
// section 9 uses fp16).  Each core slice G_s gets a power-of-two exponent
// e_s = max(-128, ceil(log2 max|G_s|) - 15) (0 for an all-zero slice) so that the stored
// fp16 values keep full precision and stay below 2^15; the floor keeps e_s in the blob's
// signed byte (it only binds for cores below 2^-113).  fp32 factors are copied unchanged
// with e_s = 0.
#include "common.h"
#include "kernels.h"

namespace {

JOLT_DEV uint16_t f32_to_f16_bits(float x) {
  _Float16 h = (_Float16)x;
  uint16_t b;
  __builtin_memcpy(&b, &h, 2);
  return b;
}

// exact ceil(log2(x)) for finite x > 0
JOLT_DEV int ceil_log2_f(float x) {
  int e;
  float f = frexpf(x, &e);       // x = f 2^e, 0.5 <= f < 1
  return f == 0.5f ? e - 1 : e;
}

// one workgroup per (slice, cell): exponent of the slice and its fp16/fp32 copy
__global__ void __launch_bounds__(256) k_core_pack(SerCore a) {
  const int s = blockIdx.x, cell = blockIdx.y;
  const SerCell &c = a.cells[cell];
  const int rT = c.r_T, rd = c.r_d;
  if (s >= a.m || rT == 0) return;
  const float *G = c.G + (int64_t)s * c.g_slice_stride;
  __shared__ float red[4];
  float mx = 0.f;
  for (int q = threadIdx.x; q < rT * rd; q += 256) {
    const int r = q / rd, k = q % rd;
    mx = fmaxf(mx, fabsf(G[(int64_t)r * c.g_ld + k]));
  }
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  int e = 0;
  if (c.f16 && mx > 0.f) e = max(-128, ceil_log2_f(mx) - 15);
  if (threadIdx.x == 0) c.gexp[s] = (int8_t)e;
  // the power of two is applied to each value (2^-e itself may lie outside fp32's range)
  for (int q = threadIdx.x; q < rT * rd; q += 256) {
    const int r = q / rd, k = q % rd;
    const float v = ldexpf(G[(int64_t)r * c.g_ld + k], -e);
    const int64_t o = ((int64_t)s * rT + r) * rd + k;
    if (c.f16) reinterpret_cast<uint16_t *>(c.G_out)[o] = f32_to_f16_bits(v);
    else reinterpret_cast<float *>(c.G_out)[o] = v;
  }
}

// dense factor (rows x cols from a strided fp32 source) into the blob
__global__ void k_factor_pack(SerFactor a) {
  const int cell = blockIdx.y;
  const SerFactorCell &c = a.cells[cell];
  const int64_t n = (int64_t)c.rows * c.cols;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = q / c.cols, k = q % c.cols;
    const float v = c.src[r * c.ld + k];
    if (c.f16) reinterpret_cast<uint16_t *>(c.dst)[q] = f32_to_f16_bits(v);
    else reinterpret_cast<float *>(c.dst)[q] = v;
  }
}

}  // namespace

hipError_t launch_core_pack(const SerCore &a, int n_cells, hipStream_t st) {
  hipLaunchKernelGGL(k_core_pack, dim3(a.m, n_cells), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_factor_pack(const SerFactor &a, int n_cells, int64_t max_elems, hipStream_t st) {
  if (max_elems <= 0) return hipSuccess;
  int64_t blocks = (max_elems + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_factor_pack, dim3((unsigned)blocks, n_cells), dim3(256), 0, st, a);
  return hipGetLastError();
}

// Achievable-peak microbenchmarks on gfx950, reported next to the spec peaks
// as a second roofline denominator:
//   * bf16 matrix-core rate: every wave keeps four independent
//     v_mfma_f32_32x32x16_bf16 accumulators busy (2 waves per SIMD on every
//     CU), so the result includes the clock the chip holds under full
//     matrix load;
//   * HBM read rate: a grid-stride stream of 16-byte loads over a buffer
//     much larger than the last-level cache.
#include "pic_internal.hpp"

namespace pic {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256, 2) void peak_mfma_kernel(float *out, int32_t iters) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(threadIdx.x * 0.001f + i);
    b[i] = (__bf16)(i * 0.5f);
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int i = 0; i < iters; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// Four independent 16-byte loads in flight per lane per trip.
__global__ __launch_bounds__(256) void peak_read_kernel(const uint4 *src, int64_t n16, float *out) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  out[blockIdx.x * blockDim.x + threadIdx.x] = (float)acc;
}

}  // namespace

// 512 workgroups x 4 waves: 2 waves per SIMD on all 256 CUs.
constexpr int kPeakBlocks = 512, kPeakThreads = 256;

int64_t peak_out_floats() { return (int64_t)kPeakBlocks * kPeakThreads; }

double peak_mfma_flops(int32_t iters) {
  return (double)kPeakBlocks * (kPeakThreads / 64) * iters * 4.0 * 32.0 * 32.0 * 16.0 * 2.0;
}

hipError_t launch_peak_mfma(float *out, int32_t iters, hipStream_t st) {
  hipLaunchKernelGGL(peak_mfma_kernel, dim3(kPeakBlocks), dim3(kPeakThreads), 0, st, out, iters);
  return hipGetLastError();
}

hipError_t launch_peak_read(const void *src, int64_t bytes, float *out, hipStream_t st) {
  hipLaunchKernelGGL(peak_read_kernel, dim3(kPeakBlocks), dim3(kPeakThreads), 0, st,
                     (const uint4 *)src, bytes / 16, out);
  return hipGetLastError();
}

}  // namespace pic

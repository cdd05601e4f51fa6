// Achievable-peak microbenchmarks on gfx950, reported next to the spec peaks
// as a second roofline denominator:
//   * bf16 matrix-core rate: every wave keeps four independent
//     v_mfma_f32_32x32x16_bf16 accumulators busy (2 waves per SIMD on every
//     CU), so the result includes the clock the chip holds under full
//     matrix load;
//   * HBM read rate: a grid-stride stream of 16-byte nontemporal loads over
//     a buffer much larger than the last-level cache, 512 workgroups x 256
//     lanes x 4 loads in flight (the fastest of the stream shapes measured
//     on MI355X: 7.06 TB/s; 1024-4096 workgroups, 8 loads per lane, plain
//     loads and per-workgroup contiguous blocks all read slower);
//   * HBM write rate: a grid-stride stream of 16-byte stores.
// The read and write kernels also calibrate the traffic counters: one
// dispatch moves exactly the buffer's bytes.
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

// Four independent 16-byte nontemporal loads in flight per lane per trip.
constexpr int kReadUnroll = 4;
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 *global_u32x4;
__device__ __forceinline__ uint4 load_nt(const uint4 *p) {
  const u32x4 w = __builtin_nontemporal_load((global_u32x4)p);
  return make_uint4(w.x, w.y, w.z, w.w);
}
__global__ __launch_bounds__(256) void peak_read_kernel(const uint4 *src, int64_t n16, float *out) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + (kReadUnroll - 1) * stride < n16; i += kReadUnroll * stride) {
    uint4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) v[u] = load_nt(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  out[blockIdx.x * blockDim.x + threadIdx.x] = (float)acc;
}

// 16-byte stores of a lane-dependent pattern, grid stride.
__global__ __launch_bounds__(256) void peak_write_kernel(uint4 *dst, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) {
    const uint32_t x = (uint32_t)i;
    dst[i] = make_uint4(x, x ^ 0x55555555u, x ^ 0xAAAAAAAAu, ~x);
  }
}

}  // namespace

// 512 workgroups x 4 waves: 2 waves per SIMD on all 256 CUs (matrix rate,
// read stream); 1024 workgroups for the write stream.
constexpr int kPeakBlocks = 512, kPeakThreads = 256, kStreamBlocks = 1024;

int64_t peak_out_floats() { return (int64_t)kStreamBlocks * kPeakThreads; }

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

hipError_t launch_peak_write(void *dst, int64_t bytes, hipStream_t st) {
  hipLaunchKernelGGL(peak_write_kernel, dim3(kStreamBlocks), dim3(kPeakThreads), 0, st,
                     (uint4 *)dst, bytes / 16);
  return hipGetLastError();
}

}  // namespace pic

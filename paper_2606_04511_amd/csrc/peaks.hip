// peaks.hip -- microbenchmarks of the hardware limits the SparDA kernels are measured against:
// streaming HBM reads, reads of randomly placed 16 KiB blocks (the shape of attended KV blocks)
// and back-to-back bf16 MFMA of both gfx950 bf16 shapes.  Built into its own library for the benchmark; not part of the
// SparDA C ABI.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_util.hpp"

namespace {

// Every lane reads 16-byte words with the non-temporal hint (the hint the decode kernels use; on
// this part it streams about 15 % faster than ordinary loads), 8 in flight, grid-stride over the
// buffer.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4* __restrict__ p, size_t n16, uint32_t* sink) {
  constexpr int U = 8;
  const size_t tid = blockIdx.x * (size_t)256 + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * 256;
  uint32_t acc = 0;
  for (size_t i = tid; i + (U - 1) * stride < n16; i += U * stride) {
    uint4 w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) w[u] = sparda::ld16_nt(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= w[u].x ^ w[u].y ^ w[u].z ^ w[u].w;
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;  // keeps the loads; practically never taken
}

// Workgroups read whole 16 KiB blocks whose indices come from idx (non-temporal hint, 1 KiB
// contiguous per wavefront load).
__global__ __launch_bounds__(256) void block_read_kernel(const uint4* __restrict__ p, const uint32_t* __restrict__ idx,
                                                         int n_idx, uint32_t* sink) {
  uint32_t acc = 0;
  for (int c = blockIdx.x; c < n_idx; c += gridDim.x) {
    const uint4* q = p + (size_t)idx[c] * 1024;
    uint4 w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) w[u] = sparda::ld16_nt(q + threadIdx.x + 256 * u);
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= w[u].x ^ w[u].y ^ w[u].z ^ w[u].w;
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

// Eight independent accumulator chains of v_mfma_f32_16x16x32_bf16 per wavefront.
__global__ __launch_bounds__(256) void mfma_loop_kernel(int iters, float* sink) {
  using namespace sparda;
  const int lane = threadIdx.x & 63;
  uint4 wa = make_uint4(0x3f803f80u + lane, 0x3f003f00u, 0x3e803e80u, 0x3f803f80u);
  uint4 wb = make_uint4(0x3f803f80u, 0x3e803e80u + lane, 0x3f003f00u, 0x3f803f80u);
  const bf16x8 a = as_bf16x8(wa), b = as_bf16x8(wb);
  f32x4 c[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) c[k] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int k = 0; k < 8; ++k) c[k] = mfma16x16x32(a, b, c[k]);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += c[k][0] + c[k][1] + c[k][2] + c[k][3];
  if (s == 1.2345f) sink[0] = s;
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Four independent accumulator chains of v_mfma_f32_32x32x16_bf16 per wavefront (twice the
// flops per instruction; on gfx950 this shape sustains about 1.5 times the 16x16x32 rate).
__global__ __launch_bounds__(256) void mfma32_loop_kernel(int iters, float* sink) {
  using namespace sparda;
  const int lane = threadIdx.x & 63;
  uint4 wa = make_uint4(0x3f803f80u + lane, 0x3f003f00u, 0x3e803e80u, 0x3f803f80u);
  uint4 wb = make_uint4(0x3f803f80u, 0x3e803e80u + lane, 0x3f003f00u, 0x3f803f80u);
  const bf16x8 a = as_bf16x8(wa), b = as_bf16x8(wb);
  f32x16 c[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int j = 0; j < 16; ++j) c[k][j] = 0.f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int k = 0; k < 4; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[k], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) s += c[k][0] + c[k][15];
  if (s == 1.2345f) sink[0] = s;
}

}  // namespace

extern "C" {

// bytes: readable size of p (a multiple of 16); grid: workgroups of 256 threads.
int peaks_stream_read(const void* p, size_t bytes, int grid, void* sink, hipStream_t stream) {
  if (!p || !sink || bytes < 16 || grid < 1) return -1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(p), bytes / 16,
                     static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

// idx: n_idx block indices, each < bytes / 16384 of p (the caller checks).
int peaks_block_read(const void* p, const uint32_t* idx, int n_idx, int grid, void* sink, hipStream_t stream) {
  if (!p || !idx || !sink || n_idx < 1 || grid < 1) return -1;
  hipLaunchKernelGGL(block_read_kernel, dim3(grid), dim3(256), 0, stream, static_cast<const uint4*>(p), idx, n_idx,
                     static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

// Each of grid x 4 wavefronts issues 8 x iters MFMAs of 16 x 16 x 32 (16384 flops each).
int peaks_mfma_bf16(int grid, int iters, void* sink, hipStream_t stream) {
  if (!sink || grid < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(grid), dim3(256), 0, stream, iters, static_cast<float*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

// Each of grid x 4 wavefronts issues 4 x iters MFMAs of 32 x 32 x 16 (32768 flops each).
int peaks_mfma32_bf16(int grid, int iters, void* sink, hipStream_t stream) {
  if (!sink || grid < 1 || iters < 1) return -1;
  hipLaunchKernelGGL(mfma32_loop_kernel, dim3(grid), dim3(256), 0, stream, iters, static_cast<float*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // extern "C"

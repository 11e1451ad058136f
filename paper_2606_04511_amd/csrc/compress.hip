// compress.hip -- mean-pooled block keys K~ (paper Sec. 3, Eq. 2, with window = stride = 64).
//
// One workgroup per (block j, batch*group row).  The block's 64 x 128 bf16 keys are one
// contiguous 16 KiB run; 256 threads read it with 16-byte loads (thread t: dims 8*(t%16)..+7 of
// rows t/16 + 16 i), 1 KiB contiguous per wavefront load.  Partial sums are float64, so the
// 64-term sum of bf16 values is exact and the result does not depend on the reduction order;
// the mean is rounded once to bf16.  HBM-bound: 16 KiB read + 256 B written per block.
#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

__global__ __launch_bounds__(256) void compress_kernel(const uint16_t* __restrict__ k, uint16_t* __restrict__ kc,
                                                       int64_t t_cap, int64_t nc_cap, int32_t blk_begin) {
  __shared__ double part[16][kHeadDim + 1];
  const int j = blk_begin + (int)blockIdx.x;
  const int64_t row = blockIdx.y;
  const int tid = threadIdx.x;
  const int c = tid & 15;  // dims 8c .. 8c+7
  const int rg = tid >> 4; // token rows rg + 16 i
  const uint16_t* src = k + (row * t_cap + (int64_t)j * kBlock) * kHeadDim + c * 8;
  uint4 w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = ld16(src + (rg + 16 * i) * kHeadDim);
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[0] += bf16lo(w[i].x); acc[1] += bf16hi(w[i].x);
    acc[2] += bf16lo(w[i].y); acc[3] += bf16hi(w[i].y);
    acc[4] += bf16lo(w[i].z); acc[5] += bf16hi(w[i].z);
    acc[6] += bf16lo(w[i].w); acc[7] += bf16hi(w[i].w);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[rg][c * 8 + e] = acc[e];
  __syncthreads();
  if (tid < kHeadDim) {
    double s = 0.0;
#pragma unroll
    for (int g = 0; g < 16; ++g) s += part[g][tid];
    kc[(row * nc_cap + j) * kHeadDim + tid] = f64_to_bf16(s * (1.0 / kBlock));
  }
}

hipError_t launch_compress(const uint16_t* k, uint16_t* kc, int32_t rows, int64_t t_cap, int64_t nc_cap,
                           int32_t blk_begin, int32_t blk_end, hipStream_t stream) {
  const int n = blk_end - blk_begin;
  if (n <= 0) return hipSuccess;
  dim3 grid((unsigned)n, (unsigned)rows);
  hipLaunchKernelGGL(compress_kernel, grid, dim3(256), 0, stream, k, kc, t_cap, nc_cap, blk_begin);
  return hipGetLastError();
}

}  // namespace sparda

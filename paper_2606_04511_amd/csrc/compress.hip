// compress.hip -- mean-pooled compressed keys K~ (paper Sec. 3, Eq. 2): window i holds the mean of
// the keys of tokens [i s, i s + l).  The grids served are (64, 64) -- one key per 64-token
// block -- and the paper's (32, 16).
//
// One workgroup per (window i, batch*group row).  The window's l x 128 bf16 keys are one
// contiguous run; 256 threads read it with 16-byte loads (thread t: dims 8*(t%16)..+7 of token
// rows t/16 + 16 x), 1 KiB contiguous per wavefront load.  Partial sums are float64, so the sum
// of at most 64 bf16 values is exact and the result does not depend on the reduction order; the
// mean is rounded once to bf16.  HBM-bound: 2 l x 128 bytes read + 256 B written per window.
#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

template <int NX>  // token rows per thread: window length / 16
__global__ __launch_bounds__(256) void compress_kernel(const uint16_t* __restrict__ k, uint16_t* __restrict__ kc,
                                                       int64_t t_cap, int64_t nc_cap, int32_t stride,
                                                       int32_t w_begin) {
  // Partial sums, dim 8 c + e at 9 c + e of its row: groups of 8 doubles 9 apart and rows 144
  // apart put the writes of 32 lanes on distinct banks (the reads take at most two per bank).
  __shared__ double part[16][144];
  const int i = w_begin + (int)blockIdx.x;
  const int64_t row = blockIdx.y;
  const int tid = threadIdx.x;
  const int c = tid & 15;  // dims 8c .. 8c+7
  const int rg = tid >> 4; // token rows rg + 16 x
  const uint16_t* src = k + (row * t_cap + (int64_t)i * stride) * kHeadDim + c * 8;
  uint4 w[NX];
#pragma unroll
  for (int x = 0; x < NX; ++x) w[x] = ld16(src + (rg + 16 * x) * kHeadDim);
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
  for (int x = 0; x < NX; ++x) {
    acc[0] += bf16lo(w[x].x); acc[1] += bf16hi(w[x].x);
    acc[2] += bf16lo(w[x].y); acc[3] += bf16hi(w[x].y);
    acc[4] += bf16lo(w[x].z); acc[5] += bf16hi(w[x].z);
    acc[6] += bf16lo(w[x].w); acc[7] += bf16hi(w[x].w);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[rg][c * 9 + e] = acc[e];
  __syncthreads();
  if (tid < kHeadDim) {
    double s = 0.0;
#pragma unroll
    for (int g = 0; g < 16; ++g) s += part[g][(tid >> 3) * 9 + (tid & 7)];
    kc[(row * nc_cap + i) * kHeadDim + tid] = f64_to_bf16(s * (1.0 / (16 * NX)));  // exact: 16 NX is a power of 2
  }
}

hipError_t launch_compress(const uint16_t* k, uint16_t* kc, int32_t rows, int64_t t_cap, int64_t nc_cap,
                           WinGrid grid, int32_t w_begin, int32_t w_end, hipStream_t stream) {
  const int n = w_end - w_begin;
  if (n <= 0) return hipSuccess;
  dim3 grid_dim((unsigned)n, (unsigned)rows);
  if (grid.l == 64)
    hipLaunchKernelGGL(compress_kernel<4>, grid_dim, dim3(256), 0, stream, k, kc, t_cap, nc_cap, grid.s, w_begin);
  else if (grid.l == 32)
    hipLaunchKernelGGL(compress_kernel<2>, grid_dim, dim3(256), 0, stream, k, kc, t_cap, nc_cap, grid.s, w_begin);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sparda

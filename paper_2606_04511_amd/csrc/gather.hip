// gather.hip -- copy the selected KV blocks from a host-resident pool into HBM staging
// (paper Sec. 4.3: a persistent kernel with a fixed, small set of workgroups that keeps looping
// over block-transfer tasks in one launch on a dedicated stream; Alg. 2 launches it for layer
// l+1 while layer l computes).
//
// The pool is pinned host memory mapped into the GPU address space, so the kernel reads it
// directly over PCIe (zero copy) and writes HBM.  A task is one (batch, group, slot): 16 KiB of
// K and 16 KiB of V, both contiguous on each side.  Each of the 256 threads issues its eight
// 16-byte loads (four of K, four of V) before any store, so a workgroup keeps 32 KiB of PCIe
// reads in flight; n_workgroups sets how many CUs the copy occupies, which is the knob that
// trades copy speed against interference with the compute stream.
#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

__global__ __launch_bounds__(256) void gather_kernel(const uint4* __restrict__ hk, const uint4* __restrict__ hv,
                                                     const int16_t* __restrict__ sel, const int16_t* __restrict__ cnt,
                                                     uint4* __restrict__ sk, uint4* __restrict__ sv, int64_t rows,
                                                     int64_t t_cap, int32_t k_total) {
  constexpr int kVecPerBlock = kBlock * kHeadDim * 2 / 16;  // 1024 uint4 per 16 KiB block
  const int64_t n_tasks = rows * k_total;
  const int tid = threadIdx.x;
  for (int64_t task = blockIdx.x; task < n_tasks; task += gridDim.x) {
    const int64_t bm = task / k_total;
    const int s = (int)(task % k_total);
    int n = cnt[bm];
    n = n > k_total ? k_total : n;
    if (s >= n) continue;
    const int64_t j = sel[bm * k_total + s];
    if (j < 0 || (j + 1) * kBlock > t_cap) continue;
    const int64_t src = ((bm * t_cap + j * kBlock) * kHeadDim * 2) / 16;
    const int64_t dst = (task * kBlock * kHeadDim * 2) / 16;
    uint4 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = hk[src + tid + 256 * i];
#pragma unroll
    for (int i = 0; i < 4; ++i) b[i] = hv[src + tid + 256 * i];
#pragma unroll
    for (int i = 0; i < 4; ++i) sk[dst + tid + 256 * i] = a[i];
#pragma unroll
    for (int i = 0; i < 4; ++i) sv[dst + tid + 256 * i] = b[i];
    static_assert(kVecPerBlock == 4 * 256, "one 16 KiB block = 4 uint4 per thread");
  }
}

hipError_t launch_gather(const uint16_t* host_k, const uint16_t* host_v, const int16_t* sel, const int16_t* cnt,
                         uint16_t* stage_k, uint16_t* stage_v, int64_t rows, int64_t t_cap, int32_t k_total,
                         int32_t n_workgroups, hipStream_t stream) {
  const int64_t n_tasks = rows * k_total;
  const int64_t grid = n_workgroups < n_tasks ? n_workgroups : n_tasks;
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)grid), dim3(256), 0, stream, reinterpret_cast<const uint4*>(host_k),
                     reinterpret_cast<const uint4*>(host_v), sel, cnt, reinterpret_cast<uint4*>(stage_k),
                     reinterpret_cast<uint4*>(stage_v), rows, t_cap, k_total);
  return hipGetLastError();
}

}  // namespace sparda

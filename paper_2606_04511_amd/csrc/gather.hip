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

// ---- write-back of new KV rows into the host pools ------------------------------------------
//
// The asynchronous CPU write-back of newly created KV entries (Sec. 5.3, prefill throughput): rows produced on the GPU
// (the decoded token's K and V, or a prefill chunk's) are stored into the pinned host pools that
// later gathers read.  A persistent grid of n_workgroups; each thread moves 16-byte pieces with
// zero-copy stores through the mapped pointers.  Task = one (row, token) pair of K and V:
// 2 x 256 bytes, 16 pieces each, so 16 threads per task and 16 tasks per 256-thread workgroup pass.
__global__ __launch_bounds__(256) void writeback_kernel(const uint4* __restrict__ kn, const uint4* __restrict__ vn,
                                                        uint4* __restrict__ hk, uint4* __restrict__ hv, int64_t rows,
                                                        int32_t n_new, int64_t pos0, int64_t t_cap) {
  constexpr int kPieces = kHeadDim * 2 / 16;  // 16-byte pieces per token row
  const int64_t n_tasks = rows * n_new;
  const int piece = threadIdx.x % kPieces, slot = threadIdx.x / kPieces;
  for (int64_t task = (int64_t)blockIdx.x * (256 / kPieces) + slot; task < n_tasks;
       task += (int64_t)gridDim.x * (256 / kPieces)) {
    const int64_t bm = task / n_new;
    const int64_t t = task - bm * n_new;
    const int64_t src = task * kPieces + piece;
    const int64_t dst = (bm * t_cap + pos0 + t) * kPieces + piece;
    const uint4 a = kn[src], b = vn[src];
    hk[dst] = a;
    hv[dst] = b;
  }
}

hipError_t launch_writeback(const uint16_t* k_new, const uint16_t* v_new, uint16_t* host_k, uint16_t* host_v,
                            int64_t rows, int32_t n_new, int64_t pos0, int64_t t_cap, int32_t n_workgroups,
                            hipStream_t stream) {
  const int64_t n_tasks = rows * n_new;
  const int64_t need = (n_tasks + 15) / 16;
  const int64_t grid = n_workgroups < need ? n_workgroups : need;
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(writeback_kernel, dim3((unsigned)grid), dim3(256), 0, stream, reinterpret_cast<const uint4*>(k_new),
                     reinterpret_cast<const uint4*>(v_new), reinterpret_cast<uint4*>(host_k),
                     reinterpret_cast<uint4*>(host_v), rows, n_new, pos0, t_cap);
  return hipGetLastError();
}

// ---- the decoded token into the staged copy of its own block ------------------------------------
//
// Alg. 2 appends each decoded token's K/V to the cache.  In an offloaded layer the attended blocks
// were copied into staging before the token existed (layer l's prefetch is launched during layer
// l - 1), so the token's row is written into every staging slot s < cnt whose block is the
// token's own, p / 64, at row p % 64.  One wavefront per (batch, group) row: a ballot over the set
// finds the slots, lanes 0-15 move the 256-byte K row and lanes 16-31 the V row of each.
__global__ __launch_bounds__(256) void stage_append_kernel(const uint4* __restrict__ kn, const uint4* __restrict__ vn,
                                                           const int16_t* __restrict__ sel,
                                                           const int16_t* __restrict__ cnt, int64_t p,
                                                           uint4* __restrict__ sk, uint4* __restrict__ sv, int64_t rows,
                                                           int32_t K) {
  constexpr int kPieces = kHeadDim * 2 / 16;  // 16-byte pieces per token row
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  int n = cnt[row];
  n = n < 0 ? 0 : (n > K ? K : n);
  const int j = (int)(p / kBlock), t = (int)(p % kBlock);
  const int piece = lane & (kPieces - 1);
  const bool is_k = lane < kPieces, is_v = lane >= kPieces && lane < 2 * kPieces;
  const uint4 w = is_k ? kn[row * kPieces + piece] : (is_v ? vn[row * kPieces + piece] : make_uint4(0u, 0u, 0u, 0u));
  for (int s0 = 0; s0 < n; s0 += kWave) {
    const int s = s0 + lane;
    uint64_t hit = __ballot(s < n && (int)sel[row * K + s] == j);
    while (hit) {
      const int slot = s0 + (int)__builtin_ctzll(hit);
      hit &= hit - 1;
      const int64_t dst = ((row * K + slot) * kBlock + t) * kPieces + piece;
      if (is_k) sk[dst] = w;
      if (is_v) sv[dst] = w;
    }
  }
}

hipError_t launch_stage_append(const uint16_t* k_new, const uint16_t* v_new, const int16_t* sel, const int16_t* cnt,
                               int64_t p, uint16_t* stage_k, uint16_t* stage_v, int64_t rows, int32_t k_total,
                               hipStream_t stream) {
  hipLaunchKernelGGL(stage_append_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream,
                     reinterpret_cast<const uint4*>(k_new), reinterpret_cast<const uint4*>(v_new), sel, cnt, p,
                     reinterpret_cast<uint4*>(stage_k), reinterpret_cast<uint4*>(stage_v), rows, k_total);
  return hipGetLastError();
}

// ---- staging plan of step-to-step reuse (the NOSI engine of the paper's efficiency setup,
// App. C: a layer keeps the blocks its previous decode step attended and fetches only the newly
// selected ones) --------------------------------------------------------------------------------
//
// Slot t of a row's staging holds the first slot_len[t] tokens of block slot_blk[t] (-1: empty).
// A staged block serves the query at p when it covers every token of the block up to p:
// need(j) = min(64, p + 1 - 64 j).  Slots are examined in ascending order; a slot is kept when
// its block is an entry of the new set S not yet claimed by a lower slot and it covers need(j).
// The entries of S that no kept slot holds are fetched, in entry order, into the free slots in
// ascending order; slots left unused are emptied.  One wavefront per row; the set and the claim
// flags live in the wavefront's LDS.

constexpr int kPlanMaxK = 1024;

__device__ __forceinline__ int plan_need(int j, int64_t p) {
  const int64_t n = p + 1 - (int64_t)j * kBlock;
  return n > kBlock ? kBlock : (int)n;
}

__global__ __launch_bounds__(256) void plan_staging_kernel(const int16_t* __restrict__ sel,
                                                           const int16_t* __restrict__ cnt, int64_t p,
                                                           int16_t* __restrict__ slot_blk, int16_t* __restrict__ slot_len,
                                                           int16_t* __restrict__ fetch, int16_t* __restrict__ staged,
                                                           int16_t* __restrict__ stage_cnt, int32_t* __restrict__ n_fetch,
                                                           int64_t rows, int32_t K) {
  __shared__ int s_set[4][kPlanMaxK];
  __shared__ int s_held[4][kPlanMaxK];
  __shared__ int s_kept[4][kPlanMaxK];
  __shared__ int s_free[4][kPlanMaxK];
  __shared__ int s_att[4][kPlanMaxK];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= rows) return;
  int* set = s_set[wave];
  int* held = s_held[wave];
  int* kept = s_kept[wave];
  int* freel = s_free[wave];
  int* satt = s_att[wave];  // the block each slot holds for this step, -1 none
  const int16_t* srow = sel + row * K;
  int16_t* blk = slot_blk + row * K;
  int16_t* len = slot_len + row * K;
  int16_t* fet = fetch + row * K;
  int16_t* att = staged + row * K;
  int n = cnt[row];
  n = n < 0 ? 0 : (n > K ? K : n);
  for (int i = lane; i < K; i += kWave) {
    set[i] = i < n ? (int)srow[i] : -1;
    held[i] = 0;
  }
  wave_lds_sync();
  // kept slots, in ascending slot order (a slot claims the first unclaimed matching entry)
  for (int t = 0; t < K; ++t) {
    const int j = blk[t];
    bool keep = false;
    if (j >= 0 && len[t] >= plan_need(j, p)) {
      for (int i0 = 0; i0 < n; i0 += kWave) {
        const int i = i0 + lane;
        const uint64_t hit = __ballot(i < n && set[i] == j && held[i] == 0);
        if (hit) {
          const int first = i0 + (int)__builtin_ctzll(hit);
          if (lane == 0) held[first] = 1;
          keep = true;
          break;
        }
      }
    }
    if (lane == 0) kept[t] = keep ? 1 : 0;
    wave_lds_sync();
  }
  // free slots in ascending order
  int n_free = 0;
  for (int t0 = 0; t0 < K; t0 += kWave) {
    const int t = t0 + lane;
    const bool fr = t < K && kept[t] == 0;
    const uint64_t b = __ballot(fr);
    if (fr) freel[n_free + mbcnt64(b)] = t;
    n_free += __popcll(b);
  }
  for (int t = lane; t < K; t += kWave) {
    fet[t] = -1;
    satt[t] = kept[t] ? (int)blk[t] : -1;
  }
  wave_lds_sync();
  // missing entries in entry order into the free slots in ascending order
  int n_miss = 0;
  for (int i0 = 0; i0 < n; i0 += kWave) {
    const int i = i0 + lane;
    const int j = i < n ? set[i] : -1;
    const bool miss = i < n && held[i] == 0 && j >= 0;
    const uint64_t b = __ballot(miss);
    const int r = n_miss + mbcnt64(b);
    if (miss && r < n_free) {
      const int t = freel[r];
      fet[t] = (int16_t)j;
      satt[t] = j;
      blk[t] = (int16_t)j;
      len[t] = (int16_t)plan_need(j, p);
    }
    n_miss += __popcll(b);
  }
  wave_lds_sync();
  for (int t = lane; t < K; t += kWave) {
    const int a = satt[t];
    att[t] = (int16_t)a;
    if (a < 0) {
      blk[t] = -1;
      len[t] = 0;
    }
  }
  if (lane == 0) {
    stage_cnt[row] = (int16_t)K;
    n_fetch[row] = n_miss;
  }
}

hipError_t launch_plan_staging(const int16_t* sel, const int16_t* cnt, int64_t p, int16_t* slot_blk, int16_t* slot_len,
                               int16_t* fetch, int16_t* staged, int16_t* stage_cnt, int32_t* n_fetch, int64_t rows,
                               int32_t k_total, hipStream_t stream) {
  if (k_total > kPlanMaxK) return hipErrorInvalidValue;
  hipLaunchKernelGGL(plan_staging_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, sel, cnt, p,
                     slot_blk, slot_len, fetch, staged, stage_cnt, n_fetch, rows, k_total);
  return hipGetLastError();
}

}  // namespace sparda

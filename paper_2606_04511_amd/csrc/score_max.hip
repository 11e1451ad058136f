// score_max.hip -- the Forecast prefill score contraction on 32x32x16 MFMA (Sec. 4.1, Eq. 4):
// each row's largest candidate score (a measurement of the contraction alone), and the window
// scores of the row-wise selection path (at the end of this file).
//
// The score contraction on its own: every
// candidate block of every query row is scored and each row's scores are reduced on chip to
// their maximum, so that one float per row leaves the kernel.  It isolates the dense contraction
// that the fused select kernel performs before its per-row top-k, on the (64, 64) key grid.
//
// Work unit: the rows of one (batch, group) whose positions fall in one 64-token block (at most
// 64 rows, all with the candidate range [n_init, blk - n_local]).  A workgroup of four
// wavefronts owns one unit.  Each wavefront holds the unit's F rows as the B operand of
// v_mfma_f32_32x32x16_bf16 (two N-tiles of 32 rows, 64 VGPRs) and takes every fourth M-tile of
// 32 candidates, reading the K~ rows of its next M-tile (L2-resident) while the current one is
// multiplied.  The dot product's dimension order is free: lane half h of k-step 4 u + i holds
// dimensions 64 u + 32 h + 8 i .. + 7 of both operands, so a lane reads 64 contiguous bytes of a
// row per u.  Candidates past the range load the last candidate again (a repeated score leaves
// a maximum unchanged) and rows past the unit load its last row (their maximum is not written),
// so every load is unconditional and in bounds.  An accumulator lane holds 16 scores of one
// query column (lane % 32); the two lane halves and the four wavefronts are merged at the end.
//
// Units run from the most candidates to the fewest.  Consecutive workgroups take consecutive
// (batch, group) pairs, and workgroups are dealt to the 8 XCDs in turn, so with a pair count that
// is a multiple of 8 every workgroup of one group lands on one XCD and its K~ stays in that L2.
#include <math.h>

#include <algorithm>

#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

namespace {

constexpr int kSmThreads = 256;
constexpr int kSmWaves = kSmThreads / kWave;
constexpr int kRowU4 = kHeadDim * 2 / 16;  // 16-byte pieces per 128-dim bf16 row

typedef float f32x16 __attribute__((ext_vector_type(16)));

// The 8 k-step fragments (8 bf16 each) of one row for lane half h.
__device__ __forceinline__ void load_frags(const uint4* row, int h, uint4 (&x)[8]) {
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) x[4 * u + i] = row[8 * u + 4 * h + i];
}

// One M-tile of 32 keys against both N-tiles: the products only.
__device__ __forceinline__ void mma_tile(const uint4 (&a)[8], const uint4 (&fb)[2][8], f32x16& c0, f32x16& c1) {
#pragma unroll
  for (int e = 0; e < 16; ++e) c0[e] = c1[e] = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const bf16x8 av = as_bf16x8(a[s]);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(fb[0][s]), c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(fb[1][s]), c1, 0, 0, 0);
  }
}

// One M-tile of 32 candidates against both N-tiles; folds the scores into the running maxima.
__device__ __forceinline__ void score_tile(const uint4 (&a)[8], const uint4 (&fb)[2][8], float& run0, float& run1) {
  f32x16 c0, c1;
#pragma unroll
  for (int e = 0; e < 16; ++e) c0[e] = c1[e] = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const bf16x8 av = as_bf16x8(a[s]);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(fb[0][s]), c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(fb[1][s]), c1, 0, 0, 0);
  }
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    run0 = fmaxf(run0, c0[e]);
    run1 = fmaxf(run1, c1[e]);
  }
}

__global__ __launch_bounds__(kSmThreads) void score_rowmax_kernel(ScoreMaxArgs a) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar loop control
  const int n = lane & 31, h = lane >> 5;
  const int grp = blockIdx.x % a.n_groups;                       // (batch, group) pair
  const int unit = a.n_units - 1 - (int)(blockIdx.x / a.n_groups);  // most candidates first
  const int blk = a.blk0 + unit;
  const int64_t p_lo = max((int64_t)blk * kBlock, a.q_pos0);
  const int64_t p_hi = min((int64_t)blk * kBlock + kBlock, a.q_pos0 + a.n_q);
  const int nr = (int)(p_hi - p_lo);  // 1..64 rows
  const int64_t row0 = (int64_t)grp * a.n_q + (p_lo - a.q_pos0);
  const int c_hi = blk - a.n_local;
  const int n_cand = c_hi >= a.n_init ? c_hi - a.n_init + 1 : 0;
  if (n_cand == 0) {
    if ((int)threadIdx.x < nr) a.row_max[row0 + threadIdx.x] = -INFINITY;
    return;
  }
  __shared__ float part[kSmWaves][64];

  // B operand: the unit's F rows 32 nt + n (clamped to the last row).
  uint4 fb[2][8];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int r = min(32 * nt + n, nr - 1);
    load_frags(reinterpret_cast<const uint4*>(a.f) + (row0 + r) * kRowU4, h, fb[nt]);
  }

  const uint4* kc = reinterpret_cast<const uint4*>(a.kc) + ((int64_t)grp * a.nc_cap + a.n_init) * kRowU4;
  const int n_mt = (n_cand + 31) / 32;
  float run0 = -INFINITY, run1 = -INFINITY;
  if (w < n_mt) {
    // Two register buffers in turn: the M-tile after the current one is requested before the
    // current one is multiplied (past the end the last M-tile is requested again), so the wait
    // before the products covers only the current tile's loads.
    uint4 ab[2][8];
    auto arow = [&](int mt) { return kc + (int64_t)min(32 * min(mt, n_mt - 1) + n, n_cand - 1) * kRowU4; };
    load_frags(arow(w), h, ab[0]);
    for (int mt = w; mt < n_mt; mt += 2 * kSmWaves) {
      load_frags(arow(mt + kSmWaves), h, ab[1]);
      __builtin_amdgcn_sched_barrier(0);  // keep the request ahead of the products
      score_tile(ab[0], fb, run0, run1);
      load_frags(arow(mt + 2 * kSmWaves), h, ab[0]);
      __builtin_amdgcn_sched_barrier(0);
      if (mt + kSmWaves < n_mt) score_tile(ab[1], fb, run0, run1);
    }
  }
  // Lanes n and n + 32 hold the two row halves of column n.
  run0 = fmaxf(run0, __shfl_xor(run0, 32));
  run1 = fmaxf(run1, __shfl_xor(run1, 32));
  if (h == 0) {
    part[w][n] = run0;
    part[w][32 + n] = run1;
  }
  __syncthreads();
  if ((int)threadIdx.x < nr) {
    const int t = threadIdx.x;
    a.row_max[row0 + t] = fmaxf(fmaxf(part[0][t], part[1][t]), fmaxf(part[2][t], part[3][t]));
  }
}

// ---- the persistent form: the group's K~ in LDS --------------------------------------------
//
// When every row of the call has at most kSlMaxCand candidates, one 512-thread workgroup per CU
// stages its group's candidate keys in LDS once (272-byte row pitch: the 16 rows a quarter
// wavefront reads start 4 banks apart, so a 16-byte read is conflict-free) and its eight
// wavefronts take whole units from an LDS counter.  A wavefront requests the next unit's F rows
// before it multiplies the current unit, whose A fragments come from LDS.  A group's units are
// dealt to its workgroups in a serpentine over descending candidate counts, so each workgroup's
// list is balanced and sorted most-expensive first.

constexpr int kSlThreads = 512;
constexpr int kSlWaves = kSlThreads / kWave;
constexpr int kSlMaxCand = 512;
constexpr int kSlPitchU4 = kRowU4 + 1;  // 16-byte pieces per staged row (272 B)

__device__ __forceinline__ void load_lds_frags(const uint4* row, int h, uint4 (&x)[8]) {
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) x[4 * u + i] = row[8 * u + 4 * h + i];
}

struct SlUnit {
  int blk, nr, n_cand;
  int64_t row0;
};

// The i-th unit of workgroup slot s of p slots (serpentine over descending block index), or
// blk < 0 past the end.
__device__ __forceinline__ SlUnit sl_unit(const ScoreMaxArgs& a, int grp, int s, int p, int i) {
  SlUnit u;
  const int g = i * p + ((i & 1) ? p - 1 - s : s);
  if (g >= a.n_units) {
    u.blk = -1;
    u.nr = u.n_cand = 0;
    u.row0 = 0;
    return u;
  }
  u.blk = a.blk0 + a.n_units - 1 - g;
  const int64_t p_lo = max((int64_t)u.blk * kBlock, a.q_pos0);
  const int64_t p_hi = min((int64_t)u.blk * kBlock + kBlock, a.q_pos0 + a.n_q);
  u.nr = (int)(p_hi - p_lo);
  u.row0 = (int64_t)grp * a.n_q + (p_lo - a.q_pos0);
  const int c_hi = u.blk - a.n_local;
  u.n_cand = c_hi >= a.n_init ? c_hi - a.n_init + 1 : 0;
  return u;
}

__device__ __forceinline__ void load_unit_f(const ScoreMaxArgs& a, const SlUnit& u, int n, int h,
                                            uint4 (&fb)[2][8]) {
  const int nr = max(u.nr, 1);
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int r = min(32 * nt + n, nr - 1);
    load_frags(reinterpret_cast<const uint4*>(a.f) + (u.row0 + r) * kRowU4, h, fb[nt]);
  }
}

// Scores one unit against the staged keys and writes its rows' maxima.
__device__ __forceinline__ void sl_score_unit(const ScoreMaxArgs& a, const SlUnit& u, const uint4* kst,
                                              const uint4 (&fb)[2][8], int n, int h) {
  float run0 = -INFINITY, run1 = -INFINITY;
  const int n_mt = (u.n_cand + 31) / 32;
  // A fragments one M-tile ahead, in two register sets (reads past the end repeat the last tile)
  auto arow = [&](int mt) { return kst + min(32 * min(mt, n_mt - 1) + n, u.n_cand - 1) * kSlPitchU4; };
  uint4 a0[8], a1[8];
  load_lds_frags(arow(0), h, a0);
  for (int mt = 0; mt < n_mt; mt += 2) {
    load_lds_frags(arow(mt + 1), h, a1);
    __builtin_amdgcn_sched_barrier(0);
    score_tile(a0, fb, run0, run1);
    load_lds_frags(arow(mt + 2), h, a0);
    __builtin_amdgcn_sched_barrier(0);
    if (mt + 1 < n_mt) score_tile(a1, fb, run0, run1);
  }
  run0 = fmaxf(run0, __shfl_xor(run0, 32));
  run1 = fmaxf(run1, __shfl_xor(run1, 32));
  if (h == 0) {
    if (n < u.nr) a.row_max[u.row0 + n] = run0;
    if (32 + n < u.nr) a.row_max[u.row0 + 32 + n] = run1;
  }
}

__global__ __launch_bounds__(kSlThreads) void score_rowmax_lds_kernel(ScoreMaxArgs a, int slots) {
  __shared__ uint4 kst[kSlMaxCand * kSlPitchU4];  // [c_max][kSlPitchU4] used
  __shared__ int next_unit;
  const int lane = threadIdx.x & 63;
  const int n = lane & 31, h = lane >> 5;
  const int grp = blockIdx.x % a.n_groups;
  const int slot = blockIdx.x / a.n_groups;
  if (threadIdx.x == 0) next_unit = kSlWaves;
  // the largest candidate count of the call: the last row's
  const int c_hi = (int)((a.q_pos0 + a.n_q - 1) / kBlock) - a.n_local;
  const int c_max = c_hi >= a.n_init ? c_hi - a.n_init + 1 : 0;
  const uint4* kc = reinterpret_cast<const uint4*>(a.kc) + ((int64_t)grp * a.nc_cap + a.n_init) * kRowU4;
  if (c_max > 0) {
    // Every load in flight before the first LDS store.  Pieces past the staged rows are clamped
    // to the last piece: loaded and stored again with the same value (no branch for the
    // compiler to sink a load into).
    constexpr int kIt = kSlMaxCand * kRowU4 / kSlThreads / 2;  // two rounds of 8 pieces
    const int n_pc = c_max * kRowU4;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      uint4 t[kIt];
#pragma unroll
      for (int k = 0; k < kIt; ++k)
        t[k] = kc[min((int)threadIdx.x + (half * kIt + k) * kSlThreads, n_pc - 1)];
#pragma unroll
      for (int k = 0; k < kIt; ++k) {
        const int q = min((int)threadIdx.x + (half * kIt + k) * kSlThreads, n_pc - 1);
        kst[(q / kRowU4) * kSlPitchU4 + q % kRowU4] = t[k];
      }
    }
  }

  // Each wavefront starts with unit w of the slot's list; later units come from the counter.
  // Even wavefronts request their first F rows before the staging barrier and odd ones after
  // it, so that the two wavefronts of a SIMD do not wait for one burst together: the first can
  // multiply while the second one's rows arrive.
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  SlUnit cur = sl_unit(a, grp, slot, slots, w);
  uint4 fb[2][8], fn[2][8];
  const bool first_early = (w & 1) == 0;
  if (first_early && cur.blk >= 0 && cur.n_cand > 0) load_unit_f(a, cur, n, h, fb);
  __syncthreads();
  if (!first_early && cur.blk >= 0 && cur.n_cand > 0) load_unit_f(a, cur, n, h, fb);

  while (cur.blk >= 0) {
    int j = 0;
    if (lane == 0) j = atomicAdd(&next_unit, 1);
    j = __builtin_amdgcn_readfirstlane(j);
    const SlUnit nxt = sl_unit(a, grp, slot, slots, j);
    // The next unit's F rows are requested before this unit's products (past the end, this
    // unit's rows again: in bounds and never used).
    load_unit_f(a, nxt.blk >= 0 && nxt.n_cand > 0 ? nxt : cur, n, h, fn);
    __builtin_amdgcn_sched_barrier(0);
    if (cur.n_cand == 0) {
      if (lane < cur.nr) a.row_max[cur.row0 + lane] = -INFINITY;
    } else {
      sl_score_unit(a, cur, kst, fb, n, h);
    }
    cur = nxt;
    if (cur.blk < 0) break;
    // the same with the buffers' roles exchanged
    if (lane == 0) j = atomicAdd(&next_unit, 1);
    j = __builtin_amdgcn_readfirstlane(j);
    const SlUnit nx2 = sl_unit(a, grp, slot, slots, j);
    load_unit_f(a, nx2.blk >= 0 && nx2.n_cand > 0 ? nx2 : cur, n, h, fb);
    __builtin_amdgcn_sched_barrier(0);
    if (cur.n_cand == 0) {
      if (lane < cur.nr) a.row_max[cur.row0 + lane] = -INFINITY;
    } else {
      sl_score_unit(a, cur, kst, fn, n, h);
    }
    cur = nx2;
  }
}

// ---- window scores of many rows, for the row-wise selection path -----------------------------
//
// Multi-row calls whose rows have more than kSelTileMaxCand candidates keep every window score in
// the workspace (row stride ws_stride, window wf at slot 0) for the row-wise top-k.  The same
// units (the rows of one (batch, group) inside one 64-token block) score the windows [wf, wl] of
// their last row on 32x32x16 MFMA, A = 32 windows of K~ per M-tile (from L2, one M-tile ahead),
// B = the unit's 64 F rows, so each key fragment serves 64 rows.  Accumulator element e of lane
// (n, h) is window 8 (e / 4) + 4 h + e % 4 of the M-tile for query column n: each group of four
// elements is one 16-byte store.  Earlier rows of a unit get up to three windows past their own
// last visible one; the top-k never reads them.

__global__ __launch_bounds__(kSmThreads) void tile_score_kernel(SelectArgs a, int blk0, int n_units) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int n_groups = a.batch * a.n_kv_heads;
  const int grp = blockIdx.x % n_groups;
  const int unit = n_units - 1 - (int)(blockIdx.x / n_groups);
  const int blk = blk0 + unit;
  const int64_t p_lo = max((int64_t)blk * kBlock, a.q_pos0);
  const int64_t p_hi = min((int64_t)blk * kBlock + kBlock, a.q_pos0 + a.n_q);
  const int nr = (int)(p_hi - p_lo);
  const int64_t row0 = (int64_t)grp * a.n_q + (p_lo - a.q_pos0);
  const RowGeom g = row_geom(p_hi - 1, a.n_init, a.n_local, a.k_total);
  if (g.n_take >= g.n_cand) return;  // then every row of the unit takes all its candidates
  int32_t wf, wl;
  row_windows(g, a.grid, p_hi - 1, &wf, &wl);
  const int nwu = wl - wf + 1;

  uint4 fb[2][8];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int r = min(32 * nt + n, nr - 1);
    load_frags(reinterpret_cast<const uint4*>(a.f) + (row0 + r) * kRowU4, h, fb[nt]);
  }
  const uint4* kc = reinterpret_cast<const uint4*>(a.kc) + ((int64_t)grp * a.nc_cap + wf) * kRowU4;
  const int n_mt = (nwu + 31) / 32;
  float* out0 = a.ws + (row0 + n) * a.ws_stride;
  float* out1 = a.ws + (row0 + 32 + n) * a.ws_stride;
  auto store = [&](int mt, const f32x16& c0, const f32x16& c1) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int x = 32 * mt + 8 * q + 4 * h;
      if (x < nwu) {
        if (n < nr) *reinterpret_cast<float4*>(out0 + x) = make_float4(c0[4 * q], c0[4 * q + 1], c0[4 * q + 2], c0[4 * q + 3]);
        if (32 + n < nr)
          *reinterpret_cast<float4*>(out1 + x) = make_float4(c1[4 * q], c1[4 * q + 1], c1[4 * q + 2], c1[4 * q + 3]);
      }
    }
  };
  if (w < n_mt) {
    uint4 ab[2][8];
    auto arow = [&](int mt) { return kc + (int64_t)min(32 * min(mt, n_mt - 1) + n, nwu - 1) * kRowU4; };
    load_frags(arow(w), h, ab[0]);
    for (int mt = w; mt < n_mt; mt += 2 * kSmWaves) {
      load_frags(arow(mt + kSmWaves), h, ab[1]);
      __builtin_amdgcn_sched_barrier(0);  // keep the request ahead of the products
      f32x16 c0, c1;
      mma_tile(ab[0], fb, c0, c1);
      store(mt, c0, c1);
      load_frags(arow(mt + 2 * kSmWaves), h, ab[0]);
      __builtin_amdgcn_sched_barrier(0);
      if (mt + kSmWaves < n_mt) {
        mma_tile(ab[1], fb, c0, c1);
        store(mt + kSmWaves, c0, c1);
      }
    }
  }
}

}  // namespace

hipError_t launch_score_rowmax(const ScoreMaxArgs& a, hipStream_t stream) {
  const int c_hi = (int)((a.q_pos0 + a.n_q - 1) / kBlock) - a.n_local;
  const int c_max = c_hi >= a.n_init ? c_hi - a.n_init + 1 : 0;
  // Persistent form whenever the keys fit: about one workgroup per CU and at least one unit per
  // wavefront.  Workgroup b serves group b % n_groups, so with 8 | n_groups a group's workgroups
  // share an XCD.
  if (c_max <= kSlMaxCand) {
    const int slots = std::max(1, std::min(a.n_units / kSlWaves, 256 / a.n_groups));
    hipLaunchKernelGGL(score_rowmax_lds_kernel, dim3((unsigned)(slots * a.n_groups)), dim3(kSlThreads), 0, stream,
                       a, slots);
    return hipGetLastError();
  }
  const int64_t wgs = (int64_t)a.n_units * a.n_groups;
  hipLaunchKernelGGL(score_rowmax_kernel, dim3((unsigned)wgs), dim3(kSmThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_tile_scores(const SelectArgs& a, hipStream_t stream) {
  const int blk0 = (int)(a.q_pos0 / kBlock);
  const int n_units = (int)((a.q_pos0 + a.n_q - 1) / kBlock) - blk0 + 1;
  const int64_t wgs = (int64_t)n_units * a.batch * a.n_kv_heads;
  hipLaunchKernelGGL(tile_score_kernel, dim3((unsigned)wgs), dim3(kSmThreads), 0, stream, a, blk0, n_units);
  return hipGetLastError();
}

}  // namespace sparda

// select_block.hpp -- block-wide exact top-k over scores held in LDS, shared by the fused decode
// selectors (the Forecast indexer and the multi-head selector it replaces).
#pragma once
#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

constexpr int kDecThreads = 512;  // 8 wavefronts per row

// Forced blocks of a row: initial blocks first, the chosen candidates after them (written by the
// select routine), then the local window, then -1 padding up to k_total.
__device__ __forceinline__ void emit_forced(int16_t* out, const RowGeom& g, int k_total, int lane) {
  for (int i = lane; i < g.init_hi; i += kWave) out[i] = (int16_t)i;
  const int n_loc = g.blk - g.local_lo + 1;
  for (int i = lane; i < n_loc; i += kWave) out[g.init_hi + g.n_take + i] = (int16_t)(g.local_lo + i);
  for (int i = g.n_forced + g.n_take + lane; i < k_total; i += kWave) out[i] = (int16_t)-1;
}


// Block-wide count of flagged items before each thread's first item, where thread t holds the
// P consecutive items P t .. P t + P - 1 in order, plus the total.  Ballots and mbcnt inside the
// wavefront, one LDS exchange of the wavefront totals (wave_cnt: kDecThreads/64 ints).  Contains
// two barriers (the second lets the next call reuse wave_cnt).
template <int P>
__device__ __forceinline__ int block_flag_prefix(const bool (&f)[P], int* wave_cnt, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int in_wave = 0, before = 0;
#pragma unroll
  for (int e = 0; e < P; ++e) {
    const uint64_t b = __ballot(f[e]);
    in_wave += (int)__popcll(b);
    before += mbcnt64(b);
  }
  if (lane == 0) wave_cnt[wave] = in_wave;
  __syncthreads();
  int all = 0;
#pragma unroll
  for (int w = 0; w < kDecThreads / 64; ++w) {
    const int c = wave_cnt[w];
    before += w < wave ? c : 0;
    all += c;
  }
  __syncthreads();
  *total = all;
  return before;
}

// The whole workgroup selects the n_take largest of the C block scores bs[0 .. C) (ties: lower
// index) by a radix select of 8 bits per pass over an LDS histogram, and writes cand_lo + i of the
// chosen ones in ascending order to chosen_out[0 .. n_take).  0 < n_take < C.  hist: 256 uint32
// (16-byte aligned), wave_cnt: kDecThreads / 64 ints, pick: 3 ints, all LDS.  Every thread of the
// workgroup must call it.
__device__ __forceinline__ void block_topk_emit(const float* bs, int C, int n_take, int cand_lo, int16_t* chosen_out,
                                                uint32_t* hist, int* wave_cnt, int* pick) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Radix select of the n_take-th largest key, 8 bits per pass, over the whole workgroup.
  uint32_t prefix = 0u, mask = 0u;
  int remaining = n_take;
  bool take_all = false;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    for (int i = tid; i < C; i += kDecThreads) {
      const uint32_t kk = score_key(bs[i]);
      if ((kk & mask) == prefix) atomicAdd(&hist[(kk >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      const uint4 h = reinterpret_cast<const uint4*>(hist)[63 - lane];
      const int lsum = (int)(h.x + h.y + h.z + h.w);
      const int incl = wave_incl_scan(lsum);
      const int excl = incl - lsum;
      if (excl < remaining && remaining <= incl) {
        int above = excl, d = 255 - 4 * lane, eq = (int)h.w;
        if (above + (int)h.w < remaining) {
          above += (int)h.w; d -= 1; eq = (int)h.z;
          if (above + (int)h.z < remaining) {
            above += (int)h.z; d -= 1; eq = (int)h.y;
            if (above + (int)h.y < remaining) { above += (int)h.y; d -= 1; eq = (int)h.x; }
          }
        }
        pick[0] = d;
        pick[1] = above;
        pick[2] = eq;
      }
    }
    __syncthreads();
    const int d = pick[0], above = pick[1], eq = pick[2];
    remaining -= above;
    prefix |= (uint32_t)d << shift;
    mask |= 0xffu << shift;
    take_all = (eq == remaining);
    __syncthreads();
    if (take_all) break;
  }

  // Emit in ascending candidate order; equal keys at the threshold go to the lowest indices.
  // Thread t takes candidates 4 t .. 4 t + 3 of each run of 4 kDecThreads, so thread order is
  // candidate order and one flag prefix per run places them (two in the tie case).
  constexpr int kPer = 4;
  int base = 0, tie_base = 0;
  for (int c0 = 0; c0 < C; c0 += kPer * kDecThreads) {
    uint32_t kk[kPer];
    bool valid[kPer], ch[kPer];
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const int i = c0 + kPer * tid + e;
      valid[e] = i < C;
      kk[e] = score_key(bs[min(i, C - 1)]);  // in bounds for every thread
    }
    if (take_all) {
#pragma unroll
      for (int e = 0; e < kPer; ++e) ch[e] = valid[e] && (kk[e] & mask) >= prefix;
    } else {
      bool tie[kPer];
#pragma unroll
      for (int e = 0; e < kPer; ++e) tie[e] = valid[e] && kk[e] == prefix;
      int n_ties;
      int trank = tie_base + block_flag_prefix(tie, wave_cnt, &n_ties);
      tie_base += n_ties;
#pragma unroll
      for (int e = 0; e < kPer; ++e) {
        ch[e] = valid[e] && (kk[e] > prefix || (tie[e] && trank < remaining));
        trank += tie[e] ? 1 : 0;
      }
    }
    int n_chosen;
    int pos = base + block_flag_prefix(ch, wave_cnt, &n_chosen);
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      if (ch[e]) {
        if (pos < n_take) chosen_out[pos] = (int16_t)(cand_lo + c0 + kPer * tid + e);  // never past the row's slots
        ++pos;
      }
    }
    base += n_chosen;
  }
}

}  // namespace sparda

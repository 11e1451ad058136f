// select_block.hpp -- block-wide exact top-k over scores held in LDS, shared by the fused decode
// selectors (the Forecast indexer and the multi-head selector it replaces).
#pragma once
#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

constexpr int kDecThreads = 512;  // 8 wavefronts per row
constexpr int kTopkLds = 512;     // uint32 of LDS scratch that block_topk_emit takes (`hist`)
constexpr int kTopkList = 64;     // most scores in the threshold bin that one wavefront ranks

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

// One wavefront selects the n_take largest keys among n_cand candidates (ties: lower index) and
// writes their indices cand_lo + i in ascending order to out[0 .. n_take).  key_of(i) returns
// score_key of candidate i.  hist: 256 uint32 of wave-private, 16-byte aligned LDS.
template <class KeyFn>
__device__ void wave_topk_emit(KeyFn key_of, int n_cand, int n_take, int cand_lo, uint32_t* hist, int16_t* out) {
  const int lane = threadIdx.x & (kWave - 1);
  if (n_take >= n_cand) {
    for (int i = lane; i < n_cand; i += kWave) out[i] = (int16_t)(cand_lo + i);
    return;
  }
  if (n_take <= 0) return;
  uint32_t prefix = 0u, mask = 0u;
  int remaining = n_take;  // still to take among keys that match `prefix` under `mask`
  bool take_all = false;
  for (int pass = 0; pass < 4 && !take_all; ++pass) {
    const int shift = 24 - 8 * pass;
    reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0u, 0u, 0u, 0u);
    wave_lds_sync();
    for (int i = lane; i < n_cand; i += kWave) {
      const uint32_t kk = key_of(i);
      if ((kk & mask) == prefix) atomicAdd(&hist[(kk >> shift) & 255u], 1u);
    }
    wave_lds_sync();
    // Lane l owns digits 255-4l (h.w) down to 252-4l (h.x): a descending scan over lanes.
    const uint4 h = reinterpret_cast<const uint4*>(hist)[63 - lane];
    const int lsum = (int)(h.x + h.y + h.z + h.w);
    const int incl = wave_incl_scan(lsum);
    const int excl = incl - lsum;
    const uint64_t hit = __ballot(excl < remaining && remaining <= incl);
    const int src = hit ? (int)__builtin_ctzll(hit) : 0;  // exactly one lane holds the k-th key
    int above = excl, d = 255 - 4 * lane, eq = (int)h.w;
    if (above + (int)h.w < remaining) {
      above += (int)h.w; d -= 1; eq = (int)h.z;
      if (above + (int)h.z < remaining) {
        above += (int)h.z; d -= 1; eq = (int)h.y;
        if (above + (int)h.y < remaining) { above += (int)h.y; d -= 1; eq = (int)h.x; }
      }
    }
    above = readlane_i(above, src);
    d = readlane_i(d, src);
    eq = readlane_i(eq, src);
    remaining -= above;
    prefix |= (uint32_t)d << shift;
    mask |= 0xffu << shift;
    take_all = (eq == remaining);
    wave_lds_sync();
  }
  int base = 0, tie_base = 0;
  for (int i0 = 0; i0 < n_cand; i0 += kWave) {
    const int i = i0 + lane;
    const bool valid = i < n_cand;
    const uint32_t kk = valid ? key_of(i) : 0u;
    bool chosen;
    if (take_all) {
      chosen = valid && (kk & mask) >= prefix;
    } else {  // prefix is the exact k-th key; equal keys go to the lowest indices
      const bool tie = valid && kk == prefix;
      const uint64_t tb = __ballot(tie);
      const int trank = tie_base + mbcnt64(tb);
      tie_base += __popcll(tb);
      chosen = valid && (kk > prefix || (tie && trank < remaining));
    }
    const uint64_t cb = __ballot(chosen);
    const int pos = base + mbcnt64(cb);
    if (chosen && pos < n_take) out[pos] = (int16_t)(cand_lo + i);  // never past the row's slots
    base += __popcll(cb);
  }
}

// The radix form of block_topk_emit: the n_take-th largest key by 8 bits per pass over an LDS
// histogram (hist[0 .. 256)), then the ordered emission with a rank among the keys equal to it.
// Used where the value-binned form cannot rank the threshold bin.
__device__ __forceinline__ void radix_topk_emit(const float* bs, int C, int n_take, int cand_lo, int16_t* chosen_out,
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

// Bin of score s among 256 equal-width bins over [lo, lo + 256 / scale]: non-decreasing in s
// (each step rounds monotonically), so a higher bin holds only larger scores.
__device__ __forceinline__ int lin_bin(float s, float lo, float scale) {
  return (int)fminf((s - lo) * scale, 255.0f);
}

// The whole workgroup selects the n_take largest of the C block scores bs[0 .. C) (ties: lower
// index) and writes cand_lo + i of the chosen ones in ascending order to chosen_out[0 .. n_take).
// 0 < n_take < C.  hist: kTopkLds uint32 (16-byte aligned), wave_cnt: kDecThreads / 64 ints,
// pick: 3 ints, all LDS.  Every thread of the workgroup must call it.
//
// The scores' range [min, max] is cut into 256 equal-width bins, and one LDS histogram finds the
// bin holding the n_take-th largest score.  That bin's scores (usually a handful: the threshold
// sits in the upper tail) are collected, and every wavefront ranks them by (score, then lower
// index), which gives the last chosen pair (kk, ki): a score is chosen when its key is above kk,
// or equal to it at an index no higher than ki.  Thread t handles candidates 4 t .. 4 t + 3 of
// each run of 4 kDecThreads, so thread order is candidate order and one flag prefix per run
// places the chosen ones.  Four barriers for up to 2048 candidates.  Ranges that do not bin
// (non-finite or equal extremes) and threshold bins of more than kTopkList scores take the
// radix form.
// LDS use: hist[0 .. 256) histogram, [256 .. 272) wavefront extremes, then the emission's
// wavefront counts (two alternating sets of 8), [272 .. 400) the threshold bin's (key, index)
// pairs, [400] their count.
// Publish one wavefront's key extremes (kmin, kmax: per lane) for block_topk_emit: DPP inside
// 16-lane rows, then the four rows' results, into hist[256 + wave] and hist[264 + wave].
__device__ __forceinline__ void topk_publish_extremes(uint32_t kmin, uint32_t kmax, uint32_t* hist) {
  constexpr int kWaves = kDecThreads / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  kmin = row16_min(kmin);
  kmax = row16_max(kmax);
  kmin = min(min((uint32_t)readlane_i((int)kmin, 0), (uint32_t)readlane_i((int)kmin, 16)),
             min((uint32_t)readlane_i((int)kmin, 32), (uint32_t)readlane_i((int)kmin, 48)));
  kmax = max(max((uint32_t)readlane_i((int)kmax, 0), (uint32_t)readlane_i((int)kmax, 16)),
             max((uint32_t)readlane_i((int)kmax, 32), (uint32_t)readlane_i((int)kmax, 48)));
  if (lane == 0) {
    hist[256 + wave] = kmin;
    hist[256 + kWaves + wave] = kmax;
  }
}

// hist's state that block_topk_emit expects when its caller prepared it (prepared = true): the
// histogram and the threshold bin's count cleared, and every wavefront's key extremes published
// (topk_publish_extremes over keys that bound every score of bs), followed by a barrier.
__device__ __forceinline__ void topk_clear(uint32_t* hist) {
  const int tid = threadIdx.x;
  if (tid < 256) hist[tid] = 0u;
  if (tid == 0) hist[400] = 0u;
}

__device__ __forceinline__ void block_topk_emit(const float* bs, int C, int n_take, int cand_lo, int16_t* chosen_out,
                                                uint32_t* hist, int* wave_cnt, int* pick, bool prepared = false) {
  constexpr int kPer = 4, kRun = kPer * kDecThreads, kWaves = kDecThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t* ext = hist + 256;
  uint32_t* list = hist + 272;
  uint32_t* list_n = hist + 400;
  uint32_t kmin = 0xffffffffu, kmax = 0u;
  if (!prepared) {  // extremes of the keys
    for (int c0 = 0; c0 < C; c0 += kRun) {
#pragma unroll
      for (int e = 0; e < kPer; ++e) {
        const int i = c0 + kPer * tid + e;
        if (i < C) {
          const uint32_t kk = score_key(bs[i]);
          kmin = min(kmin, kk);
          kmax = max(kmax, kk);
        }
      }
    }
    topk_publish_extremes(kmin, kmax, hist);
    topk_clear(hist);
    __syncthreads();
  }
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    kmin = min(kmin, ext[w]);
    kmax = max(kmax, ext[kWaves + w]);
  }
  const float lo = key_value(kmin), hi = key_value(kmax);
  const float scale = 256.0f / (hi - lo);
  // uniform: every thread computed the same extremes
  if (!(__builtin_isfinite(lo) && __builtin_isfinite(hi) && hi > lo && __builtin_isfinite(scale) && scale > 0.0f)) {
    radix_topk_emit(bs, C, n_take, cand_lo, chosen_out, hist, wave_cnt, pick);
    return;
  }
  for (int c0 = 0; c0 < C; c0 += kRun) {
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const int i = c0 + kPer * tid + e;
      if (i < C) atomicAdd(&hist[lin_bin(bs[i], lo, scale)], 1u);
    }
  }
  __syncthreads();
  // Every wavefront finds the bin holding the n_take-th largest score, counted from the top: lane
  // l owns bins 255 - 4 l (h.w) down to 252 - 4 l (h.x).
  int tb, above, eq;
  {
    const uint4 h = reinterpret_cast<const uint4*>(hist)[63 - lane];
    const int lsum = (int)(h.x + h.y + h.z + h.w);
    const int incl = wave_incl_scan_dpp(lsum);
    const int excl = incl - lsum;
    const uint64_t hit = __ballot(excl < n_take && n_take <= incl);
    const int src = hit ? (int)__builtin_ctzll(hit) : 0;  // exactly one lane holds the bin
    int ab = excl, d = 255 - 4 * lane, q = (int)h.w;
    if (ab + (int)h.w < n_take) {
      ab += (int)h.w; d -= 1; q = (int)h.z;
      if (ab + (int)h.z < n_take) {
        ab += (int)h.z; d -= 1; q = (int)h.y;
        if (ab + (int)h.y < n_take) { ab += (int)h.y; d -= 1; q = (int)h.x; }
      }
    }
    above = readlane_i(ab, src);
    tb = readlane_i(d, src);
    eq = readlane_i(q, src);
  }
  if (eq > kTopkList) {  // uniform
    __syncthreads();     // every wavefront has read the histogram the radix form clears
    radix_topk_emit(bs, C, n_take, cand_lo, chosen_out, hist, wave_cnt, pick);
    return;
  }
  for (int c0 = 0; c0 < C; c0 += kRun) {
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const int i = c0 + kPer * tid + e;
      if (i < C) {
        const float v = bs[i];
        if (lin_bin(v, lo, scale) == tb) {
          const uint32_t slot = atomicAdd(list_n, 1u);
          if (slot < (uint32_t)kTopkList) {
            list[2 * slot] = score_key(v);
            list[2 * slot + 1] = (uint32_t)i;
          }
        }
      }
    }
  }
  __syncthreads();
  // every wavefront ranks the bin's pairs: pairs with a larger key, or the same key at a lower index
  uint32_t kk_last;
  int ki_last;
  {
    const uint32_t mk = lane < eq ? list[2 * lane] : 0u;
    const int mi = lane < eq ? (int)list[2 * lane + 1] : 0;
    int rank = 0;
    for (int j = 0; j < eq; ++j) {
      const uint32_t jk = (uint32_t)readlane_i((int)mk, j);
      const int ji = readlane_i(mi, j);
      rank += (jk > mk || (jk == mk && ji < mi)) ? 1 : 0;
    }
    const uint64_t last = __ballot(lane < eq && rank == n_take - above - 1);
    const int src = last ? (int)__builtin_ctzll(last) : 0;
    kk_last = (uint32_t)readlane_i((int)mk, src);
    ki_last = readlane_i(mi, src);
  }
  // emission: one flag prefix per run, the wavefront counts in two alternating sets
  int base = 0;
  for (int c0 = 0, run = 0; c0 < C; c0 += kRun, ++run) {
    uint32_t* cnt = ext + kWaves * (run & 1);
    bool ch[kPer];
    int in_wave = 0, before = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const int i = c0 + kPer * tid + e;
      const uint32_t kk = score_key(bs[min(i, C - 1)]);  // in bounds for every thread
      ch[e] = i < C && (kk > kk_last || (kk == kk_last && i <= ki_last));
      const uint64_t b = __ballot(ch[e]);
      in_wave += (int)__popcll(b);
      before += mbcnt64(b);
    }
    if (lane == 0) cnt[wave] = (uint32_t)in_wave;
    __syncthreads();
    int all = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int c = (int)cnt[w];
      before += w < wave ? c : 0;
      all += c;
    }
    int pos = base + before;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      if (ch[e]) {
        if (pos < n_take) chosen_out[pos] = (int16_t)(cand_lo + c0 + kPer * tid + e);  // never past the row's slots
        ++pos;
      }
    }
    base += all;
  }
}

// The fused decode selection of query row `row` (one (batch, group) at position a.q_pos0), run by
// a workgroup of kDecThreads threads (every thread must call it): the forced blocks, the window
// scores F_row . K~_i into sc (LDS, kDecodeMaxCand floats), their max-pool to block scores on a
// windowed grid, then block_topk_emit.  hist (kTopkLds uint32, 16-byte aligned), wave_cnt
// (kDecThreads / 64 ints) and pick (3 ints) are LDS.  The row's set (a.k_total entries) goes to
// out and its count to *cnt_out (global or LDS), complete once every thread has returned and
// synchronised.
__device__ __forceinline__ void decode_select_row(const SelectArgs& a, int64_t row, float* sc, uint32_t* hist,
                                                  int* wave_cnt, int* pick, int16_t* out, int16_t* cnt_out) {

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const RowGeom g = row_geom(a.q_pos0, a.n_init, a.n_local, a.k_total);
  if (wave == 0) emit_forced(out, g, a.k_total, lane);
  if (tid == 0) *cnt_out = (int16_t)(g.n_forced + g.n_take);
  int16_t* chosen_out = out + g.init_hi;
  const int C = g.n_cand;
  if (g.n_take >= C) {
    for (int i = tid; i < C; i += kDecThreads) chosen_out[i] = (int16_t)(g.cand_lo + i);
    return;
  }
  if (g.n_take <= 0) return;

  // Window scores: lane reads dims 8*(lane%16).. of window wf + base + 4 i + lane/16 (1 KiB per
  // load) into sc[base + 4 i + lane/16].
  int32_t wf, wl;
  row_windows(g, a.grid, a.q_pos0, &wf, &wl);
  const int NW = wl - wf + 1;  // windows scored (C for the one-key-per-block grid)
  {
    const int c = lane & 15, rs = lane >> 4;
    const uint4 fw = ld16(a.f + row * kHeadDim + c * 8);
    const float f0 = bf16lo(fw.x), f1 = bf16hi(fw.x), f2 = bf16lo(fw.y), f3 = bf16hi(fw.y);
    const float f4 = bf16lo(fw.z), f5 = bf16hi(fw.z), f6 = bf16lo(fw.w), f7 = bf16hi(fw.w);
    const uint16_t* kbase = a.kc + (row * a.nc_cap + wf) * kHeadDim + c * 8;
    // Double-buffered: the next 64 windows' loads are in flight while this wave scores the
    // current ones.
    uint4 kw[16], kn[16];
    uint32_t kmin = 0xffffffffu, kmax = 0u;  // key extremes of the scores this lane stores
    topk_clear(hist);
    // Indices past the last window read the last one again (never stored), so the loads stay
    // branch-free.
    auto load = [&](int base, uint4 (&w)[16]) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int idx = min(base + 4 * i + rs, NW - 1);
        w[i] = ld16_nt(kbase + (int64_t)idx * kHeadDim);
      }
    };
    int base = wave * 64;
    if (base < NW) load(base, kw);
    for (; base < NW; base += kDecThreads) {
      if (base + kDecThreads < NW) load(base + kDecThreads, kn);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float d = f0 * bf16lo(kw[i].x);
        d = fmaf(f1, bf16hi(kw[i].x), d);
        d = fmaf(f2, bf16lo(kw[i].y), d);
        d = fmaf(f3, bf16hi(kw[i].y), d);
        d = fmaf(f4, bf16lo(kw[i].z), d);
        d = fmaf(f5, bf16hi(kw[i].z), d);
        d = fmaf(f6, bf16lo(kw[i].w), d);
        d = fmaf(f7, bf16hi(kw[i].w), d);
        d = row16_sum(d);
        const int idx = base + 4 * i + rs;
        if (c == 0 && idx < NW) {
          sc[idx] = d;
          const uint32_t kk = score_key(d);
          kmin = min(kmin, kk);
          kmax = max(kmax, kk);
        }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) kw[i] = kn[i];
    }
    // the window scores bound the (max-pooled) block scores: the top-k's bins need no pass of
    // their own
    topk_publish_extremes(kmin, kmax, hist);
  }
  __syncthreads();
  // Block scores: the window scores themselves, or their max-pool into sc[NW .. NW + C).
  const float* bs = sc;
  if (!grid_is_blocks(a.grid)) {
    const int32_t wvis = grid_win_vis(a.grid, a.q_pos0);
    for (int i = tid; i < C; i += kDecThreads) {
      const int32_t j = g.cand_lo + i;
      const int32_t lo = grid_win_lo(a.grid, j), hi = min(grid_win_hi(a.grid, j), wvis);
      float m = sc[lo - wf];
      for (int32_t w = lo + 1; w <= hi; ++w) m = fmaxf(m, sc[w - wf]);
      sc[NW + i] = m;
    }
    bs = sc + NW;
    __syncthreads();
  }

  block_topk_emit(bs, C, g.n_take, g.cand_lo, chosen_out, hist, wave_cnt, pick, true);
}

// Max-pooled score of candidate i (block cand_lo + i) over the window scores w[0 .. ] of windows
// wf, wf + 1, ...: the windows that overlap the block and are complete at the row's position.
__device__ __forceinline__ float pooled_score(const float* w, const WinGrid& grid, int32_t j, int32_t wf,
                                              int32_t wvis) {
  const int32_t lo = grid_win_lo(grid, j), hi = min(grid_win_hi(grid, j), wvis);
  float m = w[lo - wf];
  for (int32_t i = lo + 1; i <= hi; ++i) m = fmaxf(m, w[i - wf]);
  return m;
}

// The split decode path's selection of row `row`: its window scores are already in the
// workspace (row stride a.ws_stride, window wf at offset 0).  They are loaded into sc (LDS,
// kDecodeMaxCand floats), max-pooled to block scores on a windowed grid, and block_topk_emit
// selects; the set goes to out and the count to *cnt_out, complete once every thread has
// returned and synchronised.  Every thread of a kDecThreads workgroup must call it.
__device__ __forceinline__ void decode_topk_row(const SelectArgs& a, int64_t row, float* sc, uint32_t* hist,
                                                int* wave_cnt, int* pick, int16_t* out, int16_t* cnt_out) {

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const RowGeom g = row_geom(a.q_pos0, a.n_init, a.n_local, a.k_total);
  if (wave == 0) emit_forced(out, g, a.k_total, lane);
  if (tid == 0) *cnt_out = (int16_t)(g.n_forced + g.n_take);
  int16_t* chosen_out = out + g.init_hi;
  const int C = g.n_cand;
  if (g.n_take >= C) {
    for (int i = tid; i < C; i += kDecThreads) chosen_out[i] = (int16_t)(g.cand_lo + i);
    return;
  }
  if (g.n_take <= 0) return;
  int32_t wf, wl;
  row_windows(g, a.grid, a.q_pos0, &wf, &wl);
  const int NW = wl - wf + 1;
  const float* src = a.ws + row * a.ws_stride;
  // Sixteen loads in flight per thread before any is stored (indices past the row read its last
  // score again and are not stored): one memory latency per 8192 scores instead of sixteen.
  constexpr int kLdBatch = 16;
  uint32_t kmin = 0xffffffffu, kmax = 0u;  // key extremes of the scores this thread stores
  topk_clear(hist);
  for (int b0 = 0; b0 < NW; b0 += kLdBatch * kDecThreads) {
    float t[kLdBatch];
#pragma unroll
    for (int k = 0; k < kLdBatch; ++k) t[k] = src[min(b0 + k * kDecThreads + tid, NW - 1)];
#pragma unroll
    for (int k = 0; k < kLdBatch; ++k)
      if (b0 + k * kDecThreads + tid < NW) {
        sc[b0 + k * kDecThreads + tid] = t[k];
        const uint32_t kk = score_key(t[k]);
        kmin = min(kmin, kk);
        kmax = max(kmax, kk);
      }
  }
  topk_publish_extremes(kmin, kmax, hist);
  __syncthreads();
  const float* bs = sc;
  if (!grid_is_blocks(a.grid)) {
    const int32_t wvis = grid_win_vis(a.grid, a.q_pos0);
    for (int i = tid; i < C; i += kDecThreads) sc[NW + i] = pooled_score(sc, a.grid, g.cand_lo + i, wf, wvis);
    bs = sc + NW;
    __syncthreads();
  }
  block_topk_emit(bs, C, g.n_take, g.cand_lo, chosen_out, hist, wave_cnt, pick, true);
}

}  // namespace sparda

// select_multihead.hip -- the InfLLM-V2 multi-head block selector (paper Sec. 3, "three-stage
// block representation"), the baseline that the Forecast indexer of Sec. 4.1 replaces.
//
// Per query row at position p of group m: each of the group's G query heads scores every
// compressed key complete at p (windows 0 .. vis(p)), z_hi = scale * q_h . K~_i; a softmax over i
// turns each head's scores into weights; the shared score of window i is the sum of the G heads'
// weights; a block's score is the max-pool of the shared scores over the windows that overlap it
// and are complete at p; the top-k candidates join the forced blocks exactly as in select.hip.
//
// Scores are taken in the exp2 domain (scale * log2 e folded into the query row) with float32
// accumulation, and each head's softmax subtracts that head's exact maximum, so every exponent
// is <= 0.
//
// Paths:
//  * fused decode (n_q == 1, G in {1, 2, 4, 8}, G * windows + candidates <= kMhLdsFloats): one
//    512-thread workgroup per (batch, group) row.  K~ is read once, 1 KiB per wavefront load as
//    in the Forecast decode kernel, and each loaded window is scored by all G heads into LDS;
//    the per-head maximum and sum, the shared scores, the max-pool and the block-wide top-k
//    (select_block.hpp) all stay on the CU.
//  * fused two-pass decode (n_q == 1, any other G <= 16, windows + candidates <= kMhLdsFloats):
//    a 16-window tile times the group's heads is one MFMA chain (A = 16 windows' keys, B = the
//    G query rows padded to 16 columns).  Pass 1 keeps an online maximum and sum of 2^z per head,
//    pass 2 reads the keys again and adds each head's normalised weight into the shared score
//    of the window, in LDS.
//  * multi-row tiles (at least 16 rows, G in {1, 2, 4, 8, 16}): mh_tile_kernel scores 64 (row,
//    head) columns per unit on MFMA in two passes (per-head maximum and sum, then the normalised
//    weights summed over each row's heads) into the shared scores of the workspace, and
//    select.hip's row-wise top-k pools and selects.
//  * row-wise (everything else): mh_score_kernel writes every head's score of every complete
//    window of every row to the workspace, mh_norm_kernel (one workgroup per row) turns them into
//    the shared scores of the windows that overlap the row's candidates, and the same row-wise
//    top-k pools and selects.
#include <math.h>

#include "device_util.hpp"
#include "launch.hpp"
#include "head_tiles.hpp"
#include "select_block.hpp"

namespace sparda {

constexpr int kMhLdsFloats = 38400;  // fused decode: G * windows + candidates floats (150 KiB)
constexpr int kMhMaxRowG = 16;
constexpr int kMhTileMinRows = 16;  // multi-row calls with at least this many rows use MFMA tiles

__device__ __forceinline__ float wave_max_f(float x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x = fmaxf(x, __shfl_xor(x, d, kWave));
  return x;
}
__device__ __forceinline__ float wave_sum_f(float x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, kWave);
  return x;
}

// 8 query dims as floats, scaled into the exp2 domain.
__device__ __forceinline__ void load_q8(const uint16_t* src, float s, float (&q)[8]) {
  const uint4 w = ld16(src);
  q[0] = bf16lo(w.x) * s; q[1] = bf16hi(w.x) * s; q[2] = bf16lo(w.y) * s; q[3] = bf16hi(w.y) * s;
  q[4] = bf16lo(w.z) * s; q[5] = bf16hi(w.z) * s; q[6] = bf16lo(w.w) * s; q[7] = bf16hi(w.w) * s;
}

__device__ __forceinline__ float dot8(const float (&q)[8], const uint4& k) {
  float d = q[0] * bf16lo(k.x);
  d = fmaf(q[1], bf16hi(k.x), d);
  d = fmaf(q[2], bf16lo(k.y), d);
  d = fmaf(q[3], bf16hi(k.y), d);
  d = fmaf(q[4], bf16lo(k.z), d);
  d = fmaf(q[5], bf16hi(k.z), d);
  d = fmaf(q[6], bf16lo(k.w), d);
  d = fmaf(q[7], bf16hi(k.w), d);
  return d;
}

// ---- fused decode ---------------------------------------------------------------------------

template <int G>
__global__ __launch_bounds__(kDecThreads) void mh_decode_kernel(SelectArgs a) {
  __shared__ float zs[kMhLdsFloats];  // head h's score of window i at zs[h NV + i]
  __shared__ __align__(16) uint32_t hist[kTopkLds];
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  __shared__ float red[kDecThreads / 64][G];
  const int64_t row = blockIdx.x;  // b * Hkv + m
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t p = a.q_pos0;
  const RowGeom g = row_geom(p, a.n_init, a.n_local, a.k_total);
  int16_t* out = a.sel + row * a.k_total;
  if (wave == 0) emit_forced(out, g, a.k_total, lane);
  if (tid == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
  int16_t* chosen_out = out + g.init_hi;
  const int C = g.n_cand;
  if (g.n_take >= C) {
    for (int i = tid; i < C; i += kDecThreads) chosen_out[i] = (int16_t)(g.cand_lo + i);
    return;
  }
  if (g.n_take <= 0) return;
  const int NV = grid_win_vis(a.grid, p) + 1;  // windows 0 .. NV - 1 (the host checked NV <= nc_cap)

  {  // scores: lane reads dims 8 (lane % 16) .. of window base + 4 i + lane / 16
    const int c = lane & 15, rs = lane >> 4;
    float qf[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) load_q8(a.q + (row * G + h) * kHeadDim + c * 8, a.scale_log2, qf[h]);
    const uint16_t* kbase = a.kc + row * a.nc_cap * kHeadDim + c * 8;
    uint4 kw[16], kn[16];
    auto load = [&](int base, uint4 (&w)[16]) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int idx = min(base + 4 * i + rs, NV - 1);  // past the last window: a repeat, never stored
        w[i] = ld16(kbase + (int64_t)idx * kHeadDim);
      }
    };
    int base = wave * 64;
    if (base < NV) load(base, kw);
    for (; base < NV; base += kDecThreads) {
      if (base + kDecThreads < NV) load(base + kDecThreads, kn);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int idx = base + 4 * i + rs;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float d = row16_sum(dot8(qf[h], kw[i]));
          if (c == h && idx < NV) zs[h * NV + idx] = d;
        }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) kw[i] = kn[i];
    }
  }
  __syncthreads();

  // Per-head softmax over the NV windows: exact maximum, then exp2 and the sum.
  float mx[G], inv[G];
#pragma unroll
  for (int h = 0; h < G; ++h) mx[h] = -INFINITY;
  for (int i = tid; i < NV; i += kDecThreads)
#pragma unroll
    for (int h = 0; h < G; ++h) mx[h] = fmaxf(mx[h], zs[h * NV + i]);
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float m = wave_max_f(mx[h]);
    if (lane == 0) red[wave][h] = m;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float m = red[0][h];
#pragma unroll
    for (int w = 1; w < kDecThreads / 64; ++w) m = fmaxf(m, red[w][h]);
    mx[h] = m;
    inv[h] = 0.f;
  }
  __syncthreads();
  for (int i = tid; i < NV; i += kDecThreads)
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float e = exp2f(zs[h * NV + i] - mx[h]);
      zs[h * NV + i] = e;
      inv[h] += e;
    }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float s = wave_sum_f(inv[h]);
    if (lane == 0) red[wave][h] = s;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kDecThreads / 64; ++w) s += red[w][h];
    inv[h] = 1.0f / s;
  }
  // Shared scores over head 0's slots: each thread reads and writes only its own windows.
  for (int i = tid; i < NV; i += kDecThreads) {
    float s = 0.f;
#pragma unroll
    for (int h = 0; h < G; ++h) s = fmaf(zs[h * NV + i], inv[h], s);
    zs[i] = s;
  }
  __syncthreads();

  // Block scores: max-pool of the shared scores (the identity on the one-key-per-block grid).
  float* bs = zs + G * NV;
  for (int i = tid; i < C; i += kDecThreads) {
    const int32_t j = g.cand_lo + i;
    const int32_t lo = grid_win_lo(a.grid, j), hi = min(grid_win_hi(a.grid, j), NV - 1);
    float m = zs[lo];
    for (int32_t w = lo + 1; w <= hi; ++w) m = fmaxf(m, zs[w]);
    bs[i] = m;
  }
  __syncthreads();
  block_topk_emit(bs, C, g.n_take, g.cand_lo, chosen_out, hist, wave_cnt, pick);
}

// ---- fused two-pass decode (MFMA scores) ------------------------------------------------------

// Lane l of a wavefront: column n = l % 16 (head n of the group), lane group j = l / 16.  A window
// tile t covers windows 16 t .. 16 t + 15; the accumulator element e of lane (n, j) is head n's
// score of window 16 t + 4 j + e.
__global__ __launch_bounds__(kDecThreads) void mh_decode2_kernel(SelectArgs a) {
  __shared__ float zs[kMhLdsFloats];  // shared scores of windows [0, NV), then block scores
  __shared__ __align__(16) uint32_t hist[kTopkLds];
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  __shared__ float red_m[kDecThreads / 64][16], red_s[kDecThreads / 64][16];
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, j = lane >> 4;
  const int G = a.group_size;
  const int64_t p = a.q_pos0;
  const RowGeom g = row_geom(p, a.n_init, a.n_local, a.k_total);
  int16_t* out = a.sel + row * a.k_total;
  if (wave == 0) emit_forced(out, g, a.k_total, lane);
  if (tid == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
  int16_t* chosen_out = out + g.init_hi;
  const int C = g.n_cand;
  if (g.n_take >= C) {
    for (int i = tid; i < C; i += kDecThreads) chosen_out[i] = (int16_t)(g.cand_lo + i);
    return;
  }
  if (g.n_take <= 0) return;
  const int NV = grid_win_vis(a.grid, p) + 1;
  const int n_tiles = (NV + 15) >> 4;

  // B: head n's dims 8 j + 32 ks .. + 7 (zero columns past the group's heads)
  bf16x8 qb[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {  // columns past the heads read head 0 (a valid address), zeroed
    const uint4 v = ld16(a.q + (row * G + (n < G ? n : 0)) * kHeadDim + 8 * j + 32 * ks);
    qb[ks] = as_bf16x8(n < G ? v : make_uint4(0u, 0u, 0u, 0u));
  }
  // A: window 16 t + n's dims 8 j + 32 ks .. + 7 (windows past the last read the last again)
  const uint16_t* kb = a.kc + row * a.nc_cap * kHeadDim + 8 * j;
  auto load_tile = [&](int t, uint4 (&w)[4]) {
    const int win = min(16 * t + n, NV - 1);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) w[ks] = ld16(kb + (int64_t)win * kHeadDim + 32 * ks);
  };
  auto score_tile = [&](const uint4 (&w)[4], int t, float (&z)[4]) {
    f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(as_bf16x8(w[ks]), qb[ks], c);
#pragma unroll
    for (int e = 0; e < 4; ++e) z[e] = 16 * t + 4 * j + e < NV ? c[e] * a.scale_log2 : -INFINITY;
  };

  // Pass 1: online maximum and sum of 2^z per lane, then per head (column n).
  float m_run = -INFINITY, s_run = 0.f;
  {
    uint4 w0[4], w1[4];
    int t = wave;
    if (t < n_tiles) load_tile(t, w0);
    for (; t < n_tiles; t += 2 * (kDecThreads / 64)) {
      const int t1 = t + kDecThreads / 64;
      if (t1 < n_tiles) load_tile(t1, w1);
      float z[4];
      score_tile(w0, t, z);
      float mt = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
      float mn = fmaxf(m_run, mt);
      if (mn > -INFINITY) {
        s_run = s_run * exp2f(m_run - mn) + exp2f(z[0] - mn) + exp2f(z[1] - mn) + exp2f(z[2] - mn) + exp2f(z[3] - mn);
        m_run = mn;
      }
      if (t1 >= n_tiles) break;
      const int t2 = t1 + kDecThreads / 64;
      if (t2 < n_tiles) load_tile(t2, w0);
      score_tile(w1, t1, z);
      mt = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
      mn = fmaxf(m_run, mt);
      if (mn > -INFINITY) {
        s_run = s_run * exp2f(m_run - mn) + exp2f(z[0] - mn) + exp2f(z[1] - mn) + exp2f(z[2] - mn) + exp2f(z[3] - mn);
        m_run = mn;
      }
    }
  }
  // combine the four lane groups of each column, then the wavefronts
  auto merge = [](float& m, float& s, float m2, float s2) {
    const float mn = fmaxf(m, m2);
    if (mn > -INFINITY) {
      s = s * exp2f(m - mn) + s2 * exp2f(m2 - mn);
      m = mn;
    }
  };
  merge(m_run, s_run, __shfl_xor(m_run, 16, kWave), __shfl_xor(s_run, 16, kWave));
  merge(m_run, s_run, __shfl_xor(m_run, 32, kWave), __shfl_xor(s_run, 32, kWave));
  if (lane < 16) {
    red_m[wave][n] = m_run;
    red_s[wave][n] = s_run;
  }
  __syncthreads();
  float M = red_m[0][n], S = red_s[0][n];
#pragma unroll
  for (int w = 1; w < kDecThreads / 64; ++w) merge(M, S, red_m[w][n], red_s[w][n]);
  const float inv = n < G ? 1.0f / S : 0.f;  // columns past the group's heads add nothing

  // Pass 2: the shared score of each window, the sum over the columns of each lane group.
  {
    uint4 w0[4];
    for (int t = wave; t < n_tiles; t += kDecThreads / 64) {
      load_tile(t, w0);
      float z[4];
      score_tile(w0, t, z);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float sh = row16_sum(n < G ? exp2f(z[e] - M) * inv : 0.f);
        const int win = 16 * t + 4 * j + e;
        if (n == e && win < NV) zs[win] = sh;
      }
    }
  }
  __syncthreads();

  float* bs = zs + NV;
  for (int i = tid; i < C; i += kDecThreads) {
    const int32_t jb = g.cand_lo + i;
    const int32_t lo = grid_win_lo(a.grid, jb), hi = min(grid_win_hi(a.grid, jb), NV - 1);
    float m = zs[lo];
    for (int32_t w = lo + 1; w <= hi; ++w) m = fmaxf(m, zs[w]);
    bs[i] = m;
  }
  __syncthreads();
  block_topk_emit(bs, C, g.n_take, g.cand_lo, chosen_out, hist, wave_cnt, pick);
}

// ---- row-wise path --------------------------------------------------------------------------

// grid.x = row * n_chunks + chunk; a chunk is 256 windows, 64 per wavefront.  Head h's score of
// window i goes to ws[row * ws_stride + h * hstride + i].
__global__ __launch_bounds__(256) void mh_score_kernel(SelectArgs a, int n_chunks, int64_t hstride) {
  const int64_t row = blockIdx.x / n_chunks;
  const int chunk = (int)(blockIdx.x % n_chunks);
  const int r = (int)(row % a.n_q);
  const int64_t bm = row / a.n_q;
  const int64_t p = a.q_pos0 + r;
  const RowGeom g = row_geom(p, a.n_init, a.n_local, a.k_total);
  if (g.n_take >= g.n_cand) return;  // the row takes every candidate: no scores needed
  const int NV = grid_win_vis(a.grid, p) + 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, rs = lane >> 4;
  const int first = chunk * 256 + wave * 64;
  if (first >= NV) return;
  const uint16_t* kbase = a.kc + bm * a.nc_cap * kHeadDim + c * 8;
  uint4 kw[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) kw[i] = ld16(kbase + (int64_t)min(first + 4 * i + rs, NV - 1) * kHeadDim);
  float* zrow = a.ws + row * a.ws_stride;
  // Lane c keeps head c's scores (c < G), so that each window's G scores leave in one store.
  float keep[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) keep[i] = 0.f;
  for (int h = 0; h < a.group_size; ++h) {
    float qf[8];
    load_q8(a.q + ((bm * a.group_size + h) * a.n_q + r) * kHeadDim + c * 8, a.scale_log2, qf);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float d = row16_sum(dot8(qf, kw[i]));
      keep[i] = c == h ? d : keep[i];
    }
  }
  if (c < a.group_size) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int idx = first + 4 * i + rs;
      if (idx < NV) zrow[c * hstride + idx] = keep[i];
    }
  }
}

// One workgroup per row: each head's maximum and sum over the row's complete windows, then the
// shared score of every window that overlaps a candidate, written after the G heads' rows at
// offset (window - first such window), where select.hip's row-wise top-k reads it.
__global__ __launch_bounds__(256) void mh_norm_kernel(SelectArgs a, int64_t hstride) {
  __shared__ float red[4][kMhMaxRowG];
  __shared__ float mx[kMhMaxRowG], inv[kMhMaxRowG];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t row = blockIdx.x;
  const int r = (int)(row % a.n_q);
  const int64_t p = a.q_pos0 + r;
  const RowGeom g = row_geom(p, a.n_init, a.n_local, a.k_total);
  if (g.n_take >= g.n_cand) return;
  const int G = a.group_size;
  const int NV = grid_win_vis(a.grid, p) + 1;
  int32_t wf, wl;
  row_windows(g, a.grid, p, &wf, &wl);
  const float* zrow = a.ws + row * a.ws_stride;
  float* shared = a.ws + row * a.ws_stride + G * hstride;
  for (int h = 0; h < G; ++h) {
    float m = -INFINITY;
    for (int i = tid; i < NV; i += 256) m = fmaxf(m, zrow[h * hstride + i]);
    m = wave_max_f(m);
    if (lane == 0) red[wave][h] = m;
  }
  __syncthreads();
  if (tid < G) mx[tid] = fmaxf(fmaxf(red[0][tid], red[1][tid]), fmaxf(red[2][tid], red[3][tid]));
  __syncthreads();
  for (int h = 0; h < G; ++h) {
    const float m = mx[h];
    float s = 0.f;
    for (int i = tid; i < NV; i += 256) s += exp2f(zrow[h * hstride + i] - m);
    s = wave_sum_f(s);
    if (lane == 0) red[wave][h] = s;
  }
  __syncthreads();
  if (tid < G) inv[tid] = 1.0f / (red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid]);
  __syncthreads();
  for (int i = wf + tid; i <= wl; i += 256) {
    float s = 0.f;
    for (int h = 0; h < G; ++h) s = fmaf(exp2f(zrow[h * hstride + i] - mx[h]), inv[h], s);
    shared[i - wf] = s;
  }
}

// ---- multi-row tiles (MFMA, two passes) ------------------------------------------------------
//
// Multi-row calls with G in {1, 2, 4, 8, 16}: a unit is U = 64 / G consecutive rows of one
// (batch, group) with their heads, 64 (row, head) columns (head_tiles.hpp), scored against the
// windows complete at the unit's last row; each row stores its shared scores of the windows
// [wf, wl] it selects from, where the row-wise top-k reads them (window wf + x at slot x).

template <int G>
__global__ __launch_bounds__(kMtThreads) void mh_tile_kernel(SelectArgs a, int n_units, int64_t hstride) {
  constexpr int U = 64 / G;
  __shared__ float red_m[kMtWaves][64], red_s[kMtWaves][64];
  const int lane = threadIdx.x & 63;
  const int n = lane & 31;
  const int n_groups = a.batch * a.n_kv_heads;
  const int grp = blockIdx.x % n_groups;
  const int unit = n_units - 1 - (int)(blockIdx.x / n_groups);  // latest rows (most windows) first
  const int r0 = unit * U;
  const int nr = min(U, a.n_q - r0);
  const int64_t p_last = a.q_pos0 + r0 + nr - 1;
  const RowGeom gl = row_geom(p_last, a.n_init, a.n_local, a.k_total);
  if (gl.n_take >= gl.n_cand) return;  // then every row of the unit takes all its candidates
  HeadTileRows t;
  t.n_keys = grid_win_vis(a.grid, p_last) + 1;
  t.lo = 0;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int c = 32 * nt + n;
    const int rr = min(c / G, nr - 1);
    const int64_t p = a.q_pos0 + r0 + rr;
    t.q[nt] = reinterpret_cast<const uint4*>(a.q) + (((int64_t)grp * G + c % G) * a.n_q + r0 + rr) * kMtRowU4;
    t.vis[nt] = grid_win_vis(a.grid, p);
    const RowGeom g = row_geom(p, a.n_init, a.n_local, a.k_total);
    int32_t wf, wl;
    row_windows(g, a.grid, p, &wf, &wl);
    t.lo = wf;  // the same for every row
    const bool own = (n % G) == 0 && c / G < nr && g.n_take < g.n_cand;
    t.hi[nt] = own ? wl : -1;
    t.out[nt] = a.ws + ((int64_t)grp * a.n_q + r0 + rr) * a.ws_stride + G * hstride;
  }
  head_tile_shared_weights<G>(t, reinterpret_cast<const uint4*>(a.kc) + (int64_t)grp * a.nc_cap * kMtRowU4,
                              a.scale_log2, red_m, red_s);
}

// ---- host -----------------------------------------------------------------------------------

enum MhPath { kMhOnePass, kMhTwoPass, kMhRowwise };

static MhPath mh_path(int32_t G, int32_t n_q, int64_t q_pos0, int32_t n_init, int32_t n_local, WinGrid grid) {
  if (n_q != 1 || G > 16) return kMhRowwise;
  const RowGeom g = row_geom(q_pos0, n_init, n_local, 1 << 30);
  const int64_t nv = (int64_t)grid_win_vis(grid, q_pos0) + 1;
  if ((G == 1 || G == 2 || G == 4 || G == 8) && (int64_t)G * nv + g.n_cand <= kMhLdsFloats) return kMhOnePass;
  return nv + g.n_cand <= kMhLdsFloats ? kMhTwoPass : kMhRowwise;
}

size_t multihead_ws_floats(int64_t rows, int32_t group_size, int32_t n_q, int64_t q_pos0, int32_t n_init,
                           int32_t n_local, int32_t k_total, WinGrid grid, int64_t* stride) {
  *stride = 0;
  if (mh_path(group_size, n_q, q_pos0, n_init, n_local, grid) != kMhRowwise) return 0;
  const int64_t pl = q_pos0 + n_q - 1;  // the last row scores the most windows
  const RowGeom gl = row_geom(pl, n_init, n_local, k_total);
  if (gl.n_take >= gl.n_cand) return 0;  // then every row takes all of its candidates
  const int64_t nv = (int64_t)grid_win_vis(grid, pl) + 1;
  const int64_t hstride = (nv + 3) & ~(int64_t)3;
  *stride = (group_size + 1) * hstride;
  return (size_t)rows * (size_t)*stride;
}

hipError_t launch_multihead_select(const SelectArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads * a.n_q;
  const int G = a.group_size;
  const MhPath path = mh_path(G, a.n_q, a.q_pos0, a.n_init, a.n_local, a.grid);
  if (path == kMhTwoPass) {
    hipLaunchKernelGGL(mh_decode2_kernel, dim3((unsigned)rows), dim3(kDecThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (path == kMhOnePass) {
    const dim3 grid((unsigned)rows), block(kDecThreads);
    switch (G) {
      case 1: hipLaunchKernelGGL(mh_decode_kernel<1>, grid, block, 0, stream, a); break;
      case 2: hipLaunchKernelGGL(mh_decode_kernel<2>, grid, block, 0, stream, a); break;
      case 4: hipLaunchKernelGGL(mh_decode_kernel<4>, grid, block, 0, stream, a); break;
      default: hipLaunchKernelGGL(mh_decode_kernel<8>, grid, block, 0, stream, a); break;
    }
    return hipGetLastError();
  }
  if (G > kMhMaxRowG) return hipErrorInvalidValue;
  SelectArgs t = a;
  if (a.ws_stride > 0) {  // some row scores its candidates
    const int64_t hstride = a.ws_stride / (G + 1);
    const int64_t pl = a.q_pos0 + a.n_q - 1;
    const int nv = grid_win_vis(a.grid, pl) + 1;
    const bool tiles = a.n_q >= kMhTileMinRows && (G == 1 || G == 2 || G == 4 || G == 8 || G == 16);
    if (tiles) {  // many rows: units of 64 (row, head) columns on MFMA, both passes in one kernel
      const int n_units = (a.n_q + 64 / G - 1) / (64 / G);
      const dim3 grid((unsigned)((int64_t)n_units * a.batch * a.n_kv_heads)), block(kMtThreads);
      switch (G) {
        case 1: hipLaunchKernelGGL(mh_tile_kernel<1>, grid, block, 0, stream, a, n_units, hstride); break;
        case 2: hipLaunchKernelGGL(mh_tile_kernel<2>, grid, block, 0, stream, a, n_units, hstride); break;
        case 4: hipLaunchKernelGGL(mh_tile_kernel<4>, grid, block, 0, stream, a, n_units, hstride); break;
        case 8: hipLaunchKernelGGL(mh_tile_kernel<8>, grid, block, 0, stream, a, n_units, hstride); break;
        default: hipLaunchKernelGGL(mh_tile_kernel<16>, grid, block, 0, stream, a, n_units, hstride); break;
      }
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    } else {
      const int n_chunks = (nv + 255) / 256;
      hipLaunchKernelGGL(mh_score_kernel, dim3((unsigned)(rows * n_chunks)), dim3(256), 0, stream, a, n_chunks,
                         hstride);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(mh_norm_kernel, dim3((unsigned)rows), dim3(256), 0, stream, a, hstride);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    t.ws = a.ws + G * hstride;  // the shared scores; the row stride stays ws_stride
  }
  return launch_rowwise_topk(t, stream);
}

}  // namespace sparda

// head_tiles.hpp -- per-head softmax weights over compressed keys, summed over a GQA group, for
// 64 (row, head) columns at a time on 32x32x16 MFMA.  Shared by the multi-head selector's
// multi-row path (Sec. 3, the InfLLM-V2 selector) and the indexer-training target (Sec. 4.2,
// Eq. 6), which apply the same per-head softmax and group sum to different keys.
//
// A unit is 64 / G rows of one (batch, group) with their G heads each: column c is head c % G of
// row c / G, the B operand as two N-tiles of 32 columns.  The four wavefronts of a 256-thread
// workgroup take every fourth M-tile of 32 keys over [0, n_keys), reading the key fragments from
// L2 one M-tile ahead.  The dimension order of the contraction is free: lane half h of k-step
// 4 u + i holds dimensions 64 u + 32 h + 8 i .. + 7 of both operands.  Accumulator element e of
// lane (n, h) is key 8 (e / 4) + 4 h + e % 4 of the M-tile for column n.
//  * pass 1: per column, an online maximum and sum of 2^z over the keys the column's row sees
//    (z = scale * log2 e * q . k); lane halves and wavefronts merge through LDS;
//  * pass 2: the same products again; each column's normalised weight, summed over the G
//    adjacent lanes of its row by shuffles, is the row's shared weight of the key, stored by the
//    row's first lane.
#pragma once
#include "device_util.hpp"

namespace sparda {

constexpr int kMtThreads = 256;
constexpr int kMtWaves = kMtThreads / kWave;
constexpr int kMtRowU4 = kHeadDim * 2 / 16;  // 16-byte pieces per 128-dim bf16 row

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ void mt_load_frags(const uint4* row, int h, uint4 (&x)[8]) {
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) x[4 * u + i] = row[8 * u + 4 * h + i];
}

__device__ __forceinline__ void mt_mma(const uint4 (&a)[8], const uint4 (&fb)[2][8], f32x16& c0, f32x16& c1) {
#pragma unroll
  for (int e = 0; e < 16; ++e) c0[e] = c1[e] = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const bf16x8 av = as_bf16x8(a[s]);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(fb[0][s]), c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(fb[1][s]), c1, 0, 0, 0);
  }
}

// What a lane needs about its two columns (32 nt + lane % 32, nt = 0, 1).
struct HeadTileRows {
  const uint4* q[2];  // the column's query row (128 bf16)
  int vis[2];         // keys 0 .. vis count for the column's row (vis < 0: none)
  float* out[2];      // the row's output: key i goes to out[i - lo]
  int lo;             // first key stored
  int hi[2];          // last key stored by this lane (-1: the lane stores nothing)
  int n_keys;         // keys scored: 0 .. n_keys - 1 (the unit's largest vis + 1)
};

// Every thread of the 256-thread workgroup calls it.  kc: key 0 of the group; red_m, red_s: LDS.
template <int G>
__device__ __forceinline__ void head_tile_shared_weights(const HeadTileRows& t, const uint4* kc, float sl2,
                                                         float (&red_m)[kMtWaves][64], float (&red_s)[kMtWaves][64]) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int NV = t.n_keys;
  const int n_mt = (NV + 31) / 32;
  uint4 fb[2][8];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) mt_load_frags(t.q[nt], h, fb[nt]);
  auto arow = [&](int mt) { return kc + (int64_t)min(32 * min(mt, n_mt - 1) + n, NV - 1) * kMtRowU4; };

  // Pass 1: online maximum and sum of 2^z per column.
  float mr[2] = {-INFINITY, -INFINITY}, sr[2] = {0.f, 0.f};
  auto fold = [&](int mt, const f32x16& c0, const f32x16& c1) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const f32x16& c = nt == 0 ? c0 : c1;
      float z[16];
      float mt_max = -INFINITY;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = 32 * mt + 8 * (e >> 2) + 4 * h + (e & 3);
        z[e] = key <= t.vis[nt] ? c[e] * sl2 : -INFINITY;
        mt_max = fmaxf(mt_max, z[e]);
      }
      const float mn = fmaxf(mr[nt], mt_max);
      if (mn > -INFINITY) {
        float acc = sr[nt] * exp2f(mr[nt] - mn);
#pragma unroll
        for (int e = 0; e < 16; ++e) acc += exp2f(z[e] - mn);
        sr[nt] = acc;
        mr[nt] = mn;
      }
    }
  };
  if (w < n_mt) {
    uint4 ab[2][8];
    mt_load_frags(arow(w), h, ab[0]);
    for (int mt = w; mt < n_mt; mt += 2 * kMtWaves) {
      mt_load_frags(arow(mt + kMtWaves), h, ab[1]);
      __builtin_amdgcn_sched_barrier(0);  // keep the request ahead of the products
      f32x16 c0, c1;
      mt_mma(ab[0], fb, c0, c1);
      fold(mt, c0, c1);
      mt_load_frags(arow(mt + 2 * kMtWaves), h, ab[0]);
      __builtin_amdgcn_sched_barrier(0);
      if (mt + kMtWaves < n_mt) {
        mt_mma(ab[1], fb, c0, c1);
        fold(mt + kMtWaves, c0, c1);
      }
    }
  }
  auto merge = [](float& m, float& s, float m2, float s2) {
    const float mn = fmaxf(m, m2);
    if (mn > -INFINITY) {
      s = s * exp2f(m - mn) + s2 * exp2f(m2 - mn);
      m = mn;
    }
  };
  float M[2], inv[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    merge(mr[nt], sr[nt], __shfl_xor(mr[nt], 32, kWave), __shfl_xor(sr[nt], 32, kWave));
    if (h == 0) {
      red_m[w][32 * nt + n] = mr[nt];
      red_s[w][32 * nt + n] = sr[nt];
    }
  }
  __syncthreads();
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    float m = red_m[0][32 * nt + n], sm = red_s[0][32 * nt + n];
#pragma unroll
    for (int v = 1; v < kMtWaves; ++v) merge(m, sm, red_m[v][32 * nt + n], red_s[v][32 * nt + n]);
    M[nt] = m;
    inv[nt] = sm > 0.f ? 1.0f / sm : 0.f;
  }

  // Pass 2: each row's shared weight of every key it stores.
  auto emit = [&](int mt, const f32x16& c0, const f32x16& c1) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const f32x16& c = nt == 0 ? c0 : c1;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = 32 * mt + 8 * (e >> 2) + 4 * h + (e & 3);
        float wt = key <= t.vis[nt] ? exp2f(c[e] * sl2 - M[nt]) * inv[nt] : 0.f;
#pragma unroll
        for (int d = 1; d < G; d <<= 1) wt += __shfl_xor(wt, d, kWave);
        if (key >= t.lo && key <= t.hi[nt]) t.out[nt][key - t.lo] = wt;
      }
    }
  };
  if (w < n_mt) {
    uint4 ab[2][8];
    mt_load_frags(arow(w), h, ab[0]);
    for (int mt = w; mt < n_mt; mt += 2 * kMtWaves) {
      mt_load_frags(arow(mt + kMtWaves), h, ab[1]);
      __builtin_amdgcn_sched_barrier(0);
      f32x16 c0, c1;
      mt_mma(ab[0], fb, c0, c1);
      emit(mt, c0, c1);
      mt_load_frags(arow(mt + 2 * kMtWaves), h, ab[0]);
      __builtin_amdgcn_sched_barrier(0);
      if (mt + kMtWaves < n_mt) {
        mt_mma(ab[1], fb, c0, c1);
        emit(mt + kMtWaves, c0, c1);
      }
    }
  }
}

}  // namespace sparda

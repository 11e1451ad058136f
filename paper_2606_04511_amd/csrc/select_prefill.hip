// select_prefill.hip -- fused Forecast scoring and exact top-k for multi-row (chunked prefill)
// selection (paper Sec. 4.1, Eq. 4, with the attended-set union of Eq. 1; per query row as in
// Alg. 1).
//
// One 512-thread workgroup per 64-row tile of one (batch, group); the tile's rows share the
// candidate range [n_init, n_init + C), C <= 512, and each row takes its own top-k.
//   1. F rows of the tile are staged in LDS (272-byte row pitch: conflict-free 16-byte reads).
//   2. S = F K~^T on v_mfma_f32_16x16x32_bf16 (A = F, 4 M-tiles; B = K~ rows straight from L2,
//      one 16-candidate N-tile per wavefront at a time); the fp32 score tile stays in LDS.
//   3. Selection: 8 lanes per row, each lane holds the order-preserving keys of candidates
//      8 j + lane in registers.  The exact n-th largest key is found by counting passes
//      (compare + add per candidate): a normal-model first guess from the row's mean and
//      variance, regula-falsi steps on the bracketing counts, and a key-space bisection step
//      every third pass, until exactly n keys are >= the threshold or the bracket closes on one
//      key value (a true tie, resolved by the lower block index).
//   4. Ordered emission: per-candidate flag bytes in LDS become one 64-bit mask of candidates
//      [64 s, 64 s + 64) per lane; one 8-lane prefix sum places every chosen index.
// Workgroups are ordered so that consecutive ones (which the dispatcher spreads over the 8 XCDs)
// take different groups: with 8 groups each XCD's L2 holds a single group's K~.  Tiles with the
// most candidates go first.
#include <math.h>

#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

constexpr int kPreThreads = 512;
constexpr int kPreRows = kSelTileRows;             // 64 rows per tile
constexpr int kPreLd = kSelTileMaxCand + 4;        // floats per LDS score row
constexpr int kPreFLd = kHeadDim + 8;              // bf16 per staged F row (272 B)
constexpr int kPreVals = kSelTileMaxCand / 8;      // keys per lane (8 lanes per row)

// Forced blocks, local window and padding of one row, by its 8 lanes.
__device__ __forceinline__ void emit_forced8(int16_t* out, const RowGeom& g, int k_total, int sub) {
  for (int i = sub; i < g.init_hi; i += 8) out[i] = (int16_t)i;
  const int n_loc = g.blk - g.local_lo + 1;
  for (int i = sub; i < n_loc; i += 8) out[g.init_hi + g.n_take + i] = (int16_t)(g.local_lo + i);
  for (int i = g.n_forced + g.n_take + sub; i < k_total; i += 8) out[i] = (int16_t)-1;
}

// z with P(Z > z) = p for a standard normal Z (rational approximation of Abramowitz and Stegun
// 26.2.23, |error| < 4.5e-4).  Only used as a first guess; the search is exact regardless.
__device__ __forceinline__ float upper_normal_quantile(float p) {
  p = fminf(fmaxf(p, 1e-7f), 1.f - 1e-7f);
  const bool upper = p <= 0.5f;
  const float q = upper ? p : 1.f - p;
  const float t = sqrtf(-2.f * __logf(q));
  const float z = t - (2.515517f + t * (0.802853f + t * 0.010328f)) /
                          (1.f + t * (1.432788f + t * (0.189269f + t * 0.001308f)));
  return upper ? z : -z;
}

// Four flag bytes (one per candidate) -> four consecutive bits of the bytes whose bit `b` is set.
__device__ __forceinline__ uint32_t flag_bits(uint32_t w, int b) {
  const uint32_t x = (w >> b) & 0x01010101u;
  return ((x * 0x00204081u) >> 21) & 0xfu;
}

__global__ __launch_bounds__(kPreThreads) void prefill_select_kernel(SelectArgs a, int n_tiles, int n_groups) {
  __shared__ __align__(16) float sc[kPreRows * kPreLd];
  __shared__ __align__(16) uint16_t fst[kPreRows * kPreFLd];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bm = blockIdx.x % n_groups;
  const int tile = n_tiles - 1 - (int)(blockIdx.x / n_groups);
  const int r0 = tile * kPreRows;
  const int nrows = min(kPreRows, a.n_q - r0);
  const RowGeom gl = row_geom(a.q_pos0 + r0 + nrows - 1, a.n_init, a.n_local, a.k_total);
  const int C = gl.n_cand;              // the tile's candidate count (its last row has the most)
  const bool need = gl.n_take < gl.n_cand;  // if the last row takes every candidate, all rows do

  if (need) {
    {  // stage the tile's F rows: thread -> (row tid/8, 32-byte part tid%8)
      const int rr = tid >> 3, part = tid & 7;
      uint4 w0 = make_uint4(0u, 0u, 0u, 0u), w1 = w0;
      if (rr < nrows) {
        const uint16_t* src = a.f + (bm * a.n_q + r0 + rr) * kHeadDim + part * 16;
        w0 = ld16(src);
        w1 = ld16(src + 8);
      }
      uint4* dst = reinterpret_cast<uint4*>(fst + rr * kPreFLd + part * 16);
      dst[0] = w0;
      dst[1] = w1;
    }
    __syncthreads();
    const int lr = lane & 15, kq = 8 * (lane >> 4);
    bf16x8 fa[4][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        fa[mt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(fst + (mt * 16 + lr) * kPreFLd + 32 * ks + kq));
    const int n_nt = (C + 15) >> 4;
    const uint16_t* kcb = a.kc + (bm * a.nc_cap + a.n_init) * kHeadDim + kq;
    for (int nt = wave; nt < n_nt; nt += kPreThreads / 64) {
      const int cand = nt * 16 + lr;
      bf16x8 kb[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        kb[ks] = as_bf16x8(cand < C ? ld16(kcb + (int64_t)cand * kHeadDim + 32 * ks) : make_uint4(0u, 0u, 0u, 0u));
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) acc = mfma16x16x32(fa[mt][ks], kb[ks], acc);
        float* dst = sc + (mt * 16 + 4 * (lane >> 4)) * kPreLd + nt * 16 + lr;
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[i * kPreLd] = acc[i];
      }
    }
  }
  __syncthreads();

  // ---- per-row selection: 8 lanes per row; the 32 lanes of a half-wave hold rows two apart so
  // that their LDS reads fall in distinct banks.
  const int sub = lane & 7;
  const int rr = 8 * wave + ((lane >> 5) & 1) + 2 * ((lane >> 3) & 3);
  const bool row_ok = rr < nrows;
  const int64_t row = bm * a.n_q + r0 + rr;
  const RowGeom g = row_geom(a.q_pos0 + r0 + rr, a.n_init, a.n_local, a.k_total);
  int16_t* out = a.sel + row * a.k_total;
  if (row_ok) {
    emit_forced8(out, g, a.k_total, sub);
    if (sub == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
    if (g.n_take >= g.n_cand)
      for (int i = sub; i < g.n_cand; i += 8) out[g.init_hi + i] = (int16_t)(g.cand_lo + i);
  }
  if (!need) return;
  const int n = g.n_take, Cr = g.n_cand;
  const bool search = row_ok && n > 0 && n < Cr;
  const int V = (C + 7) >> 3;  // tile-uniform key slots in use per lane

  uint32_t key[kPreVals];
  float s1 = 0.f, s2 = 0.f;
  const float* srow = sc + rr * kPreLd;
#pragma unroll
  for (int j = 0; j < kPreVals; ++j) key[j] = 0u;  // below every finite score's key
#pragma unroll
  for (int jb = 0; jb < kPreVals; jb += 8) {
    if (jb < V) {
#pragma unroll
      for (int j = jb; j < jb + 8; ++j) {
        const int c = 8 * j + sub;
        const bool valid = search && c < Cr;
        const float v = valid ? srow[c] : 0.f;
        s1 += v;
        s2 = fmaf(v, v, s2);
        key[j] = valid ? score_key(v) : 0u;
      }
    }
  }
  s1 = group8_sum(s1);
  s2 = group8_sum(s2);
  const float inv = 1.f / (float)(Cr > 0 ? Cr : 1);
  const float mu = s1 * inv;
  const float sigma = sqrtf(fmaxf(s2 * inv - mu * mu, 1e-20f));
  const float z0 = upper_normal_quantile(((float)n - 0.5f) * inv);

  // Bracket [lo, hi) in key space with count(key >= lo) = c_lo >= n > c_hi = count(key >= hi).
  uint32_t lo = 1u, hi = 0xffffffffu;
  int c_lo = Cr, c_hi = 0;
  float vlo = 0.f, vhi = 0.f;
  bool done = !search;
  for (int it = 0; it < 100; ++it) {
    if (__ballot(!done) == 0ull) break;
    uint32_t t = lo + ((hi - lo) >> 1);
    if (!done) {
      const bool lo_b = lo != 1u, hi_b = hi != 0xffffffffu;
      bool model = true;
      float tv = 0.f;
      if (it == 0) {
        tv = mu + sigma * z0;
      } else if (lo_b && hi_b) {
        if (it % 3 == 2)
          model = false;
        else
          tv = vlo + (vhi - vlo) * (((float)(c_lo - n) + 0.5f) / (float)(c_lo - c_hi));
      } else if (it >= 4) {
        model = false;
      } else if (lo_b) {
        const float z = (vlo - mu) / sigma;
        const float dens = (float)Cr * 0.39894228f * __expf(-0.5f * z * z) / sigma;
        tv = vlo + 1.5f * ((float)(c_lo - n) + 0.5f) / fmaxf(dens, 1e-30f);
      } else {
        const float z = (vhi - mu) / sigma;
        const float dens = (float)Cr * 0.39894228f * __expf(-0.5f * z * z) / sigma;
        tv = vhi - 1.5f * ((float)(n - c_hi) + 0.5f) / fmaxf(dens, 1e-30f);
      }
      if (model && isfinite(tv)) t = score_key(tv);
      if (t <= lo) t = lo + 1u;
      if (t >= hi) t = hi - 1u;
    }
    int c = 0;
#pragma unroll
    for (int jb = 0; jb < kPreVals; jb += 8) {
      if (jb < V) {
#pragma unroll
        for (int j = jb; j < jb + 8; ++j) c += key[j] >= t ? 1 : 0;
      }
    }
    c = group8_sum(c);
    if (!done) {
      if (c >= n) {
        lo = t;
        c_lo = c;
        vlo = key_value(t);
      } else {
        hi = t;
        c_hi = c;
        vhi = key_value(t);
      }
      done = (c_lo == n) || (hi - lo <= 1u);
    }
  }

  // ---- ordered emission.  Normal case: the chosen keys are those >= lo (exactly n).  Tie case
  // (the bracket closed on one key value shared by more than the remaining slots): keys > lo,
  // plus the lowest-index n - c_hi of the keys == lo.
  const bool tie_mode = search && c_lo != n;
  uint8_t* flags = reinterpret_cast<uint8_t*>(sc + rr * kPreLd);  // reuses this row's scores
  wave_lds_sync();
  if (search) {
#pragma unroll
    for (int jb = 0; jb < kPreVals; jb += 8) {
      if (jb < V) {
#pragma unroll
        for (int j = jb; j < jb + 8; ++j) {
          const int c = 8 * j + sub;
          if (c < Cr) {
            const uint32_t k = key[j];
            flags[c] = tie_mode ? (uint8_t)(k > lo ? 1 : (k == lo ? 2 : 0)) : (uint8_t)(k >= lo ? 1 : 0);
          }
        }
      }
    }
  }
  wave_lds_sync();
  const int base_c = 64 * sub;
  uint64_t ch = 0ull, tm = 0ull;
  if (search && base_c < Cr) {
    const uint4* fp = reinterpret_cast<const uint4*>(flags + base_c);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 w = fp[q];
      const uint32_t cw = flag_bits(w.x, 0) | (flag_bits(w.y, 0) << 4) | (flag_bits(w.z, 0) << 8) |
                          (flag_bits(w.w, 0) << 12);
      ch |= (uint64_t)cw << (16 * q);
      if (tie_mode) {
        const uint32_t tw = flag_bits(w.x, 1) | (flag_bits(w.y, 1) << 4) | (flag_bits(w.z, 1) << 8) |
                            (flag_bits(w.w, 1) << 12);
        tm |= (uint64_t)tw << (16 * q);
      }
    }
    const int nvalid = Cr - base_c;
    if (nvalid < 64) {
      const uint64_t m = (1ull << nvalid) - 1ull;
      ch &= m;
      tm &= m;
    }
  }
  {  // ties: the first n - c_hi in index order
    const int tcnt = __popcll(tm);
    const int tb = group8_excl_scan(tcnt, sub);
    if (tie_mode) {
      int take = min(max(n - c_hi - tb, 0), tcnt);
      while (take-- > 0) {
        const uint64_t low = tm & (~tm + 1ull);
        ch |= low;
        tm ^= low;
      }
    }
  }
  const int cb = group8_excl_scan(__popcll(ch), sub);
  if (search) {
    int16_t* dst = out + g.init_hi + cb;
    uint64_t m = ch;
    int k = 0;
    while (m) {
      const int b = __builtin_ctzll(m);
      if (cb + k < n) dst[k] = (int16_t)(g.cand_lo + base_c + b);  // never past the row's slots
      ++k;
      m &= m - 1ull;
    }
  }
}

hipError_t launch_prefill_select(const SelectArgs& a, hipStream_t stream) {
  const int n_tiles = (a.n_q + kPreRows - 1) / kPreRows;
  const int n_groups = a.batch * a.n_kv_heads;
  hipLaunchKernelGGL(prefill_select_kernel, dim3((unsigned)((int64_t)n_groups * n_tiles)), dim3(kPreThreads), 0,
                     stream, a, n_tiles, n_groups);
  return hipGetLastError();
}

}  // namespace sparda

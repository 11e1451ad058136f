// select_prefill.hip -- fused Forecast scoring and exact top-k for multi-row (chunked prefill)
// selection (paper Sec. 4.1, Eq. 4, with the attended-set union of Eq. 1; per query row as in
// Alg. 1).
//
// One 512-thread workgroup per 32-row tile of one (batch, group); the tile's rows share the
// candidate range [n_init, n_init + C), C <= 512, and each row takes its own top-k.  A tile's
// LDS (72 KB) lets two workgroups share a CU, so one tile's loads and MFMA overlap another
// tile's selection.
//   1. F rows of the tile are staged in LDS (288-byte row pitch: conflict-free 16-byte reads).
//   2. S = F K~^T on v_mfma_f32_16x16x32_bf16 (A = F, 2 M-tiles; B = K~ rows straight from L2,
//      one 16-candidate N-tile per wavefront at a time).  The fp32 score tile stays in LDS; each
//      row is split into 16 ranges of V candidates (V a multiple of 4) laid out with a stride R
//      whose quarter is odd, so that the 16 lanes that later read their ranges with 16-byte loads
//      hit disjoint bank groups.  The staged F tile occupies the tail of the score buffer until
//      every wavefront holds its F fragments.
//   3. Selection, 16 lanes (one DPP row) per query row, 4 rows per wavefront, 8 wavefronts:
//      lane s holds the order-preserving keys of candidates [s V, s V + V) in registers
//      (candidates past the tile's last one hold -inf).  The exact n-th largest key is found by
//      passes over the keys, each a compare + add per key:
//        - a first pass counts at three thresholds around a normal-model guess (mean and
//          variance of a 64-score sample of the row), which usually brackets the n-th key;
//        - regula-falsi steps on the bracketing counts (a key-space bisection step every sixth
//          pass guarantees termination) until exactly n keys are >= the threshold;
//        - a row that misses exactly one key above its bracket is finished by one max pass
//          (the largest key below the bracket is the n-th); max passes wait until no row of the
//          wavefront still counts, so the two pass kinds never run in the same iteration.
//      If the bracket closes on a key value shared by more than the open slots, the ties are
//      taken by lower block index.
//   4. Emission: each lane turns its chosen keys into a 32-bit mask in candidate order; one
//      16-lane prefix sum over the mask popcounts places every chosen index.
// Workgroups are ordered so that consecutive ones (which the dispatcher spreads over the 8 XCDs)
// take different groups: with 8 groups each XCD's L2 holds a single group's K~.  Tiles with the
// most candidates go first.
#include <math.h>

#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

constexpr int kPreThreads = 512;
constexpr int kPreWaves = kPreThreads / 64;
constexpr int kPreRows = 32;                    // rows per tile
constexpr int kPreMt = kPreRows / 16;           // MFMA M-tiles per tile
constexpr int kPreVals = kSelTileMaxCand / 16;  // key slots per lane (16 lanes per row)
constexpr int kPreLd = 16 * (kPreVals + 4);     // floats per LDS score row (16 strided ranges)
constexpr int kPreFLd = kHeadDim + 16;          // bf16 per staged F row (288 B)
constexpr int kPreFFloats = kPreRows * kPreFLd / 2;  // staged F tile, in floats
// LDS serves each half wavefront on its own from 128 four-byte banks.  A row pitch of 64 (mod 128)
// banks puts the two rows a half wavefront touches (key loads: rows rr, rr + 1; MFMA stores: rows
// 4 i + q, q = 0, 1, after the F row permutation below) on disjoint banks, and a range stride R
// with R / 4 odd spreads the 16 ranges of a row over distinct 16-byte bank groups.
static_assert(kSelTileRows % kPreRows == 0, "tiles stay inside the rows a 64-row block spans");
static_assert(kPreLd == 576 && kPreLd % 128 == 64, "bank analysis assumes a row pitch of 576 floats");

// Forced blocks, local window and padding of one row, by its 16 lanes.
__device__ __forceinline__ void emit_forced16(int16_t* out, const RowGeom& g, int k_total, int sub) {
  for (int i = sub; i < g.init_hi; i += 16) out[i] = (int16_t)i;
  const int n_loc = g.blk - g.local_lo + 1;
  for (int i = sub; i < n_loc; i += 16) out[g.init_hi + g.n_take + i] = (int16_t)(g.local_lo + i);
  for (int i = g.n_forced + g.n_take + sub; i < k_total; i += 16) out[i] = (int16_t)-1;
}

// z with P(Z > z) = p for a standard normal Z (rational approximation of Abramowitz and Stegun
// 26.2.23, |error| < 4.5e-4).  Only a first guess; the search is exact regardless.
__device__ __forceinline__ float upper_normal_quantile(float p) {
  p = fminf(fmaxf(p, 1e-7f), 1.f - 1e-7f);
  const bool upper = p <= 0.5f;
  const float q = upper ? p : 1.f - p;
  const float t = sqrtf(-2.f * __logf(q));
  const float z = t - (2.515517f + t * (0.802853f + t * 0.010328f)) /
                          (1.f + t * (1.432788f + t * (0.189269f + t * 0.001308f)));
  return upper ? z : -z;
}

__device__ __forceinline__ uint32_t key_of_value(float v) {
  // score_key without the -0 branch: v + 0 turns -0 into +0 in round-to-nearest.
  const uint32_t u = __float_as_uint(v + 0.0f);
  return u ^ (uint32_t)(((int32_t)u >> 31) | (int32_t)0x80000000);
}

__global__ __launch_bounds__(kPreThreads) void prefill_select_kernel(SelectArgs a, int n_tiles, int n_groups) {
  __shared__ __align__(16) float sc[kPreRows * kPreLd];
  uint16_t* fst = reinterpret_cast<uint16_t*>(sc + kPreRows * kPreLd - kPreFFloats);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bm = blockIdx.x % n_groups;
  const int tile = n_tiles - 1 - (int)(blockIdx.x / n_groups);
  const int r0 = tile * kPreRows;
  const int nrows = min(kPreRows, a.n_q - r0);
  const RowGeom gl = row_geom(a.q_pos0 + r0 + nrows - 1, a.n_init, a.n_local, a.k_total);
  const int C = gl.n_cand;                  // the tile's candidate count (its last row has the most)
  const bool need = gl.n_take < gl.n_cand;  // if the last row takes every candidate, all rows do
  const int V = max((C + 63) >> 6, 1) * 4;     // candidates per lane range, a multiple of 4
  const int R = V + ((V & 4) ? 8 : 4);          // range stride: R / 4 is odd

  if (need) {
    // This wavefront's N-tiles are nt = wave + 8 i (V <= 32 N-tiles, so i < 4).  Their K~ rows
    // are requested first so that the L2 latency overlaps the F staging and its barriers.
    constexpr int kNtPerWave = kPreVals / kPreWaves;  // 4
    const int lr = lane & 15, kq = 8 * (lane >> 4);
    const uint16_t* kcb = a.kc + (bm * a.nc_cap + a.n_init) * kHeadDim + kq;
    uint4 kw[kNtPerWave][4];
#pragma unroll
    for (int i = 0; i < kNtPerWave; ++i) {
      const int cand = (wave + kPreWaves * i) * 16 + lr;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        kw[i][ks] = cand < C ? ld16(kcb + (int64_t)cand * kHeadDim + 32 * ks) : make_uint4(0u, 0u, 0u, 0u);
    }
    {  // stage the tile's F rows: thread -> (row tid/16, 16-byte part tid%16)
      const int rr = tid >> 4, part = tid & 15;
      uint4 w0 = make_uint4(0u, 0u, 0u, 0u);
      if (rr < nrows) w0 = ld16(a.f + (bm * a.n_q + r0 + rr) * kHeadDim + part * 8);
      *reinterpret_cast<uint4*>(fst + rr * kPreFLd + part * 8) = w0;
    }
    static_assert(kPreThreads / 16 == kPreRows, "one thread per 16 bytes of the F tile");
    static_assert(kNtPerWave * kPreWaves * 16 == kSelTileMaxCand, "N-tiles cover every candidate slot");
    __syncthreads();
    // A-operand row lr of an M-tile is tile row 4 (lr % 4) + lr / 4, so that accumulator element
    // i of lane (n, q) holds the score of tile row 4 i + q.
    bf16x8 fa[kPreMt][4];
    const int fr = 4 * (lr & 3) + (lr >> 2);
#pragma unroll
    for (int mt = 0; mt < kPreMt; ++mt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        fa[mt][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(fst + (mt * 16 + fr) * kPreFLd + 32 * ks + kq));
    __syncthreads();  // the staged F tile is overwritten by scores below
    // V N-tiles cover all 16 V key slots; candidates past C get -inf (no key counts them).
#pragma unroll
    for (int i = 0; i < kNtPerWave; ++i) {
      const int nt = wave + kPreWaves * i;
      if (nt < V) {
        const int cand = nt * 16 + lr;
        const int col = (cand / V) * R + cand % V;
#pragma unroll
        for (int mt = 0; mt < kPreMt; ++mt) {
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
          if (nt * 16 < C) {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) acc = mfma16x16x32(fa[mt][ks], as_bf16x8(kw[i][ks]), acc);
          }
          float* dst = sc + (mt * 16 + (lane >> 4)) * kPreLd + col;
#pragma unroll
          for (int q = 0; q < 4; ++q) dst[4 * q * kPreLd] = cand < C ? acc[q] : -INFINITY;
        }
      }
    }
  }
  __syncthreads();

  // ---- per-row selection: 16 lanes per row, 4 rows per wavefront.
  const int sub = lane & 15;
  const int rr = 4 * wave + (lane >> 4);
  const bool row_ok = rr < nrows;
  const int64_t row = bm * a.n_q + r0 + rr;
  const RowGeom g = row_geom(a.q_pos0 + r0 + rr, a.n_init, a.n_local, a.k_total);
  int16_t* out = a.sel + row * a.k_total;
  if (row_ok) {
    emit_forced16(out, g, a.k_total, sub);
    if (sub == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
    if (g.n_take >= g.n_cand)
      for (int i = sub; i < g.n_cand; i += 16) out[g.init_hi + i] = (int16_t)(g.cand_lo + i);
  }
  if (!need) return;
  const int n = g.n_take, Cr = g.n_cand;
  const bool search = row_ok && n > 0 && n < Cr;
  const int cbase = sub * V;  // this lane's candidates [cbase, cbase + V), at sc[row][sub R ..]

  // Scores of all 16 V slots, compared as floats against thresholds that are kept as keys: the
  // float key_value(t) admits exactly the scores whose key is >= t (-0 and +0 share a key, and no
  // score has the key of -0).  Rows of an unaligned chunk may have fewer candidates than the tile
  // (Cr < C): their extra slots hold -inf, which no threshold admits.
  constexpr uint32_t kKeyNegInf = 0x007fffffu;  // key of -inf: below every threshold used
  float val[kPreVals];
  const float* srow = sc + rr * kPreLd + sub * R;
#pragma unroll
  for (int j = 0; j < kPreVals; ++j) val[j] = -INFINITY;
  const bool short_row = search && Cr < C;
#pragma unroll
  for (int jb = 0; jb < kPreVals; jb += 4) {
    if (jb < V) {
      const float4 v = *reinterpret_cast<const float4*>(srow + jb);
      val[jb] = v.x;
      val[jb + 1] = v.y;
      val[jb + 2] = v.z;
      val[jb + 3] = v.w;
    }
  }
  if (__ballot(short_row) != 0ull) {
#pragma unroll
    for (int j = 0; j < kPreVals; ++j)
      if (short_row && cbase + j >= Cr) val[j] = -INFINITY;
  }
  // Mean and variance from the first four slots of each lane (a 64-score sample of the row).
  float s1 = 0.f, s2 = 0.f, ns = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bool ok = j < V && cbase + j < Cr;
    const float v = ok ? val[j] : 0.f;
    s1 += v;
    s2 = fmaf(v, v, s2);
    ns += ok ? 1.f : 0.f;
  }
  s1 = row16_sum(s1);
  s2 = row16_sum(s2);
  ns = fmaxf(row16_sum(ns), 1.f);
  const float inv_s = __builtin_amdgcn_rcpf(ns);
  const float mu = s1 * inv_s;
  const float sigma = sqrtf(fmaxf(s2 * inv_s - mu * mu, 1e-20f));
  const float inv = __builtin_amdgcn_rcpf((float)(Cr > 0 ? Cr : 1));
  const float z0 = upper_normal_quantile(((float)n - 0.5f) * inv);
  // Counts per unit of score near the guess (normal model) and the first pass's spacing: about
  // 1.5 sqrt(n) + 2 counts, the typical binomial error of the model guess.
  const float dens = fmaxf((float)Cr * 0.39894228f * __expf(-0.5f * z0 * z0) / sigma, 1e-30f);
  const float step = (1.5f * sqrtf((float)n) + 2.f) * __builtin_amdgcn_rcpf(dens);
  const float t_mid = mu + sigma * z0;

  // Bracket [lo, hi) in key space: count(key >= lo) = c_lo >= n > c_hi = count(key >= hi).
  // lo starts just above -inf (every real score counts), hi just above +inf (none does).
  uint32_t lo = kKeyNegInf + 1u, hi = 0xff800001u;
  int c_lo = Cr, c_hi = 0;
  float vlo = 0.f, vhi = 0.f;
  bool lo_b = false, hi_b = false;  // vlo / vhi hold the score value of lo / hi
  bool done = !search;
  {  // first pass: three thresholds around the guess
    const float va = t_mid - step, vb = t_mid, vc = t_mid + step;
    const uint32_t ta = key_of_value(va), tb = key_of_value(vb), tc = key_of_value(vc);
    // compare against the exact values of the keys (non-finite guesses never enter the bracket)
    const float fa = key_value(ta), fb = key_value(tb), fc = key_value(tc);
    int ca = 0, cb = 0, cc = 0;
#pragma unroll
    for (int jb = 0; jb < kPreVals; jb += 4) {
      if (jb < V) {
#pragma unroll
        for (int j = jb; j < jb + 4; ++j) {
          ca += val[j] >= fa ? 1 : 0;
          cb += val[j] >= fb ? 1 : 0;
          cc += val[j] >= fc ? 1 : 0;
        }
      }
    }
    ca = row16_sum(ca);
    cb = row16_sum(cb);
    cc = row16_sum(cc);
    if (!done) {
      const uint32_t tt[3] = {ta, tb, tc};
      const int cs[3] = {ca, cb, cc};
      const float vs[3] = {va, vb, vc};
#pragma unroll
      for (int i = 0; i < 3; ++i) {
        if (tt[i] > lo && tt[i] < hi) {
          if (cs[i] >= n) { lo = tt[i]; c_lo = cs[i]; vlo = vs[i]; lo_b = true; }
          else { hi = tt[i]; c_hi = cs[i]; vhi = vs[i]; hi_b = true; }
        }
      }
      done = (c_lo == n) || (hi - lo <= 1u);
    }
  }
  float grow = 2.f * step;
  for (int it = 0; it < 100; ++it) {
    const bool want_max = !done && hi_b && (n - c_hi == 1);
    const bool want_cnt = !done && !want_max;
    if (__ballot(want_cnt) != 0ull) {
      uint32_t t = lo + ((hi - lo) >> 1);  // key-space bisection unless a model step is taken
      float tv = 0.f;
      bool have_v = false;
      if (want_cnt) {
        if (lo_b && hi_b) {
          if (it % 6 != 5) {
            tv = vlo + (vhi - vlo) * (((float)(c_lo - n) + 0.5f) * __builtin_amdgcn_rcpf((float)(c_lo - c_hi)));
            have_v = true;
          }
        } else if (it < 6) {  // one side still open: step outwards, doubling
          tv = lo_b ? vlo + grow : vhi - grow;
          grow *= 2.f;
          have_v = true;
        }
        if (have_v) {
          if (isfinite(tv))
            t = key_of_value(tv);
          else
            have_v = false;
        }
        if (t <= lo) { t = lo + 1u; have_v = false; }
        if (t >= hi) { t = hi - 1u; have_v = false; }
      }
      const float ft = key_value(t);
      int c = 0;
#pragma unroll
      for (int jb = 0; jb < kPreVals; jb += 4) {
        if (jb < V) {
#pragma unroll
          for (int j = jb; j < jb + 4; ++j) c += val[j] >= ft ? 1 : 0;
        }
      }
      c = row16_sum(c);
      if (want_cnt) {
        const float vt = have_v ? tv : key_value(t);
        if (c >= n) { lo = t; c_lo = c; vlo = vt; lo_b = true; }
        else { hi = t; c_hi = c; vhi = vt; hi_b = true; }
        done = (c_lo == n) || (hi - lo <= 1u);
      }
    } else if (__ballot(want_max) != 0ull) {
      // n - 1 keys lie at or above hi: the n-th largest is the largest key below hi.  No key
      // lies strictly between it and hi, so count(key >= m + 1) is still c_hi.
      const float fhi = key_value(hi);
      float mv = -INFINITY;
#pragma unroll
      for (int jb = 0; jb < kPreVals; jb += 4) {
        if (jb < V) {
#pragma unroll
          for (int j = jb; j < jb + 4; ++j) mv = val[j] < fhi ? fmaxf(mv, val[j]) : mv;
        }
      }
      uint32_t m = row16_max(mv == -INFINITY ? 0u : key_of_value(mv));
      if (want_max) {
        lo = m;
        hi = m + 1u;
        c_lo = -1;  // unknown: the emission takes the n - c_hi lowest-index keys equal to lo
        done = true;
      }
    } else {
      break;
    }
  }

  // ---- emission.  Normal case: the chosen keys are those >= lo (exactly n).  Tie case (the
  // bracket closed on one key value shared by more than the remaining slots): keys > lo, plus
  // the lowest-index n - c_hi of the keys == lo.
  const bool tie_mode = search && c_lo != n;
  const uint32_t thr = tie_mode ? lo + 1u : lo;
  const float fthr = key_value(thr), flo = key_value(lo);
  uint32_t ch = 0u, tm = 0u;
#pragma unroll
  for (int jb = 0; jb < kPreVals; jb += 4) {
    if (jb < V) {
#pragma unroll
      for (int j = jb; j < jb + 4; ++j)
        if (val[j] >= fthr) ch |= 1u << j;
    }
  }
  if (__ballot(tie_mode) != 0ull) {
#pragma unroll
    for (int jb = 0; jb < kPreVals; jb += 4) {
      if (jb < V) {
#pragma unroll
        for (int j = jb; j < jb + 4; ++j)
          if (val[j] == flo) tm |= 1u << j;
      }
    }
  }
  if (!search) ch = 0u;
  if (!tie_mode) tm = 0u;
  {  // ties: the first n - c_hi in index order
    const int tcnt = __popc(tm);
    const int tb = row16_excl_scan(tcnt, sub);
    if (tie_mode) {
      int take = min(max(n - c_hi - tb, 0), tcnt);
      while (take-- > 0) {
        const uint32_t low = tm & (~tm + 1u);
        ch |= low;
        tm ^= low;
      }
    }
  }
  const int cb = row16_excl_scan(__popc(ch), sub);
  if (search) {
    int16_t* dst = out + g.init_hi + cb;
    const int cand0 = g.cand_lo + cbase;
    uint32_t m = ch;
    int k = 0;
    while (m) {
      const int b = __builtin_ctz(m);
      if (cb + k < n) dst[k] = (int16_t)(cand0 + b);  // never past the row's slots
      ++k;
      m &= m - 1u;
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

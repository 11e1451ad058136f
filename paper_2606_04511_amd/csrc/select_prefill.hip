// select_prefill.hip -- fused Forecast scoring and exact top-k for multi-row (chunked prefill)
// selection (paper Sec. 4.1, Eq. 4, with the attended-set union of Eq. 1; per query row as in
// Alg. 1).
//
// Work unit: a slice of 16 consecutive query rows of one (batch, group), owned by one wavefront.
// A slice's rows share their candidate range [n_init, n_init + C) up to the rows of a block
// boundary inside the slice (those have one candidate less, masked below); each row takes its own
// top-k.
//
// Workgroups are persistent units of 8 wavefronts, several per (batch, group).  Unit u of U takes
// slice u of every even sweep of U consecutive slices and slice U - 1 - u of every odd one, which
// evens out the work (a slice's cost grows with its position).  The unit stages the K~ rows of
// its largest candidate range in LDS once (272-byte row pitch), then its wavefronts take its
// slices from an LDS counter, most candidates first.
//
// Per slice:
//   1. S^T = K~ F^T on v_mfma_f32_16x16x32_bf16: B = the slice's 16 F rows (straight from HBM,
//      prefetched one slice ahead), A = 16 staged K~ rows per M-tile.  A row m of M-tile t is
//      candidate (m / 4) Q + 4 t + m % 4 with Q = 4 ceil(C / 16), so accumulator element i of lane
//      (n, j) -- query row n, lane group j -- holds candidate j Q + 4 t + i: each row's scores sit
//      in the accumulators of its 4 lanes, every lane holding one contiguous quarter [j Q, j Q + Q)
//      of the candidates.  Scores never leave the registers.
//   2. Exact n-th largest score per row by count passes over the 4 Q registers, each a compare +
//      add per score and a 4-lane sum (two permlane swaps):
//        - a first pass counts at three thresholds around a normal-model guess (mean and variance
//          of a 64-score sample of the row), which usually brackets the n-th score;
//        - regula-falsi steps on the bracketing counts (a key-space bisection step every sixth
//          pass guarantees termination) until exactly n scores are >= the threshold;
//        - a row that misses exactly one score above its bracket is finished by one max pass.
//      Thresholds are kept as order-preserving keys and compared as the floats they encode.  If
//      the bracket closes on a value shared by more scores than open slots, the ties are taken
//      by lower block index.
//   3. Emission: a lane's chosen scores become a bit mask in candidate order; a 4-lane exclusive
//      prefix of the popcounts gives each lane its first output slot, and the lane writes its
//      indices in ascending order.
//
// On the paper's (32, 16) key grid (Sec. 3: windows of 32 tokens at stride 16, max-pooled to
// blocks) step 1 scores windows instead (prefill_select_win_kernel): block b's score is the
// largest score among windows 4b - 1 .. 4b + 3 that are complete at the row's position.
// Window-tile u puts window 4 (n_init + (m / 4) Q + u) + m % 4 in A row m, so lane (n, j)
// receives windows 4b .. 4b + 3 of block b = n_init + j Q + u in its accumulators and pools them
// with the previous tile's last window (a tile u = -1 supplies it for u = 0).  The pooled score
// lands in the key slot the block grid uses for block b, and steps 2-3 run unchanged.  The
// window keys (four times as many) do not fit in LDS at once; they are staged in chunks shared by
// a workgroup's wavefronts, which score eight slices in lockstep (see that kernel).
#include <math.h>

#include <algorithm>

#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

constexpr int kPsThreads = 512;
constexpr int kPsWaves = kPsThreads / 64;
constexpr int kPsRows = 16;                     // rows per slice (one MFMA N-tile)
constexpr int kPsMaxMt = kSelTileMaxCand / 16;  // M-tiles per slice: up to 128 key slots per lane
constexpr int kPsPitch = kHeadDim + 8;          // bf16 per staged K~ row (272 B)
constexpr int kPsStageRows = kSelTileMaxCand + 8;  // staged K~ rows, the A read-ahead's 8 included
constexpr int kPsStageK = 64;                   // sets of at most this many entries go through LDS
constexpr int kPsOutPitch = kPsStageK + 8;      // int16 per staged set row: rows 144 B apart use
                                                // distinct banks; entries 64.. are emission dummies
constexpr int kPsMaxUnits = 256;                // units per (batch, group)

struct PrefillPlan {
  int32_t n_slices;  // slices per (batch, group)
  int32_t units;     // units per (batch, group)
};

// Sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (one query row); every one of them receives it.
__device__ __forceinline__ int row4_sum(int x) {
  const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  const int y = (int)p[0] + (int)p[1];
  const auto q = __builtin_amdgcn_permlane32_swap(y, y, false, false);
  return (int)q[0] + (int)q[1];
}
__device__ __forceinline__ float row4_sum(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
__device__ __forceinline__ uint32_t row4_max(uint32_t x) {
  const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  const uint32_t y = max((uint32_t)p[0], (uint32_t)p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(y, y, false, false);
  return max((uint32_t)q[0], (uint32_t)q[1]);
}
// Exclusive prefix over the row's lanes in lane-group order j = 0..3; *total gets the row sum.
__device__ __forceinline__ int row4_excl_scan(int x, int j, int* total) {
  const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);  // p[0]: even group, p[1]: odd
  const int pair = (int)p[0] + (int)p[1];
  const auto q = __builtin_amdgcn_permlane32_swap(pair, pair, false, false);  // q[0]: groups 0-1, q[1]: 2-3
  *total = (int)q[0] + (int)q[1];
  return ((j & 1) ? (int)p[0] : 0) + ((j & 2) ? (int)q[0] : 0);
}

__device__ __forceinline__ uint32_t key_of_value(float v) {
  // score_key without the -0 branch: v + 0 turns -0 into +0 in round-to-nearest.
  const uint32_t u = __float_as_uint(v + 0.0f);
  return u ^ (uint32_t)(((int32_t)u >> 31) | (int32_t)0x80000000);
}

// Runs f(score, slot) over the lane's key slots of the first ntg groups of 4 M-tiles (slot =
// 4 t + i); M-tiles past the slice's last one hold -inf.
template <class Fn>
__device__ __forceinline__ void for_slots(const float (&acc)[kPsMaxMt][4], int ntg, Fn&& f) {
#pragma unroll
  for (int tg = 0; tg < kPsMaxMt / 4; ++tg) {
    if (tg < ntg) {
#pragma unroll
      for (int t = 4 * tg; t < 4 * tg + 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) f(acc[t][i], 4 * t + i);
    }
  }
}

// Shifts the "below" flag of one score into m: m << 1 | [x < v], as the sign bit of x - v
// (v_alignbit takes the top bit of the difference).  x >= v exactly when x - v has a clear sign
// bit: scores are finite or -inf, -0 has been turned into +0, v is finite or +inf, and float32
// denormals are kept, so the difference of two different values is never zero.  No compare
// result passes through VCC.
__device__ __forceinline__ uint32_t shift_below(uint32_t m, float x, float v) {
  return __builtin_amdgcn_alignbit(m, __float_as_uint(x - v), 31);
}

// Runs f(word, m) over the lane's slot words (32 slots, the last one possibly 16): m holds the
// "below v" flags of the word's slots, first slot highest.
template <class Fn>
__device__ __forceinline__ void below_words(const float (&acc)[kPsMaxMt][4], int ntg, float v, Fn&& f) {
#pragma unroll
  for (int d = 0; d < kPsMaxMt / 8; ++d) {
    if (2 * d < ntg) {
      uint32_t m = 0u;
#pragma unroll
      for (int t = 8 * d; t < 8 * d + 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) m = shift_below(m, acc[t][i], v);
      if (2 * d + 1 < ntg) {
#pragma unroll
        for (int t = 8 * d + 4; t < 8 * d + 8; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) m = shift_below(m, acc[t][i], v);
      }
      f(d, m);
    }
  }
}

// Number of key slots >= v, summed over the row's four lanes (padding slots hold -inf).
__device__ __forceinline__ int count_ge(const float (&acc)[kPsMaxMt][4], int ntg, float v) {
  int lt = 0;
  below_words(acc, ntg, v, [&](int, uint32_t m) { lt += __popc(m); });
  return 64 * ntg - row4_sum(lt);
}

// Bit masks over the lane's key slots with bit e of m[d] standing for slot 32 d + e (first slot
// lowest): the slots with x >= v.
__device__ __forceinline__ void ge_masks(const float (&acc)[kPsMaxMt][4], int ntg, float v, uint32_t (&m)[4]) {
#pragma unroll
  for (int d = 0; d < 4; ++d) m[d] = 0u;
  below_words(acc, ntg, v, [&](int d, uint32_t w) {
    const bool full = 2 * d + 1 < ntg;  // 32 slots, else 16 in bits 0..15
    const uint32_t ge = full ? ~w : (~w & 0xffffu) << 16;
    m[d] = __builtin_bitreverse32(ge);
  });
}

// Same layout for the slots with x == v (compared as floats).
__device__ __forceinline__ void eq_masks(const float (&acc)[kPsMaxMt][4], int ntg, float v, uint32_t (&m)[4]) {
#pragma unroll
  for (int d = 0; d < 4; ++d) m[d] = 0u;
#pragma unroll
  for (int t = 0; t < kPsMaxMt; ++t) {
    if ((t >> 2) < ntg) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (acc[t][i] == v) m[t >> 3] |= 1u << ((4 * t + i) & 31);
    }
  }
}

// Writes, in ascending slot order, cand0 + slot for every set bit of m (slot = 32 d + bit) to
// dst[k], dst[k + 1], ... while k < k_end.  The loops run while any lane of the wavefront has a bit
// left (a uniform trip count); a lane with none left writes to *dummy.
__device__ __forceinline__ void emit_bits(const uint32_t (&m)[4], int nwords, int16_t* dst, int k, int k_end,
                                          int cand0, int16_t* dummy) {
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    if (d < nwords) {
      uint32_t w = m[d];
      while (__ballot(w != 0u) != 0ull) {
        const int e = __builtin_ctz(w | 0x80000000u);  // lowest set bit (31 when none: unused)
        const bool ok = w != 0u && k < k_end;
        int16_t* p = ok ? dst + k : dummy;
        *p = (int16_t)(cand0 + 32 * d + e);
        k += w != 0u ? 1 : 0;
        w &= w - 1u;
      }
    }
  }
}

// Copies the assembled sets of a slice's valid rows (LDS rows kPsOutPitch apart) to the selection
// output.
__device__ __forceinline__ void copy_out(const SelectArgs& a, int64_t bm, int s, const int16_t* ost, int lane) {
  const int nr = min(kPsRows, a.n_q - s * kPsRows);
  const int k = a.k_total;
  int16_t* dst = a.sel + (bm * a.n_q + (int64_t)s * kPsRows) * k;
  if (((reinterpret_cast<uintptr_t>(dst) | (uintptr_t)(2 * k)) & 15u) == 0) {
    const int per_row = k / 8;  // 16-byte chunks per row
    for (int i = lane; i < nr * per_row; i += 64) {
      const int r = i / per_row, c = i - r * per_row;
      *reinterpret_cast<uint4*>(dst + r * k + 8 * c) = *reinterpret_cast<const uint4*>(ost + r * kPsOutPitch + 8 * c);
    }
  } else {
    for (int i = lane; i < nr * k; i += 64) {
      const int r = i / k;
      dst[i] = ost[r * kPsOutPitch + (i - r * k)];
    }
  }
}

// Exact n-th largest score of each row of a slice and the ordered emission of its chosen
// candidates (steps 2 and 3 above) over the key slots a scoring step left in acc.  nmt: the
// slice's M-tiles (its first four are sampled), ntg = ceil(nmt / 4), Q = 4 nmt key slots per
// lane, v: this lane's valid slots, n / Cr: the row's budget and candidate count, search: the row
// takes a strict subset, g: the row's geometry, out: the row's selection (LDS row when kStaged),
// dummy: a padding slot of that LDS row (lanes with nothing left to write store there).
template <bool kStaged>
__device__ __forceinline__ void search_emit(float (&acc)[kPsMaxMt][4], int nmt, int ntg, int Q, int v, int n, int Cr,
                                            bool search, int lg, const RowGeom& g, int16_t* out, int16_t* dummy) {
  // ---- exact n-th largest per row
  // Mean and variance of a sample: the first 16 slots of each of the row's lanes.
  float s1 = 0.f, s2 = 0.f, ns = 0.f;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool ok = t < nmt && 4 * t + i < v;
      const float x = ok ? acc[t][i] : 0.f;
      s1 += x;
      s2 = fmaf(x, x, s2);
      ns += ok ? 1.f : 0.f;
    }
  }
  s1 = row4_sum(s1);
  s2 = row4_sum(s2);
  ns = fmaxf(row4_sum(ns), 1.f);
  const float inv_s = __builtin_amdgcn_rcpf(ns);
  const float mu = s1 * inv_s;
  const float sigma = __builtin_amdgcn_sqrtf(fmaxf(s2 * inv_s - mu * mu, 1e-20f));
  const float inv = __builtin_amdgcn_rcpf((float)(Cr > 0 ? Cr : 1));
  const float z0 = upper_normal_quantile(((float)n - 0.5f) * inv);
  // Counts per unit of score near the guess (normal model) and the first pass's spacing: about
  // 1.5 sqrt(n) + 2 counts, the typical binomial error of the model guess.
  const float dens = fmaxf((float)Cr * 0.39894228f * __expf(-0.5f * z0 * z0) / sigma, 1e-30f);
  const float step = (1.5f * __builtin_amdgcn_sqrtf((float)n) + 2.f) * __builtin_amdgcn_rcpf(dens);
  const float t_mid = mu + sigma * z0;

  // Bracket [lo, hi) in key space: count(key >= lo) = c_lo >= n > c_hi = count(key >= hi).
  // lo starts just above -inf (every real score counts), hi just above +inf (none does).
  constexpr uint32_t kKeyNegInf = 0x007fffffu;  // key of -inf: below every threshold used
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
#pragma unroll
    for (int tg = 0; tg < kPsMaxMt / 4; ++tg) {
      if (tg < ntg) {
#pragma unroll
        for (int t = 4 * tg; t < 4 * tg + 4; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[t][i] += 0.0f;  // -0 becomes +0 (shift_below relies on it)
      }
    }
    int la = 0, lb = 0, lc = 0;  // slots below each threshold
#pragma unroll
    for (int d = 0; d < kPsMaxMt / 8; ++d) {
      if (2 * d < ntg) {
        uint32_t ma = 0u, mb = 0u, mc = 0u;
#pragma unroll
        for (int t = 8 * d; t < 8 * d + 8; ++t) {
          if (t < 8 * d + 4 || 2 * d + 1 < ntg) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              ma = shift_below(ma, acc[t][i], fa);
              mb = shift_below(mb, acc[t][i], fb);
              mc = shift_below(mc, acc[t][i], fc);
            }
          }
        }
        la += __popc(ma);
        lb += __popc(mb);
        lc += __popc(mc);
      }
    }
    const int ca = 64 * ntg - row4_sum(la);
    const int cb = 64 * ntg - row4_sum(lb);
    const int cc = 64 * ntg - row4_sum(lc);
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
  for (int it = 0; it < 200; ++it) {  // every sixth step bisects the key range: done within 6 * 33
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
      const int c = count_ge(acc, ntg, key_value(t));
      if (want_cnt) {
        const float vt = have_v ? tv : key_value(t);
        if (c >= n) { lo = t; c_lo = c; vlo = vt; lo_b = true; }
        else { hi = t; c_hi = c; vhi = vt; hi_b = true; }
        done = (c_lo == n) || (hi - lo <= 1u);
      }
    } else if (__ballot(want_max) != 0ull) {
      // n - 1 scores lie at or above hi: the n-th largest is the largest score below hi.  No
      // score lies strictly between it and hi, so count(key >= m + 1) is still c_hi.
      const float fhi = key_value(hi);
      float mv = -INFINITY;
      for_slots(acc, ntg, [&](float x, int) { mv = x < fhi ? fmaxf(mv, x) : mv; });
      const uint32_t m = row4_max(mv == -INFINITY ? 0u : key_of_value(mv));
      if (want_max) {
        lo = m;
        hi = m + 1u;
        c_lo = -1;  // unknown: the emission takes the n - c_hi lowest-index scores equal to lo
        done = true;
      }
    } else {
      break;
    }
  }

  // ---- emission.  The chosen scores are those >= value(lo): exactly n of them unless several
  // scores share that value (the bracket closed on one key, or the max pass found a repeated
  // value).  Then (tie case) they are the scores > value(lo) -- c_hi of them, since hi = lo + 1
  // -- plus the lowest-index n - c_hi of the scores equal to value(lo).
  uint32_t ch[4];
  ge_masks(acc, ntg, key_value(lo), ch);
  int ccnt = 0;
#pragma unroll
  for (int d = 0; d < 4; ++d) ccnt += __popc(ch[d]);
  int ctot;
  int cb = row4_excl_scan(ccnt, lg, &ctot);
  const bool tie_mode = search && ctot != n;
  if (__ballot(tie_mode) != 0ull) {
    uint32_t gt[4], tm[4];
    ge_masks(acc, ntg, key_value(lo + 1u), gt);
    eq_masks(acc, ntg, key_value(lo), tm);
    int tcnt = 0;
#pragma unroll
    for (int d = 0; d < 4; ++d) tcnt += __popc(tm[d]);
    int ttot;
    const int tb = row4_excl_scan(tcnt, lg, &ttot);
    if (tie_mode) {
      int take = min(max(n - c_hi - tb, 0), tcnt);
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        ch[d] = gt[d];
        while (take > 0 && tm[d] != 0u) {
          const uint32_t low = tm[d] & (~tm[d] + 1u);
          ch[d] |= low;
          tm[d] ^= low;
          --take;
        }
      }
    }
    ccnt = 0;
#pragma unroll
    for (int d = 0; d < 4; ++d) ccnt += __popc(ch[d]);
    cb = row4_excl_scan(ccnt, lg, &ctot);
  }
  if (kStaged) {
    // every lane runs the wave-uniform loops; rows without a search write nothing
    emit_bits(ch, (Q + 31) >> 5, out + g.init_hi, cb, search ? n : 0, g.cand_lo + lg * Q, dummy);
  } else if (search) {
    int16_t* dst = out + g.init_hi;
    const int cand0 = g.cand_lo + lg * Q;
    int k = cb;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      uint32_t m = 32 * d < Q ? ch[d] : 0u;
      while (m) {
        const int e = __builtin_ctz(m);
        if (k < n) dst[k] = (int16_t)(cand0 + 32 * d + e);  // never past the row's slots
        ++k;
        m &= m - 1u;
      }
    }
  }
}

// The block grid (one key per block).  kStaged: every set is assembled in the wavefront's LDS rows
// (k_total <= kPsStageK) and written out with 16-byte stores; otherwise entries go straight to the
// output.
template <bool kStaged>
__global__ __launch_bounds__(kPsThreads) void prefill_select_kernel(SelectArgs a, PrefillPlan plan, int n_groups) {
  __shared__ __align__(16) uint16_t kst[kPsStageRows * kPsPitch];
  __shared__ __align__(16) int16_t ost_all[kStaged ? kPsWaves * kPsRows * kPsOutPitch : 8];
  __shared__ int next_sweep;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bm = blockIdx.x % n_groups;
  const int u = (int)(blockIdx.x / n_groups);
  // Sweeps of U consecutive slices: unit u takes slice u of every even sweep and slice U - 1 - u
  // of every odd one.  A slice's cost grows with its position, so this back-and-forth order gives
  // every unit about the same work without a cost model.
  const int ns = plan.n_slices, U = plan.units;
  if (u >= ns) return;  // uniform over the workgroup
  auto slice_of = [&](int i) { return i < 0 ? -1 : i * U + ((i & 1) ? U - 1 - u : u); };
  int i_top = (ns - 1) / U;             // the last sweep, partial unless U divides ns
  if (slice_of(i_top) >= ns) --i_top;   // then it may not reach this unit (the first sweep always does)
  const int s_last = slice_of(i_top);   // the unit's last slice

  // ---- stage the K~ rows of the unit's largest candidate range (its last row), zero-padded to
  // whole M-tiles and the read-ahead rows.  Rows that take every candidate are never scored, and
  // neither is a unit whose last row takes every candidate (earlier rows have at most as many
  // candidates and at least as large a budget).
  {
    const RowGeom gl = row_geom(a.q_pos0 + min(a.n_q, (s_last + 1) * kPsRows) - 1, a.n_init, a.n_local, a.k_total);
    const int c_stage = gl.n_take < gl.n_cand ? gl.n_cand : 0;
    const int c_fill = c_stage > 0 ? ((c_stage + 15) & ~15) + 8 : 0;
    const uint16_t* kcb = a.kc + (bm * a.nc_cap + a.n_init) * kHeadDim;
    for (int i = tid; i < c_fill * 16; i += kPsThreads) {
      const int c = i >> 4, part = i & 15;
      const uint4 w = c < c_stage ? ld16(kcb + (int64_t)c * kHeadDim + part * 8) : make_uint4(0u, 0u, 0u, 0u);
      *reinterpret_cast<uint4*>(kst + c * kPsPitch + part * 8) = w;
    }
  }
  if (tid == 0) next_sweep = i_top;
  __syncthreads();

  const int lr = lane & 15, lg = lane >> 4;
  int16_t* ost = ost_all + (kStaged ? wave * kPsRows * kPsOutPitch : 0);
  // Sweeps are taken from the last (most candidates first); -1 once none is left.
  auto grab = [&]() -> int {
    int i = 0;
    if (lane == 0) i = atomicSub(&next_sweep, 1);
    return slice_of(__builtin_amdgcn_readfirstlane(i));
  };
  auto load_f = [&](int s, uint4 (&fw)[4]) {
    const int r = s * kPsRows + lr;
    if (s >= 0 && r < a.n_q) {
      const uint16_t* fp = a.f + (bm * a.n_q + r) * kHeadDim + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) fw[ks] = ld16(fp + 32 * ks);
    } else {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) fw[ks] = make_uint4(0u, 0u, 0u, 0u);
    }
  };

  int s = grab();
  int s_prev = -1;  // slice whose assembled sets still wait in LDS
  uint4 fnext[4];
  load_f(s, fnext);
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): the first slice's F is in registers
  while (s >= 0) {
    uint4 fw[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) fw[ks] = fnext[ks];
    const int s_next = grab();
    load_f(s_next, fnext);
    // The previous slice's sets leave LDS now: these stores are long complete when the next
    // slice waits for the F rows requested just above.
    if (kStaged && s_prev >= 0) {
      wave_lds_sync();
      copy_out(a, bm, s_prev, ost, lane);
    }

    // ---- row geometry, forced blocks, padding, rows that take every candidate
    const int r = s * kPsRows + lr;
    const bool row_ok = r < a.n_q;
    const int64_t row = bm * a.n_q + r;
    const RowGeom g = row_geom(a.q_pos0 + r, a.n_init, a.n_local, a.k_total);
    int16_t* out = kStaged ? ost + lr * kPsOutPitch : a.sel + row * a.k_total;
    if (row_ok) {
      for (int i = lg; i < g.init_hi; i += 4) out[i] = (int16_t)i;
      const int n_loc = g.blk - g.local_lo + 1;
      for (int i = lg; i < n_loc; i += 4) out[g.init_hi + g.n_take + i] = (int16_t)(g.local_lo + i);
      for (int i = g.n_forced + g.n_take + lg; i < a.k_total; i += 4) out[i] = (int16_t)-1;
      if (lg == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
      if (g.n_take >= g.n_cand)
        for (int i = lg; i < g.n_cand; i += 4) out[g.init_hi + i] = (int16_t)(g.cand_lo + i);
    }
    const int64_t p_last = a.q_pos0 + min(a.n_q, (s + 1) * kPsRows) - 1;  // the slice's last row
    const RowGeom gs = row_geom(p_last, a.n_init, a.n_local, a.k_total);
    s_prev = s;
    s = s_next;
    if (gs.n_take >= gs.n_cand) continue;  // the slice's last row takes every candidate: all rows do

    // ---- scores: S^T = K~ F^T, one M-tile of 16 candidates at a time
    const int C = gs.n_cand;
    const int nmt = __builtin_amdgcn_readfirstlane((C + 15) >> 4);
    const int ntg = (nmt + 3) >> 2;  // groups of 4 M-tiles the slot loops run over
    const int Q = 4 * nmt;
    const int n = g.n_take, Cr = g.n_cand;
    const bool search = row_ok && n > 0 && n < Cr;
    const int v = search ? min(max(Cr - lg * Q, 0), Q) : Q;  // this lane's valid key slots
    float acc[kPsMaxMt][4];
    {
      bf16x8 fb[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) fb[ks] = as_bf16x8(fw[ks]);
      const uint16_t* ab = kst + ((lr >> 2) * Q + (lr & 3)) * kPsPitch + 8 * lg;
      // A fragments are read two M-tiles ahead of the MFMAs that use them (past the last M-tile
      // this reads rows up to 16 nmt + 7: inside the staged array).
      uint4 aw[3][4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) aw[0][ks] = *reinterpret_cast<const uint4*>(ab + 32 * ks);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) aw[1][ks] = *reinterpret_cast<const uint4*>(ab + 4 * kPsPitch + 32 * ks);
#pragma unroll
      for (int t = 0; t < kPsMaxMt; ++t) {
        if (t < nmt) {
#pragma unroll
          for (int ks = 0; ks < 4; ++ks)
            aw[(t + 2) % 3][ks] = *reinterpret_cast<const uint4*>(ab + 4 * (t + 2) * kPsPitch + 32 * ks);
          f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(as_bf16x8(aw[t % 3][ks]), fb[ks], c);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[t][i] = c[i];
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[t][i] = -INFINITY;
        }
      }
      // Key slots past the row's candidates (the last lane group's tail, rows with fewer
      // candidates than the slice) hold -inf, which no threshold admits.
#pragma unroll
      for (int t = 0; t < kPsMaxMt; ++t) {
        if (t < nmt && __ballot(4 * t + 4 > v) != 0ull) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (4 * t + i >= v) acc[t][i] = -INFINITY;
        }
      }
    }

    search_emit<kStaged>(acc, nmt, ntg, Q, v, n, Cr, search, lg, g, out, out + kPsStageK + lg);
  }
  if (kStaged && s_prev >= 0) {
    wave_lds_sync();
    copy_out(a, bm, s_prev, ost, lane);
  }
}

// ---- the (32, 16) window grid, scored in lockstep from LDS
//
// Read straight from L2 by every wavefront, the window keys of a unit are fetched once per slice:
// about 4 TB at the 32K prefill, and a kernel that does so waits on them.  This kernel takes a
// unit's slices in groups of kPwWaves consecutive ones, one per wavefront, all laid out with the
// quarter Q of the group's last slice (the one with the most candidates; rows with fewer get
// -inf slots).  Every wavefront of the group then reads the same window keys: chunks of
// kPwTiles window-tiles (4 kPwTiles windows of each quarter) are staged once per workgroup in
// LDS, double-buffered (a chunk is loaded piece by piece, M-tile by M-tile, while the previous
// one is scored), and the A fragments come from there.  Search and emission are the block grid's.
// Two 4-wavefront workgroups share a CU and drift apart, so that one's MFMA scoring overlaps the
// other's VALU search (a group's wavefronts are otherwise in the same phase).
// Once a group is scored the chunk buffers are free: each wavefront assembles its slice's sets
// there (rows of k_total rounded up to 8, plus 8 padding slots) and copies them out with 16-byte
// stores, for any k_total up to kPwStageKMax (a barrier before the next group's first staging
// protects them); larger sets are written straight to the output.
constexpr int kPwWaves = 4;                         // wavefronts (slices in lockstep) per workgroup
constexpr int kPwThreads = 64 * kPwWaves;
constexpr int kPwMt = 2;                            // M-tiles per staged chunk
constexpr int kPwTiles = 4 * kPwMt;                 // window-tiles per staged chunk
constexpr int kPwWin = 4 * kPwTiles;                // windows per quarter per chunk
constexpr int kPwPitch = kHeadDim + 16;             // bf16 per staged window row (288 B)
constexpr int kPwQuarter = kPwWin * kPwPitch + 64;  // uint16 per staged quarter (+128 B): with the
                                                    // 288-byte rows, the 16 rows one A read takes
                                                    // (4 quarters x 4 windows) count no LDS bank
                                                    // conflicts (272-byte rows with a 64-byte
                                                    // quarter shift count 3.8 cycles per read)
constexpr int kPwChunk = 4 * kPwQuarter;            // uint16 per chunk buffer
constexpr int kPwStageLd = 4 * kPwWin * 16 / kPwThreads;  // 16-byte staging pieces per thread
constexpr int kPwWinPerThr = kPwThreads / 16;       // windows of a quarter covered by one piece index
static_assert(kPwStageLd == 8 && kPwWin == 2 * kPwWinPerThr,
              "staging: thread t takes windows t / 16 and t / 16 + kPwWinPerThr of each quarter");
static_assert(kPwStageLd % kPwMt == 0, "each M-tile stages the same number of pieces");
constexpr int kPwStageKMax = 256;                   // largest k_total assembled in LDS
static_assert(kPwWaves * kPsRows * (kPwStageKMax + 8) <= 2 * kPwChunk, "set rows fit in the chunk buffers");
static_assert(2 * (2 * kPwChunk * 2) <= 160 * 1024, "two workgroups per CU");

__host__ __device__ inline int pw_out_pitch(int k_total) { return ((k_total + 7) & ~7) + 8; }

// Copies the assembled sets of a slice's valid rows (LDS rows `pitch` apart) to the output.
__device__ __forceinline__ void copy_out_rows(const SelectArgs& a, int64_t bm, int s, const int16_t* ost, int pitch,
                                              int lane) {
  const int nr = min(kPsRows, a.n_q - s * kPsRows);
  const int k = a.k_total;
  int16_t* dst = a.sel + (bm * a.n_q + (int64_t)s * kPsRows) * k;
  if (((reinterpret_cast<uintptr_t>(dst) | (uintptr_t)(2 * k)) & 15u) == 0) {
    const int per_row = k / 8;  // 16-byte chunks per row
    for (int i = lane; i < nr * per_row; i += 64) {
      const int r = i / per_row, c = i - r * per_row;
      *reinterpret_cast<uint4*>(dst + r * k + 8 * c) = *reinterpret_cast<const uint4*>(ost + r * pitch + 8 * c);
    }
  } else {
    for (int i = lane; i < nr * k; i += 64) {
      const int r = i / k;
      dst[i] = ost[r * pitch + (i - r * k)];
    }
  }
}

// kStaged: a slice's sets are assembled in the chunk buffers once the group is scored (k_total <=
// kPwStageKMax); otherwise they go straight to the output.
template <bool kStaged>
__global__ __launch_bounds__(kPwThreads, 2) void prefill_select_win_kernel(SelectArgs a, PrefillPlan plan, int n_groups) {
  __shared__ __align__(16) uint16_t wst[2 * kPwChunk];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bm = blockIdx.x % n_groups;
  const int u = (int)(blockIdx.x / n_groups);
  // Sweeps of U consecutive groups of kPwWaves slices: unit u takes group u of every even sweep
  // and group U - 1 - u of every odd one.  A group's cost grows with its position, so this
  // back-and-forth order gives every unit about the same work without a cost model.
  const int ns = plan.n_slices, U = plan.units;
  const int ng = (ns + kPwWaves - 1) / kPwWaves;
  if (u >= ng) return;  // uniform over the workgroup
  auto group_of = [&](int i) { return i * U + ((i & 1) ? U - 1 - u : u); };
  auto group_hi = [&](int gi) { return min(ns, kPwWaves * (gi + 1)); };
  int i_top = (ng - 1) / U;                // the last sweep, partial unless U divides ng
  if (group_of(i_top) >= ng) --i_top;      // then it may not reach this unit (the first sweep always does)
  const int lr = lane & 15, lg = lane >> 4;
  const int opitch = pw_out_pitch(a.k_total);
  int16_t* ost = reinterpret_cast<int16_t*>(wst) + wave * kPsRows * opitch;  // this wavefront's set rows
  const uint16_t* kcg = a.kc + bm * a.nc_cap * kHeadDim;  // the group's window keys
  auto load_f = [&](int s, int s_lo, uint4 (&fw)[4]) {
    const int r = s * kPsRows + lr;
    if (s >= s_lo && r < a.n_q) {
      const uint16_t* fp = a.f + (bm * a.n_q + r) * kHeadDim + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) fw[ks] = ld16(fp + 32 * ks);
    } else {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) fw[ks] = make_uint4(0u, 0u, 0u, 0u);
    }
  };

  uint4 fnext[4];
  load_f(group_hi(group_of(i_top)) - 1 - wave, kPwWaves * group_of(i_top), fnext);
  // Sweeps from the last (most candidates first); wavefront w takes slice g_hi - 1 - w.
  for (int i = i_top; i >= 0; --i) {
    const int gi = group_of(i);
    const int g_lo = kPwWaves * gi, g_hi = group_hi(gi);
    const int s = g_hi - 1 - wave;
    const bool have = s >= g_lo;
    uint4 fw[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) fw[ks] = fnext[ks];

    const int r = s * kPsRows + lr;
    const bool row_ok = have && r < a.n_q;
    const int64_t row = bm * a.n_q + r;
    const RowGeom g = row_geom(a.q_pos0 + (row_ok ? r : 0), a.n_init, a.n_local, a.k_total);
    int16_t* out = kStaged ? ost + lr * opitch : a.sel + row * a.k_total;
    // The group's last row (the most candidates and windows of any row of the group), and this
    // wavefront's slice.
    const int64_t pg_last = a.q_pos0 + min((int64_t)a.n_q, (int64_t)g_hi * kPsRows) - 1;
    const RowGeom gg = row_geom(pg_last, a.n_init, a.n_local, a.k_total);
    const bool group_scores = gg.n_take < gg.n_cand;  // else every row of the group takes everything
    const int64_t p_last = have ? a.q_pos0 + min(a.n_q, (s + 1) * kPsRows) - 1 : pg_last;
    const RowGeom gs = row_geom(p_last, a.n_init, a.n_local, a.k_total);
    const int64_t p_first = a.q_pos0 + (int64_t)(have ? s : 0) * kPsRows;
    const bool score = have && gs.n_take < gs.n_cand;  // uniform over the wavefront
    // forced blocks, padding, rows that take every candidate
    auto forced = [&]() {
      if (row_ok) {
        for (int i = lg; i < g.init_hi; i += 4) out[i] = (int16_t)i;
        const int n_loc = g.blk - g.local_lo + 1;
        for (int i = lg; i < n_loc; i += 4) out[g.init_hi + g.n_take + i] = (int16_t)(g.local_lo + i);
        for (int i = g.n_forced + g.n_take + lg; i < a.k_total; i += 4) out[i] = (int16_t)-1;
        if (lg == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
        if (g.n_take >= g.n_cand)
          for (int i = lg; i < g.n_cand; i += 4) out[g.init_hi + i] = (int16_t)(g.cand_lo + i);
      }
    };
    if (!kStaged) forced();

    const int nmt = (gg.n_cand + 15) >> 4;  // uniform over the workgroup
    const int ntg = (nmt + 3) >> 2;         // groups of 4 M-tiles the search's slot loops run over
    const int nch = (nmt + kPwMt - 1) / kPwMt;  // chunks
    const int Q = 4 * nmt;
    const int n = g.n_take, Cr = g.n_cand;
    const bool search = row_ok && n > 0 && n < Cr;
    const int v = search ? min(max(Cr - lg * Q, 0), Q) : Q;  // this lane's valid key slots
    float acc[kPsMaxMt][4];
    if (group_scores) {
      int32_t wg_first, wg_last;
      row_windows(gg, a.grid, pg_last, &wg_first, &wg_last);
      (void)wg_first;
      const int cl = gg.cand_lo;
      // Chunk c holds, for quarter q, windows 4 (cl + q Q + kPwTiles c) .. + kPwWin - 1; windows
      // past the group's last one repeat it (their scores never reach a valid slot).  Thread t
      // stages 16-byte part t % 16 of windows t / 16 and t / 16 + kPwWinPerThr of every quarter:
      // pieces x = 0 .. 7.
      const int st_w = tid >> 4, st_part = tid & 15;
      auto stage_piece = [&](int c, int x) -> uint4 {
        const int q = x >> 1, w = st_w + kPwWinPerThr * (x & 1);
        const int win = min(4 * (cl + q * Q + kPwTiles * c) + w, wg_last);
        return ld16(kcg + (int64_t)win * kHeadDim + st_part * 8);
      };
      auto stage_put = [&](int b, int x, uint4 val) {
        const int q = x >> 1, w = st_w + kPwWinPerThr * (x & 1);
        *reinterpret_cast<uint4*>(wst + b * kPwChunk + q * kPwQuarter + w * kPwPitch + st_part * 8) = val;
      };
      bf16x8 fb[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) fb[ks] = as_bf16x8(fw[ks]);
      const int bo = cl + lg * Q;  // first block of the scores this lane holds
      // Windows past the row's last complete one score -inf; only a slice whose candidate windows
      // reach past its first row's last complete window has any (n_local = 1).
      const bool need_vis = score && grid_win_hi(a.grid, gs.cand_lo + gs.n_cand - 1) > grid_win_vis(a.grid, p_first);
      const int vis = need_vis ? grid_win_vis(a.grid, a.q_pos0 + r) : 0x7fffffff;
      const bool vis_on = __ballot(need_vis) != 0ull;  // uniform: whether any window needs the mask
      float carry = -INFINITY;  // window 4 b - 1 of the next block: the previous tile's last window
      {
        uint4 sw[kPwStageLd];
#pragma unroll
        for (int x = 0; x < kPwStageLd; ++x) sw[x] = stage_piece(0, x);
        if (score) {
          // window-tile -1 (its last window is window 4 bo - 1), from the key cache
          const int wa = min(max(4 * (cl + (lr >> 2) * Q - 1) + (lr & 3), 0), wg_last);
          const uint16_t* pa = kcg + (int64_t)wa * kHeadDim + 8 * lg;
          f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(as_bf16x8(ld16(pa + 32 * ks)), fb[ks], c);
          carry = 4 * bo - 1 >= 0 ? c[3] : -INFINITY;  // window 4 bo - 1 exists unless bo = 0
        }
        if (kStaged) __syncthreads();  // the previous group's set rows have left the buffers
#pragma unroll
        for (int x = 0; x < kPwStageLd; ++x) stage_put(0, x, sw[x]);
      }
      __syncthreads();  // chunk 0 staged
      constexpr int kPer = kPwStageLd / kPwMt;  // pieces of the next chunk staged per M-tile
#pragma unroll
      for (int c = 0; c < kPsMaxMt / kPwMt; ++c) {
        if (c < nch) {  // uniform over the workgroup
          const uint16_t* ab = wst + (c & 1) * kPwChunk + (lr >> 2) * kPwQuarter + (lr & 3) * kPwPitch + 8 * lg;
          const bool st_next = c + 1 < nch;  // then chunk c has all its M-tiles
#pragma unroll
          for (int k = 0; k < kPwMt; ++k) {
            const int mt = kPwMt * c + k;
            if (mt < nmt) {
              uint4 sp[kPer];
              if (st_next) {
#pragma unroll
                for (int x = 0; x < kPer; ++x) sp[x] = stage_piece(c + 1, kPer * k + x);
              }
              if (score) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  const uint16_t* ap = ab + 4 * (4 * k + i) * kPwPitch;  // window-tile 4 k + i of the chunk
                  f32x4 cc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                  for (int ks = 0; ks < 4; ++ks)
                    cc = mfma16x16x32(as_bf16x8(*reinterpret_cast<const uint4*>(ap + 32 * ks)), fb[ks], cc);
                  if (vis_on) {
                    // window 4 (bo + u) + e is visible iff it is <= vis: all-ones mask selects -inf
                    const int d = vis - 4 * (bo + 4 * mt + i);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                      const uint32_t m = (uint32_t)((d - e) >> 31);
                      cc[e] = __uint_as_float((m & 0xff800000u) | (~m & __float_as_uint(cc[e])));
                    }
                  }
                  acc[mt][i] = fmaxf(fmaxf(fmaxf(cc[0], cc[1]), fmaxf(cc[2], cc[3])), carry);
                  carry = cc[3];
                }
              } else {  // defined on every path, so that no slot lives on from an earlier group
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[mt][i] = -INFINITY;
              }
              if (st_next) {
#pragma unroll
                for (int x = 0; x < kPer; ++x) stage_put((c + 1) & 1, kPer * k + x, sp[x]);
              }
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[mt][i] = -INFINITY;
            }
          }
          __syncthreads();  // chunk c scored everywhere; chunk c + 1 staged
        } else {
#pragma unroll
          for (int k = 0; k < kPwMt; ++k)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[kPwMt * c + k][i] = -INFINITY;
        }
      }
    } else if (kStaged) {
      __syncthreads();  // the previous group's set rows have left the buffers
    }
    // the next group's F rows, requested after the scoring, whose registers they would crowd
    if (i > 0) load_f(group_hi(group_of(i - 1)) - 1 - wave, kPwWaves * group_of(i - 1), fnext);
    if (kStaged) forced();  // the buffers are free now

    if (score) {
      // Key slots past the row's candidates (the last lane group's tail, rows with fewer
      // candidates than the group's last row) hold -inf, which no threshold admits.
#pragma unroll
      for (int t = 0; t < kPsMaxMt; ++t) {
        if (t < nmt && __ballot(4 * t + 4 > v) != 0ull) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (4 * t + i >= v) acc[t][i] = -INFINITY;
        }
      }
      search_emit<kStaged>(acc, nmt, ntg, Q, v, n, Cr, search, lg, g, out, out + opitch - 8 + lg);
    }
    if (kStaged && have) {
      wave_lds_sync();
      copy_out_rows(a, bm, s, ost, opitch, lane);
    }
  }
}

hipError_t launch_prefill_select(const SelectArgs& a, hipStream_t stream) {
  const int n_groups = a.batch * a.n_kv_heads;
  const int ns = (a.n_q + kPsRows - 1) / kPsRows;
  if (ns > 65535) return hipErrorInvalidValue;
  const bool win = !grid_is_blocks(a.grid);
  if (win && !(a.grid.l == 32 && a.grid.s == 16)) return hipErrorInvalidValue;
  // persistent units: one per CU for the block grid, two per CU for the window grid
  const int units_target = win ? 512 : 256;
  int units = n_groups >= units_target ? 1 : units_target / n_groups;
  units = std::max(1, std::min(units, std::min(ns, kPsMaxUnits)));
  // Both kernels take their slices (window grid: groups of kPwWaves slices) by unit index in
  // back-and-forth sweeps.
  if (win) units = std::min(units, (ns + kPwWaves - 1) / kPwWaves);
  PrefillPlan plan;
  plan.n_slices = ns;
  plan.units = units;
  const dim3 grid((unsigned)((int64_t)n_groups * units));
  const bool staged = a.k_total <= kPsStageK;
  if (win && a.k_total <= kPwStageKMax)
    hipLaunchKernelGGL((prefill_select_win_kernel<true>), grid, dim3(kPwThreads), 0, stream, a, plan, n_groups);
  else if (win)
    hipLaunchKernelGGL((prefill_select_win_kernel<false>), grid, dim3(kPwThreads), 0, stream, a, plan, n_groups);
  else if (staged)
    hipLaunchKernelGGL((prefill_select_kernel<true>), grid, dim3(kPsThreads), 0, stream, a, plan, n_groups);
  else
    hipLaunchKernelGGL((prefill_select_kernel<false>), grid, dim3(kPsThreads), 0, stream, a, plan, n_groups);
  return hipGetLastError();
}

}  // namespace sparda

// attention.hip -- block-sparse attention over the attended block sets (paper Sec. 4.1, Eq. 5,
// over the set of Eq. 1): o = softmax(sm_scale * q K_S^T) V_S for the tokens t <= p of the
// attended blocks S, all G query heads of a GQA group sharing S.
//
// Work unit: one query row (batch b, group m, row r) and a split of its selected-block list.  A
// workgroup has 8 wavefronts; each wavefront walks blocks split_begin + wave, +8, ... with its own
// online-softmax state, then the 8 states are merged through LDS.  With 256 or more rows (e.g.
// batch 32 x 8 groups) a row is one split and the workgroup writes the bf16 output directly;
// with fewer rows the block list is split, the merged (max, sum, acc) partials go to the
// workspace, and a combine kernel merges them by log-sum-exp.
//
// Per 64-token block a wavefront:
//   * loads the 16 KiB K block as the MFMA A operand (token rows x head-dim columns, 16-byte
//     loads, 64 contiguous bytes per row segment) and the 16 KiB V block as 16 fully
//     contiguous 1 KiB wavefront loads, both issued before any math;
//   * computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (M = 16 tokens, N = the G <= 16 heads
//     of the group, K = 32 head dims): 16 MFMAs per block;
//   * masks tokens after p (the query's own block), exponentiates in the exp2 domain, and
//     passes P through a 4 KiB per-wave LDS slice;
//   * accumulates P V on the VALU (lane = 8 head dims x one token in four): decode has only G
//     query rows per block, so the PV product is bandwidth-bound work, not an MFMA contraction.
#include <math.h>

#include "device_util.hpp"
#include "launch.hpp"
#include "select_block.hpp"

namespace sparda {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kAttnWaves = 8;        // wavefronts per attention workgroup
constexpr int kRowsFillChip = 256;   // rows at which one workgroup per row fills 256 CUs
constexpr int kMaxSplits = 64;
constexpr int kKstPitch = kHeadDim + 16;  // uint16 per staged K row (288 B)
constexpr int kStepMaxK = 1024;           // largest k_total of the fused decode step (its set lives in LDS)

// LDS of one attention workgroup.  kst: K of each wavefront's current block, transposed through
// LDS: read from HBM as 1 KiB rows of 4 tokens (the access pattern streams faster than 16 token
// rows x 64 bytes), stored at a 288-byte row pitch whose A-operand reads (16 rows x 4 chunks)
// count no bank conflicts.  The merge of the wavefront states reuses this space after the loop.
template <int G, int NW>
struct AttnLds {
  uint16_t kst[NW][kBlock * kKstPitch];
  float p_lds[NW][64][G];
  float st_m[NW][G], st_l[NW][G];
};

// Attention of query row `row`, split `split` of its block list, by a workgroup of NW
// wavefronts (every thread must call it).  srow: the row's a.k_total entries (global or LDS),
// n_listed: its count.
template <int G, int NW>
__device__ __forceinline__ void attend_row(const AttnArgs& a, int64_t row, int split, AttnLds<G, NW>& L,
                                           const int16_t* srow, int n_listed) {
  auto& kst = L.kst;
  auto& p_lds = L.p_lds;
  auto& st_m = L.st_m;
  auto& st_l = L.st_l;
  static_assert(sizeof(float) * G * kHeadDim <= sizeof(uint16_t) * kBlock * kKstPitch, "a wavefront's merge state fits in its K slice");
  // wavefront w's (G x kHeadDim) partial output, in its own K slice once its blocks are done
  auto st_acc = [&](int w) { return reinterpret_cast<float (*)[kHeadDim]>(&kst[w][0]); };
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = (int)(row % a.n_q);
  const int64_t bm = row / a.n_q;
  const int m = (int)(bm % a.n_kv_heads);
  const int b = (int)(bm / a.n_kv_heads);
  const int64_t p = a.q_pos0 + r;
  const int blk = (int)(p / kBlock);
  const int n = n_listed > a.k_total ? a.k_total : (n_listed < 0 ? 0 : n_listed);
  const int s_begin = split * a.blocks_per_split;
  const int s_end = min(n, s_begin + a.blocks_per_split);
  const int64_t Hq = (int64_t)a.n_kv_heads * G;
  const float zscale = a.sm_scale * kLog2e;

  const int hh = lane & 15;   // S^T column (head) of this lane; also the PV dim chunk
  const int grp = lane >> 4;  // k-chunk of the MFMA operands; also the PV token phase
  bf16x8 qb[4];
  {
    const uint16_t* qrow = a.q + (((int64_t)b * Hq + (int64_t)m * G + hh) * a.n_q + r) * kHeadDim + 8 * grp;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qb[ks] = as_bf16x8(hh < G ? ld16(qrow + 32 * ks) : make_uint4(0u, 0u, 0u, 0u));
  }
  float m_run = -INFINITY, l_run = 0.f;
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;

  // The attended tokens are a union of blocks: an entry whose block an earlier entry of the row
  // already lists is skipped.  Lane e holds entry e (e < 64): the walk reads entries below 64 from
  // it, so it issues no loads of its own between the blocks' loads.
  const int entry = lane < n ? (int)srow[lane] : -1;
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the query and the entries are in registers
  // First entry at or after s (stepping by NW) that names a visible block no earlier entry names;
  // *jo gets its block.  Returns a value >= s_end when there is none.
  auto next_block = [&](int s, int* jo) {
    for (; s < s_end; s += NW) {
      const int j = s < 64 ? __builtin_amdgcn_readlane(entry, s) : __builtin_amdgcn_readfirstlane((int)srow[s]);
      if (j < 0 || j > blk) continue;
      bool dup = __ballot(lane < s && entry == j) != 0ull;
      for (int e0 = 64; e0 < s; e0 += 64) {
        const int e = e0 + lane;
        dup |= __ballot(e < s && (int)srow[e] == j) != 0ull;
      }
      if (!dup) {
        *jo = j;
        return s;
      }
    }
    return s;
  };
  auto kv_base = [&](int s, int j) -> int64_t {
    return a.kv_mode == 0 ? (bm * a.t_cap + (int64_t)j * kBlock) * kHeadDim : ((bm * a.k_total + s) * kBlock) * kHeadDim;
  };
  // Rows of 4 tokens, 1 KiB per wavefront load, for K and V alike.  K pieces [lo, hi).
  uint4 kw[16], vw[16];
  auto load_k = [&](int64_t base, int lo, int hi) {
#pragma unroll
    for (int it = 0; it < 16; ++it)
      if (it >= lo && it < hi) kw[it] = ld16_nt(a.k + base + (4 * it + grp) * kHeadDim + 8 * hh);
  };
  auto load_v = [&](int64_t base) {
#pragma unroll
    for (int it = 0; it < 16; ++it) vw[it] = ld16_nt(a.v + base + (4 * it + grp) * kHeadDim + 8 * hh);
  };
  uint16_t* ks_w = &kst[wave][0];
  // Software pipeline over the wavefront's blocks: the first half of the next block's K is
  // requested as soon as the current K has gone through the MFMAs (its registers are free once the
  // K is in the LDS slice), so the wavefront has loads in flight while it computes; the rest of
  // that K and its V follow at the top of the next iteration (all of it would not fit beside V).
  constexpr int kKAhead = G <= 4 ? 4 : 0;  // K pieces requested one block ahead (none above 4 heads: they would spill)
  int j = 0;
  int s = next_block(s_begin + wave, &j);
  if (s < s_end) load_k(kv_base(s, j), 0, kKAhead);
  while (s < s_end) {
    int jn = 0;
    const int sn = next_block(s + NW, &jn);
    const int64_t base = kv_base(s, j);
    const int64_t base_n = sn < s_end ? kv_base(sn, jn) : 0;
    load_k(base, kKAhead, 16);
    load_v(base);
    wave_lds_sync();  // the previous block's K reads are done
#pragma unroll
    for (int it = 0; it < 16; ++it) *reinterpret_cast<uint4*>(ks_w + (4 * it + grp) * kKstPitch + 8 * hh) = kw[it];
    wave_lds_sync();

    f32x4 st[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      st[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 kf = *reinterpret_cast<const uint4*>(ks_w + (16 * tt + hh) * kKstPitch + 32 * ks + 8 * grp);
        st[tt] = mfma16x16x32(as_bf16x8(kf), qb[ks], st[tt]);
      }
    }
    if (sn < s_end) load_k(base_n, 0, kKAhead);
    // lane holds S^T[token 16 tt + 4 grp + i][head hh]
    const int last = (j == blk) ? (int)(p - (int64_t)j * kBlock) : kBlock - 1;
    float z[4][4];
    float bmax = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = 16 * tt + 4 * grp + i;
        z[tt][i] = tok <= last ? st[tt][i] * zscale : -INFINITY;
        bmax = fmaxf(bmax, z[tt][i]);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float m_new = fmaxf(m_run, bmax);  // token 0 of a block is always <= p: finite
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pz = exp2f(z[tt][i] - m_new);
        psum += pz;
        if (hh < G) p_lds[wave][16 * tt + 4 * grp + i][hh] = pz;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
    wave_lds_sync();
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ah = readlane_f(alpha, h);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] *= ah;
    }
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const int tok = 4 * it + grp;
      const bool ok = tok <= last;  // never multiply by unwritten values after p
      const uint4 w = ok ? vw[it] : make_uint4(0u, 0u, 0u, 0u);
      const float v8[8] = {bf16lo(w.x), bf16hi(w.x), bf16lo(w.y), bf16hi(w.y),
                           bf16lo(w.z), bf16hi(w.z), bf16lo(w.w), bf16hi(w.w)};
      float pr[G];
#pragma unroll
      for (int h = 0; h < G; ++h) pr[h] = p_lds[wave][tok][h];
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pr[h], v8[e], acc[h][e]);
    }
    wave_lds_sync();
    s = sn;
    j = jn;
  }
  // Sum the four token phases of each head-dim chunk.
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = acc[h][e];
      x += __shfl_xor(x, 16, 64);
      x += __shfl_xor(x, 32, 64);
      acc[h][e] = x;
    }
  if (lane < G) {
    st_m[wave][lane] = m_run;
    st_l[wave][lane] = l_run;
  }
  if (lane < 16) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) st_acc(wave)[h][8 * lane + e] = acc[h][e];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * kHeadDim; idx += NW * 64) {
    const int h = idx / kHeadDim, d = idx % kHeadDim;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, st_m[w][h]);
    float L = 0.f, A = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float mw = st_m[w][h];
        if (mw != -INFINITY) {
          const float sc = exp2f(mw - M);
          L = fmaf(st_l[w][h], sc, L);
          A = fmaf(st_acc(w)[h][d], sc, A);
        }
      }
    }
    if (a.n_splits == 1) {
      a.o[(((int64_t)b * Hq + (int64_t)m * G + h) * a.n_q + r) * kHeadDim + d] = f32_to_bf16(L > 0.f ? A / L : 0.f);
    } else {
      float* pp = a.ws + ((row * a.n_splits + split) * G + h) * (kHeadDim + 2);
      if (d == 0) {
        pp[0] = M;
        pp[1] = L;
      }
      pp[2 + d] = A;
    }
  }
}

template <int G, int NW>
__global__ __launch_bounds__(NW * 64) void sparse_attn_kernel(AttnArgs a) {
  __shared__ __align__(16) AttnLds<G, NW> lds;
  const int64_t row = blockIdx.x;
  attend_row<G, NW>(a, row, blockIdx.y, lds, a.sel + row * a.k_total, a.cnt[row]);
}

// One decode step of a (batch, group) row: the row's Forecast selection (Sec. 4.1, Eq. 4 with
// Eq. 1), then its sparse attention over that set (Eq. 5), in one workgroup per (row, split).
// kSplitSel: the row's window scores were written to the workspace by the split decode path's
// scoring launch, and the workgroup only selects (decode_topk_row); otherwise it scores and
// selects (decode_select_row).  The selection's scores live in the attention's K (or V) slices,
// both free until the attention starts; the set itself is kept in LDS, and split 0 writes it to
// s.sel / s.cnt.  With splits (fewer rows than CUs) every split's workgroup computes the same
// selection: it reads a fraction of the attention's bytes, and the rows' attention then starts
// without another launch.  Rows finish their selection at different times, so some rows'
// attention loads already run while others select: the HBM stays busier than with a selection
// kernel followed by an attention kernel.
template <bool kSplitSel>
__device__ __forceinline__ void step_select(const SelectArgs& s, int64_t row, float* sc, uint32_t* hist, int* wave_cnt,
                                            int* pick, int16_t* set, int16_t* set_cnt) {
  if constexpr (kSplitSel)
    decode_topk_row(s, row, sc, hist, wave_cnt, pick, set, set_cnt);
  else
    decode_select_row(s, row, sc, hist, wave_cnt, pick, set, set_cnt);
  __syncthreads();  // the row's set is in LDS, and the selection's LDS is free
  if (blockIdx.y == 0) {
    for (int i = threadIdx.x; i < s.k_total; i += kDecThreads) s.sel[row * s.k_total + i] = set[i];
    if (threadIdx.x == 0) s.cnt[row] = *set_cnt;
  }
}

template <int G, int NW, bool kSplitSel>
__global__ __launch_bounds__(NW * 64) void decode_step_kernel(SelectArgs s, AttnArgs a) {
  static_assert(NW * 64 == kDecThreads, "the selection runs on the attention workgroup");
  static_assert(sizeof(float) * kDecodeMaxCand <= sizeof(uint16_t) * NW * kBlock * kKstPitch, "scores fit in the K slices");
  static_assert(sizeof(uint32_t) * kTopkLds <= sizeof(float) * NW * 64 * G, "the top-k histogram fits in the P space");
  __shared__ __align__(16) AttnLds<G, NW> lds;
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  __shared__ __align__(16) int16_t set[kStepMaxK];
  __shared__ int16_t set_cnt;
  const int64_t row = blockIdx.x;
  step_select<kSplitSel>(s, row, reinterpret_cast<float*>(&lds.kst[0][0]), reinterpret_cast<uint32_t*>(&lds.p_lds[0][0][0]),
                         wave_cnt, pick, set, &set_cnt);
  attend_row<G, NW>(a, row, blockIdx.y, lds, set, set_cnt);
}

// Decode attention for groups of 6 to 16 heads: P V on MFMA.  With this many query rows per
// block the VALU P V of sparse_attn_kernel (G x 8 FMAs per token per lane) no longer hides under
// the loads, while P V fills a 16-column MFMA tile.  Per 64-token block a wavefront:
//   * loads K and V as sparse_attn_kernel does and computes S^T = K Q^T (lane (n, g) holds
//     head n's scores of tokens 16 tt + 4 g + i);
//   * stages V in its LDS slice (272-byte rows; tokens after p are zeroed) and computes
//     O^T += V^T P^T on v_mfma_f32_16x16x32_bf16 in two 32-token chunks: the B operand of chunk c
//     is lane (n, g)'s own probabilities of tiles 2c and 2c + 1 rounded to bf16 (k = 8 g + j holds
//     token 16 (2 c + j / 4) + 4 g + j % 4), the A operand (dims x those tokens) is read from LDS;
//   * the softmax denominator sums the same bf16-rounded probabilities.
// Lane (n, g) accumulates dims 16 dt + 4 g + e of head n in o[dt]; the wavefronts' states merge
// through LDS (the V slices' space) as in sparse_attn_kernel.
constexpr int kWidePitch = 136;  // uint16 per staged V row (272 B: 16-byte aligned, bank-spread)

// LDS of one workgroup of the wide kernel: the V slices (also the wavefronts' merge space).
struct WideLds {
  uint16_t vst[kAttnWaves][kBlock * kWidePitch];
};

// The wide kernel's attention of query row `row`, split `split`, over srow (a.k_total entries,
// global or LDS) with n_listed of them valid.  Every thread of the workgroup must call it.
template <int G>
__device__ __forceinline__ void attend_row_wide(const AttnArgs& a, int64_t row, int split, WideLds& L,
                                                const int16_t* srow, int n_listed) {
  constexpr int NW = kAttnWaves;
  auto& vst = L.vst;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = (int)(row % a.n_q);
  const int64_t bm = row / a.n_q;
  const int m = (int)(bm % a.n_kv_heads);
  const int b = (int)(bm / a.n_kv_heads);
  const int64_t p = a.q_pos0 + r;
  const int blk = (int)(p / kBlock);
  const int n = n_listed > a.k_total ? a.k_total : (n_listed < 0 ? 0 : n_listed);
  const int s_begin = split * a.blocks_per_split;
  const int s_end = min(n, s_begin + a.blocks_per_split);
  const int64_t Hq = (int64_t)a.n_kv_heads * G;
  const float zscale = a.sm_scale * kLog2e;
  const int hh = lane & 15;   // head (S^T column, O^T column)
  const int grp = lane >> 4;  // k-chunk of the QK operands; token group of P; dim group of O^T
  bf16x8 qb[4];
  {  // columns past the group's heads read head 0 (a valid address) and are zeroed
    const uint16_t* qrow =
        a.q + (((int64_t)b * Hq + (int64_t)m * G + (hh < G ? hh : 0)) * a.n_q + r) * kHeadDim + 8 * grp;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 v = ld16(qrow + 32 * ks);
      qb[ks] = as_bf16x8(hh < G ? v : make_uint4(0u, 0u, 0u, 0u));
    }
  }
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint16_t* vs = vst[wave];

  const int entry = lane < n ? (int)srow[lane] : -1;
  for (int s = s_begin + wave; s < s_end; s += NW) {
    const int j = __builtin_amdgcn_readfirstlane((int)srow[s]);
    if (j < 0 || j > blk) continue;
    bool dup = __ballot(lane < s && entry == j) != 0ull;
    for (int e0 = 64; e0 < s; e0 += 64) {
      const int e = e0 + lane;
      dup |= __ballot(e < s && (int)srow[e] == j) != 0ull;
    }
    if (dup) continue;
    const int64_t base = a.kv_mode == 0 ? (bm * a.t_cap + (int64_t)j * kBlock) * kHeadDim
                                        : ((bm * a.k_total + s) * kBlock) * kHeadDim;
    const uint16_t* kb = a.k + base;
    const uint16_t* vb = a.v + base;
    uint4 kw[4][4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) kw[tt][ks] = ld16(kb + (16 * tt + hh) * kHeadDim + 32 * ks + 8 * grp);
    uint4 vw[16];
#pragma unroll
    for (int it = 0; it < 16; ++it) vw[it] = ld16(vb + (4 * it + grp) * kHeadDim + 8 * hh);

    f32x4 st[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      st[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) st[tt] = mfma16x16x32(as_bf16x8(kw[tt][ks]), qb[ks], st[tt]);
    }
    const int last = (j == blk) ? (int)(p - (int64_t)j * kBlock) : kBlock - 1;
    // V into the wavefront's LDS slice, tokens after p as zeros (their values are not written)
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const int tok = 4 * it + grp;
      *reinterpret_cast<uint4*>(vs + tok * kWidePitch + 8 * hh) = tok <= last ? vw[it] : make_uint4(0u, 0u, 0u, 0u);
    }
    float z[4][4];
    float bmax = -INFINITY;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = 16 * tt + 4 * grp + i;
        z[tt][i] = tok <= last ? st[tt][i] * zscale : -INFINITY;
        bmax = fmaxf(bmax, z[tt][i]);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float m_new = fmaxf(m_run, bmax);  // token 0 of a block is always <= p: finite
    const float alpha = exp2f(m_run - m_new);
    uint32_t pw[4][2];  // bf16 pairs of tile tt: (i = 0, 1), (i = 2, 3)
    float psum = 0.f;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int q2 = 0; q2 < 2; ++q2) {
        const uint16_t lo = f32_to_bf16(exp2f(z[tt][2 * q2] - m_new));
        const uint16_t hi = f32_to_bf16(exp2f(z[tt][2 * q2 + 1] - m_new));
        psum += __uint_as_float((uint32_t)lo << 16) + __uint_as_float((uint32_t)hi << 16);
        pw[tt][q2] = (uint32_t)lo | ((uint32_t)hi << 16);
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
    wave_lds_sync();
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const bf16x8 pb = as_bf16x8(make_uint4(pw[2 * c][0], pw[2 * c][1], pw[2 * c + 1][0], pw[2 * c + 1][1]));
      // A rows: dim 16 dt + hh; k = 8 grp + jj -> token 16 (2 c + jj / 4) + 4 grp + jj % 4
      const uint16_t* r0 = vs + (16 * (2 * c) + 4 * grp) * kWidePitch + hh;
      const uint16_t* r1 = vs + (16 * (2 * c + 1) + 4 * grp) * kWidePitch + hh;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        uint32_t aw[4];
#pragma unroll
        for (int q2 = 0; q2 < 2; ++q2) {
          aw[q2] = (uint32_t)r0[(2 * q2) * kWidePitch + 16 * dt] | ((uint32_t)r0[(2 * q2 + 1) * kWidePitch + 16 * dt] << 16);
          aw[2 + q2] =
              (uint32_t)r1[(2 * q2) * kWidePitch + 16 * dt] | ((uint32_t)r1[(2 * q2 + 1) * kWidePitch + 16 * dt] << 16);
        }
        o[dt] = mfma16x16x32(as_bf16x8(make_uint4(aw[0], aw[1], aw[2], aw[3])), pb, o[dt]);
      }
    }
    wave_lds_sync();
  }

  // Merge the wavefronts' states through the V slices' space.
  __syncthreads();
  float* st_m = reinterpret_cast<float*>(&vst[0][0]);  // [NW][16]
  float* st_l = st_m + NW * 16;                         // [NW][16]
  float* st_acc = st_l + NW * 16;                       // [NW][16][128]
  if (grp == 0) {
    st_m[wave * 16 + hh] = m_run;
    st_l[wave * 16 + hh] = l_run;
  }
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int e = 0; e < 4; ++e) st_acc[(wave * 16 + hh) * kHeadDim + 16 * dt + 4 * grp + e] = o[dt][e];
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * kHeadDim; idx += NW * 64) {
    const int h = idx / kHeadDim, d = idx % kHeadDim;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, st_m[w * 16 + h]);
    float L = 0.f, A = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float mw = st_m[w * 16 + h];
        if (mw != -INFINITY) {
          const float sc = exp2f(mw - M);
          L = fmaf(st_l[w * 16 + h], sc, L);
          A = fmaf(st_acc[(w * 16 + h) * kHeadDim + d], sc, A);
        }
      }
    }
    if (a.n_splits == 1) {
      a.o[(((int64_t)b * Hq + (int64_t)m * G + h) * a.n_q + r) * kHeadDim + d] = f32_to_bf16(L > 0.f ? A / L : 0.f);
    } else {
      float* pp = a.ws + ((row * a.n_splits + split) * G + h) * (kHeadDim + 2);
      if (d == 0) {
        pp[0] = M;
        pp[1] = L;
      }
      pp[2 + d] = A;
    }
  }
}

template <int G>
__global__ __launch_bounds__(kAttnWaves * 64) void sparse_attn_wide_kernel(AttnArgs a) {
  __shared__ __align__(16) WideLds lds;
  const int64_t row = blockIdx.x;
  attend_row_wide<G>(a, row, blockIdx.y, lds, a.sel + row * a.k_total, a.cnt[row]);
}

// The decode step with the wide kernel's attention (6 <= G <= 16): as decode_step_kernel.
template <int G, bool kSplitSel>
__global__ __launch_bounds__(kAttnWaves * 64) void decode_step_wide_kernel(SelectArgs s, AttnArgs a) {
  static_assert(kAttnWaves * 64 == kDecThreads, "the selection runs on the attention workgroup");
  static_assert(sizeof(float) * kDecodeMaxCand <= sizeof(WideLds), "scores fit in the V slices");
  __shared__ __align__(16) WideLds lds;
  __shared__ __align__(16) uint32_t hist[kTopkLds];
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  __shared__ __align__(16) int16_t set[kStepMaxK];
  __shared__ int16_t set_cnt;
  const int64_t row = blockIdx.x;
  step_select<kSplitSel>(s, row, reinterpret_cast<float*>(&lds.vst[0][0]), hist, wave_cnt, pick, set, &set_cnt);
  attend_row_wide<G>(a, row, blockIdx.y, lds, set, set_cnt);
}

// Merge the split partials of one (row, head) by log-sum-exp: 128 threads, one per head dim.
template <int G>
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnArgs a) {
  __shared__ float w_s[kMaxSplits], l_s[kMaxSplits];
  __shared__ float total_l;
  const int64_t rh = blockIdx.x;
  const int64_t row = rh / G;
  const int h = (int)(rh % G);
  const int r = (int)(row % a.n_q);
  const int64_t bm = row / a.n_q;
  const int m = (int)(bm % a.n_kv_heads);
  const int b = (int)(bm / a.n_kv_heads);
  const int64_t Hq = (int64_t)a.n_kv_heads * G;
  const int tid = threadIdx.x;
  const int64_t stride = (int64_t)G * (kHeadDim + 2);
  const float* base = a.ws + (row * a.n_splits * G + h) * (kHeadDim + 2);
  const int ns = a.n_splits;  // <= kMaxSplits
  for (int s = tid; s < ns; s += 128) {
    w_s[s] = base[s * stride];
    l_s[s] = base[s * stride + 1];
  }
  __syncthreads();
  if (tid < 64) {
    float M = -INFINITY;
    for (int s = tid; s < ns; s += 64) M = fmaxf(M, w_s[s]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
    float L = 0.f;
    for (int s = tid; s < ns; s += 64) {
      const float ms = w_s[s];
      const float wgt = (M == -INFINITY || ms == -INFINITY) ? 0.f : exp2f(ms - M);
      w_s[s] = wgt;
      L = fmaf(l_s[s], wgt, L);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) L += __shfl_xor(L, o, 64);
    if (tid == 0) total_l = L;
  }
  __syncthreads();
  float A = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float wgt = w_s[s];
    if (wgt != 0.f) A = fmaf(base[s * stride + 2 + tid], wgt, A);
  }
  const float L = total_l;
  a.o[(((int64_t)b * Hq + (int64_t)m * G + h) * a.n_q + r) * kHeadDim + tid] = f32_to_bf16(L > 0.f ? A / L : 0.f);
}

void attn_plan(int64_t rows, int32_t k_total, int32_t* n_splits, int32_t* blocks_per_split) {
  // One 8-wave workgroup per row when there are enough rows to fill the chip (no partials, no
  // combine).  With fewer rows, split the block list into about one workgroup per CU (the
  // decode kernels fit one workgroup per CU, so a second round of workgroups would only add
  // prologues and merges: 53.7 -> 44.5 us at 64 rows of 16 heads, 39.3 -> 36.0 us at 64 rows of 4),
  // keeping at least one block per wavefront.
  int ns = 1;
  if (rows < kRowsFillChip) {
    const int max_splits = (k_total + kAttnWaves - 1) / kAttnWaves;
    const int64_t want = (kRowsFillChip + rows - 1) / rows;
    ns = (int)(want < max_splits ? want : max_splits);
    if (ns > kMaxSplits) ns = kMaxSplits;
    if (ns < 1) ns = 1;
  }
  const int bps = (k_total + ns - 1) / ns;
  *n_splits = (k_total + bps - 1) / bps;
  *blocks_per_split = bps;
}

template <int G>
static hipError_t launch_g(const AttnArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads * a.n_q;
  // Up to 5 heads: P V on the VALU.  6 to 16 heads: P V on MFMA (sparse_attn_wide_kernel; at 6
  // heads the VALU kernel's accumulators no longer fit beside a block's K and V without spills).
  dim3 grid((unsigned)rows, (unsigned)a.n_splits);
  if constexpr (G <= 5)
    hipLaunchKernelGGL((sparse_attn_kernel<G, kAttnWaves>), grid, dim3(kAttnWaves * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((sparse_attn_wide_kernel<G>), grid, dim3(kAttnWaves * 64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_splits == 1) return e;
  hipLaunchKernelGGL(attn_combine_kernel<G>, dim3((unsigned)(rows * G)), dim3(128), 0, stream, a);
  return hipGetLastError();
}

template <int G, bool kWide>
static hipError_t launch_step_g(const SelectArgs& s, const AttnArgs& a, bool split_sel, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads;
  const dim3 grid((unsigned)rows, (unsigned)a.n_splits), block(kAttnWaves * 64);
  if constexpr (kWide) {
    if (split_sel)
      hipLaunchKernelGGL((decode_step_wide_kernel<G, true>), grid, block, 0, stream, s, a);
    else
      hipLaunchKernelGGL((decode_step_wide_kernel<G, false>), grid, block, 0, stream, s, a);
  } else {
    if (split_sel)
      hipLaunchKernelGGL((decode_step_kernel<G, kAttnWaves, true>), grid, block, 0, stream, s, a);
    else
      hipLaunchKernelGGL((decode_step_kernel<G, kAttnWaves, false>), grid, block, 0, stream, s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_splits == 1) return e;
  hipLaunchKernelGGL(attn_combine_kernel<G>, dim3((unsigned)(rows * G)), dim3(128), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_decode_step(const SelectArgs& s, const AttnArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads;
  const int path = select_decode_path(rows, 1, s.q_pos0, s.n_init, s.n_local, s.grid);
  const bool fused = a.n_q == 1 && s.n_q == 1 && a.kv_mode == 0 && a.k_total <= kStepMaxK && path >= 0;
  if (fused) {
    const bool split_sel = path == 1;
    if (split_sel) {
      hipError_t e = launch_decode_split_scores(s, stream);
      if (e != hipSuccess) return e;
    }
    switch (a.group_size) {
      case 1: return launch_step_g<1, false>(s, a, split_sel, stream);
      case 2: return launch_step_g<2, false>(s, a, split_sel, stream);
      case 3: return launch_step_g<3, false>(s, a, split_sel, stream);
      case 4: return launch_step_g<4, false>(s, a, split_sel, stream);
      case 5: return launch_step_g<5, false>(s, a, split_sel, stream);
      case 6: return launch_step_g<6, true>(s, a, split_sel, stream);
      case 7: return launch_step_g<7, true>(s, a, split_sel, stream);
      case 8: return launch_step_g<8, true>(s, a, split_sel, stream);
      case 9: return launch_step_g<9, true>(s, a, split_sel, stream);
      case 10: return launch_step_g<10, true>(s, a, split_sel, stream);
      case 11: return launch_step_g<11, true>(s, a, split_sel, stream);
      case 12: return launch_step_g<12, true>(s, a, split_sel, stream);
      case 13: return launch_step_g<13, true>(s, a, split_sel, stream);
      case 14: return launch_step_g<14, true>(s, a, split_sel, stream);
      case 15: return launch_step_g<15, true>(s, a, split_sel, stream);
      case 16: return launch_step_g<16, true>(s, a, split_sel, stream);
      default: return hipErrorInvalidValue;
    }
  }
  hipError_t e = launch_select(s, stream);
  if (e != hipSuccess) return e;
  return launch_sparse_attn(a, stream);
}

hipError_t launch_sparse_attn(const AttnArgs& a, hipStream_t stream) {
  if (a.kv_mode == 0 && attn_uses_tiles(a.group_size, a.n_q, a.q_pos0)) return launch_prefill_attn(a, stream);
  switch (a.group_size) {
    case 1: return launch_g<1>(a, stream);
    case 2: return launch_g<2>(a, stream);
    case 3: return launch_g<3>(a, stream);
    case 4: return launch_g<4>(a, stream);
    case 5: return launch_g<5>(a, stream);
    case 6: return launch_g<6>(a, stream);
    case 7: return launch_g<7>(a, stream);
    case 8: return launch_g<8>(a, stream);
    case 9: return launch_g<9>(a, stream);
    case 10: return launch_g<10>(a, stream);
    case 11: return launch_g<11>(a, stream);
    case 12: return launch_g<12>(a, stream);
    case 13: return launch_g<13>(a, stream);
    case 14: return launch_g<14>(a, stream);
    case 15: return launch_g<15>(a, stream);
    case 16: return launch_g<16>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sparda

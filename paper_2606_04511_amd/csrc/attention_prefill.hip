// attention_prefill.hip -- block-sparse attention for many query rows of one chunk (chunked
// prefill): paper Sec. 4.1, Eq. 5, over the per-row attended sets of Eq. 1 (Alg. 1 selects per
// query token, so neighbouring rows attend different blocks).
//
// Work unit: a tile of 128/G consecutive query rows of one (batch, group), i.e. 128 query-head
// rows, on one 256-thread workgroup; two workgroups share a CU, so a block's barrier waits for 4
// wavefronts while the other workgroup's wavefronts keep the SIMDs busy.  Wavefront w owns
// query-head rows [32 w, 32 w + 32): two MFMA N-tiles of 16 query-heads (16/G rows each), whose
// online-softmax state and output accumulators stay in registers for the whole tile.
//   1. Each row's attended blocks become a bitmap in LDS (entries outside [0, blk(p)] are
//      dropped; a block listed twice sets one bit, so it is attended once).  Their union, in
//      ascending order, is the tile's block list.  The bitmaps and the list are dynamic LDS
//      sized by the call's last row.
//   2. The tile walks its block list.  Block j's 16 KiB of K and 16 KiB of V are read from HBM
//      once per tile (16-byte loads, 1 KiB contiguous per wavefront instruction; every thread
//      loads four pieces of each) into a double-buffered LDS stage, one block ahead of the math.  K rows keep their 16-byte pieces
//      XOR-swizzled by the row; V is stored transposed (head dim x token, XOR-swizzled as well) so
//      that it can be the A operand of P V.  Both swizzles make the operand reads conflict-free
//      whether LDS serves 16 lanes of a 16-byte read from 64 banks or 32 lanes from 128.
//   3. A wavefront skips block j for an N-tile none of whose rows lists j.  Otherwise:
//        S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (M = 16 tokens, N = 16 query-heads, K = 32
//        dims); query-heads whose row does not list j, and tokens after the row's position, are
//        masked; online softmax in the exp2 domain;
//        O^T += V^T P^T on the same MFMA (M = 16 head dims, N = 16 query-heads, K = 32 tokens).
//      P needs no data movement between the two products: the staged V^T orders each 64-token
//      block as slots 4 tau + x <-> token tau + 16 x, which is exactly the token order in which
//      an S^T accumulator lane holds its 16 scores.
// Tiles with the most blocks run first; consecutive workgroups (spread over the XCDs by the
// dispatcher) take different groups, so each XCD's L2 serves one group's K and V.
#include <math.h>

#include "device_util.hpp"
#include "launch.hpp"

namespace sparda {

// The prefill attention's dynamic LDS (row bitmaps, union bitmap, union list).
extern __shared__ __align__(16) uint32_t pa_dyn[];

namespace {

constexpr int kPaThreads = 256;            // 4 wavefronts; two workgroups share a CU
constexpr int kPaQh = 128;                 // query-head rows per tile
constexpr int kPaKLd = kHeadDim;           // bf16 per staged K row; piece x of row r sits at x ^ (r % 16)
constexpr int kPaMaxBlocks = 4096;         // causal blocks a tile may span
constexpr int kPaStaticLds = 2 * 2 * kBlock * kHeadDim * 2 + 16;  // the K and V^T double buffers, n_union
constexpr int kPaLdsMax = 160 * 1024;      // LDS of one CU
constexpr float kLog2eP = 1.4426950408889634f;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const bf16x2 h = __builtin_convertvector(f32x2{lo, hi}, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

// Row bitmaps, union bitmap and union list live in dynamic LDS sized by the call (its last row's
// causal blocks): wc words per row bitmap.
__host__ __device__ inline int pa_dyn_lds_bytes(int rows, int nbt) {
  const int wc = (nbt + 31) >> 5;
  return ((4 * (rows * wc + wc) + 2 * nbt) + 15) & ~15;
}

template <int G>
__global__ __launch_bounds__(kPaThreads, 2) void prefill_attn_kernel(AttnArgs a, int n_tiles, int n_groups, int wc) {
  constexpr int TR = kPaQh / G;  // rows per tile
  constexpr int RN = 16 / G;     // rows per N-tile
  static_assert(16 % G == 0, "an N-tile holds whole rows");
  __shared__ __align__(16) uint16_t kst[2][kBlock * kPaKLd];
  __shared__ __align__(16) uint16_t vst[2][kHeadDim * kBlock];
  __shared__ int n_union;
  uint32_t* rbm = pa_dyn;                                   // [TR][wc] (a tile uses [nrows][W])
  uint32_t* ubm = pa_dyn + TR * wc;                         // [wc]
  int16_t* ulist = reinterpret_cast<int16_t*>(ubm + wc);    // [wc * 32] >= nbt

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t bm = blockIdx.x % n_groups;
  const int tile = n_tiles - 1 - (int)(blockIdx.x / n_groups);
  const int r0 = tile * TR;
  const int nrows = min(TR, a.n_q - r0);
  const int64_t p0 = a.q_pos0 + r0;
  const int nbt = (int)((p0 + nrows - 1) / kBlock) + 1;  // causal blocks of the tile's last row
  const int W = (nbt + 31) >> 5;                         // bitmap words per row

  // ---- 1. per-row bitmaps and their union
  for (int i = tid; i < nrows * W; i += kPaThreads) rbm[i] = 0u;
  for (int i = tid; i < W; i += kPaThreads) ubm[i] = 0u;
  __syncthreads();
  {
    const int kt = a.k_total;
    for (int e = tid; e < nrows * kt; e += kPaThreads) {
      const int rl = e / kt, s = e - rl * kt;
      const int64_t row = bm * a.n_q + r0 + rl;
      const int n = min(max((int)a.cnt[row], 0), kt);
      if (s < n) {
        const int j = a.sel[row * kt + s];
        const int blk = (int)((p0 + rl) / kBlock);
        if (j >= 0 && j <= blk) {
          atomicOr(&rbm[rl * W + (j >> 5)], 1u << (j & 31));
          atomicOr(&ubm[j >> 5], 1u << (j & 31));
        }
      }
    }
  }
  __syncthreads();
  if (wave == 0) {
    int base = 0;
    for (int w0 = 0; w0 < W; w0 += 64) {
      const int w = w0 + lane;
      uint32_t bits = w < W ? ubm[w] : 0u;
      const int c = __popc(bits);
      const int incl = wave_incl_scan(c);
      int pos = base + incl - c;
      while (bits) {
        ulist[pos++] = (int16_t)(w * 32 + __builtin_ctz(bits));
        bits &= bits - 1u;
      }
      base += readlane_i(incl, 63);
    }
    if (lane == 0) n_union = base;
  }

  // ---- per-lane query-head columns: lane (c, q) is column c of both N-tiles, k-chunk q
  const int c = lane & 15, q = lane >> 4;
  int rl_c[2];
  bool ok_c[2];
  int64_t pc[2];
  bf16x8 qf[2][4];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    rl_c[nt] = wave * (32 / G) + nt * RN + c / G;
    ok_c[nt] = rl_c[nt] < nrows;
    pc[nt] = p0 + rl_c[nt];
    const uint16_t* qrow = a.q + ((bm * G + c % G) * a.n_q + r0 + rl_c[nt]) * kHeadDim + 8 * q;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qf[nt][ks] = as_bf16x8(ok_c[nt] ? ld16(qrow + 32 * ks) : make_uint4(0u, 0u, 0u, 0u));
  }
  // z = zscale (q . k): a negative scale is folded into the query's sign bits (exact in bf16), so
  // that the block maximum of z is always zscale times the maximum of q . k.
  float zscale = a.sm_scale * kLog2eP;
  if (zscale < 0.f) {
    zscale = -zscale;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        uint4 w = __builtin_bit_cast(uint4, qf[nt][ks]);
        w.x ^= 0x80008000u;
        w.y ^= 0x80008000u;
        w.z ^= 0x80008000u;
        w.w ^= 0x80008000u;
        qf[nt][ks] = as_bf16x8(w);
      }
  }
  // Wait for the query fragments here, once: the loop's own loads are then the only ones in
  // flight, and the loop's waits can leave the prefetched blocks outstanding.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
  f32x4 acc[2][8];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int md = 0; md < 8; ++md) acc[nt][md] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ---- staging roles.  Every thread copies four 16-byte pieces of K and four of V per block.
  // K: token u/16, 16-byte part u%16 for u = tid + 256 x.  V: tokens tau + 16 x (x = 0..3), dims
  // 8 part .. 8 part + 7, with lane l of wavefront w taking tau = 4 w + l % 4, part = l / 4 (each
  // wavefront load instruction covers 4 whole token rows, 1 KiB contiguous).  One register set
  // holds the next block's loads while the current block is computed.
  //
  // Staged V^T: row d (head dim) holds the block's 64 tokens in slots 4 tau + x <-> token
  // tau + 16 x, 32 dwords per row; dword w of row d sits at w ^ vsw(d).  An operand read takes
  // 16 consecutive dims (16 md + c) x 4 k-chunks; vsw's low bits (from dim bits 1..3) give the
  // dims of one parity distinct dword pairs, so a half wavefront covers 64 banks of 64 and a whole
  // wavefront 128 of 128.  Its high bits (from dim bits 4, 5, constant over one read) spread the
  // transposing writes (once per block) to two lanes per bank, the least that 32 lanes of 8-byte
  // writes into one bank half can take.
  const int v_tau = 4 * (tid >> 6) + (tid & 3), v_part = (tid & 63) >> 2;
  const uint16_t* kp = a.k + bm * a.t_cap * kHeadDim + tid * 8;
  const uint16_t* vp = a.v + bm * a.t_cap * kHeadDim + v_tau * kHeadDim + 8 * v_part;
  auto vsw = [](int d) { return 2 * ((((d >> 2) & 3) | (((d >> 1) & 1) << 3)) ^ (((d >> 4) & 3) << 2)); };
  uint4 pre[8];  // K pieces 0..3, V pieces 4..7
  auto issue = [&](int j) {
    const int64_t off = (int64_t)j * kBlock * kHeadDim;
#pragma unroll
    for (int x = 0; x < 4; ++x) pre[x] = ld16(kp + off + x * 16 * kHeadDim);
#pragma unroll
    for (int x = 0; x < 4; ++x) pre[4 + x] = ld16(vp + off + x * 16 * kHeadDim);
  };
  auto stage = [&](int buf) {
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int u = tid + 256 * x;
      *reinterpret_cast<uint4*>(&kst[buf][(u >> 4) * kPaKLd + (((u & 15) ^ ((u >> 4) & 15)) * 8)]) = pre[x];
    }
    const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&pre[4]);
    const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&pre[5]);
    const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&pre[6]);
    const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&pre[7]);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int wi = i >> 1;
      uint2 d;
      if (i & 1) {
        d.x = (w0[wi] >> 16) | (w1[wi] & 0xffff0000u);
        d.y = (w2[wi] >> 16) | (w3[wi] & 0xffff0000u);
      } else {
        d.x = (w0[wi] & 0xffffu) | (w1[wi] << 16);
        d.y = (w2[wi] & 0xffffu) | (w3[wi] << 16);
      }
      const int dim = 8 * v_part + i;
      *reinterpret_cast<uint2*>(&vst[buf][2 * (dim * 32 + ((2 * v_tau) ^ vsw(dim)))]) = d;
    }
  };

  // Online softmax with a lazily raised reference: m_ref[nt] moves only when a block's maximum
  // exceeds it by more than kHeadroom (log2 units), so most blocks need no rescaling of acc.
  // P = 2^(z - m_ref) then stays below 2^kHeadroom, well inside bf16 and fp32; the final
  // normalisation by l, accumulated against the same reference, makes the result exact.
  constexpr float kHeadroom = 8.f;
  const int blk0 = (int)(p0 / kBlock);  // blocks >= blk0 may hold tokens after some row's position

  // the four lanes of a column (q = 0..3) exchange through lane ^ 16 and lane ^ 32
  const int addr32 = (lane ^ 32) << 2;
  auto xor16 = [](float x) {  // ds_swizzle, bit-mask mode: and 0x1f, xor 0x10 (within 32 lanes)
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x401F));
  };
  auto xor32 = [addr32](float x) { return __int_as_float(__builtin_amdgcn_ds_bpermute(addr32, __float_as_int(x))); };

  auto compute = [&](int j, int buf) {
    bool act[2], nt_act[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int rli = ok_c[nt] ? rl_c[nt] : 0;  // never index past the tile's bitmaps
      act[nt] = ok_c[nt] && ((rbm[rli * W + (j >> 5)] >> (j & 31)) & 1u);
      nt_act[nt] = __ballot(act[nt]) != 0ull;
    }
    if (!(nt_act[0] || nt_act[1])) return;
    // S^T[token 16 mt + 4 q + i][column c] for both N-tiles
    f32x4 st[2][4];
    const uint16_t* kb = &kst[buf][0];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      bf16x8 kf[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        kf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(kb + (16 * mt + c) * kPaKLd + (((4 * ks + q) ^ c) * 8)));
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        st[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (nt_act[nt]) {
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) st[nt][mt] = mfma16x16x32(kf[ks], qf[nt][ks], st[nt][mt]);
        }
      }
    }
    const bool diag = j >= blk0;  // uniform over the workgroup
    bf16x8 pb[2][2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      if (!nt_act[nt]) continue;
      // maximum over the visible scores: every token, except (in the tile's diagonal blocks)
      // those after the row's position
      int lim = kBlock - 1;
      float e = -INFINITY;
      if (diag) {
        const int64_t lim64 = pc[nt] - (int64_t)j * kBlock;
        lim = (int)(lim64 < kBlock ? lim64 : kBlock - 1);
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (16 * mt + 4 * q + i <= lim) e = fmaxf(e, st[nt][mt][i]);
      } else {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
          e = fmaxf(e, fmaxf(fmaxf(st[nt][mt][0], st[nt][mt][1]), fmaxf(st[nt][mt][2], st[nt][mt][3])));
      }
      float bmax = act[nt] ? e * zscale : -INFINITY;
      bmax = fmaxf(bmax, xor16(bmax));
      bmax = fmaxf(bmax, xor32(bmax));
      const bool raise = bmax > m_run[nt] + kHeadroom;  // also true on a column's first block
      if (__ballot(raise) != 0ull) {
        const float m_new = raise ? bmax : m_run[nt];
        const float alpha = raise ? __builtin_amdgcn_exp2f(m_run[nt] - m_new) : 1.f;
        m_run[nt] = m_new;
        l_run[nt] *= alpha;
#pragma unroll
        for (int md = 0; md < 8; ++md) acc[nt][md] *= alpha;
      }
      // z - m_ref as one FMA; an inactive column gets -inf, hence P = 0
      const float off = act[nt] ? -m_run[nt] : -INFINITY;
      float pz[4][4];
      float psum = 0.f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) pz[mt][i] = __builtin_amdgcn_exp2f(fmaf(st[nt][mt][i], zscale, off));
      if (diag) {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (16 * mt + 4 * q + i > lim) pz[mt][i] = 0.f;
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) psum += pz[mt][i];
      l_run[nt] += psum;
      // B operand of k-step s2: slot jj holds token 16 (jj % 4) + 4 q + 2 s2 + jj / 4
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        uint4 w;
        w.x = pack_bf16(pz[0][2 * s2], pz[1][2 * s2]);
        w.y = pack_bf16(pz[2][2 * s2], pz[3][2 * s2]);
        w.z = pack_bf16(pz[0][2 * s2 + 1], pz[1][2 * s2 + 1]);
        w.w = pack_bf16(pz[2][2 * s2 + 1], pz[3][2 * s2 + 1]);
        pb[nt][s2] = as_bf16x8(w);
      }
    }
    // O^T[dim 16 md + 4 q + i][column c] += V^T P^T
    const uint16_t* vb = &vst[buf][0];
#pragma unroll
    for (int md = 0; md < 8; ++md) {
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int dim = 16 * md + c, sw = vsw(dim), dw = 8 * q + 4 * s2;
        const uint2 v0 = *reinterpret_cast<const uint2*>(vb + 2 * (dim * 32 + (dw ^ sw)));
        const uint2 v1 = *reinterpret_cast<const uint2*>(vb + 2 * (dim * 32 + ((dw + 2) ^ sw)));
        const bf16x8 va = as_bf16x8(make_uint4(v0.x, v0.y, v1.x, v1.y));
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
          if (nt_act[nt]) acc[nt][md] = mfma16x16x32(va, pb[nt][s2], acc[nt][md]);
      }
    }
  };

  __syncthreads();  // union list and bitmaps complete
  const int nu = n_union;
  // Loads and stages run unconditionally (past the list's end they repeat its last block and
  // fill a buffer nobody reads), so that every path through the loop has the same loads in
  // flight and the compiler's waits only ever cover the block being staged.
  auto blk_at = [&](int i) { return (int)ulist[min(i, max(nu - 1, 0))]; };
  if (nu > 0) {
    issue(blk_at(0));
    stage(0);
  }
  __syncthreads();

  // Iteration it requests block it + 1, computes block it from buffer it % 2 meanwhile, then
  // stages block it + 1 into the other buffer.
  for (int it = 0; it < nu; ++it) {
    issue(blk_at(it + 1));
    compute(blk_at(it), it & 1);
    stage((it + 1) & 1);
    __syncthreads();
  }

  // ---- normalise and store: lane (c, q) holds dims 16 md + 4 q + i of its column
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    float l = l_run[nt];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const float inv = l > 0.f ? 1.f / l : 0.f;
    if (!ok_c[nt]) continue;
    uint16_t* orow = a.o + ((bm * G + c % G) * a.n_q + r0 + rl_c[nt]) * kHeadDim + 4 * q;
#pragma unroll
    for (int md = 0; md < 8; ++md) {
      const f32x4 v = acc[nt][md];
      uint2 w;
      w.x = (uint32_t)f32_to_bf16(v[0] * inv) | ((uint32_t)f32_to_bf16(v[1] * inv) << 16);
      w.y = (uint32_t)f32_to_bf16(v[2] * inv) | ((uint32_t)f32_to_bf16(v[3] * inv) << 16);
      *reinterpret_cast<uint2*>(orow + 16 * md) = w;
    }
  }
}

template <int G>
hipError_t launch_tiles(const AttnArgs& a, hipStream_t stream) {
  const int tr = kPaQh / G;
  const int n_tiles = (a.n_q + tr - 1) / tr;
  const int n_groups = a.batch * a.n_kv_heads;
  const int nbt = (int)((a.q_pos0 + a.n_q - 1) / kBlock) + 1;  // causal blocks of the call's last row
  hipLaunchKernelGGL(prefill_attn_kernel<G>, dim3((unsigned)((int64_t)n_groups * n_tiles)), dim3(kPaThreads),
                     pa_dyn_lds_bytes(tr, nbt), stream, a, n_tiles, n_groups, (nbt + 31) >> 5);
  return hipGetLastError();
}

}  // namespace

bool attn_uses_tiles(int32_t group_size, int32_t n_q, int64_t q_pos0) {
  if (n_q < 16 || group_size < 1 || group_size > 16 || 16 % group_size != 0) return false;
  const int64_t tr = kPaQh / group_size;
  // the call's last row decides the bitmap width; two workgroups share a CU while the dynamic
  // part stays within 16 KiB (contexts up to about 190K tokens at G = 4), one beyond
  const int64_t nbt = (q_pos0 + n_q - 1) / kBlock + 1;
  return nbt <= kPaMaxBlocks && kPaStaticLds + pa_dyn_lds_bytes((int)tr, (int)nbt) <= kPaLdsMax;
}

hipError_t launch_prefill_attn(const AttnArgs& a, hipStream_t stream) {
  switch (a.group_size) {
    case 1: return launch_tiles<1>(a, stream);
    case 2: return launch_tiles<2>(a, stream);
    case 4: return launch_tiles<4>(a, stream);
    case 8: return launch_tiles<8>(a, stream);
    case 16: return launch_tiles<16>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sparda

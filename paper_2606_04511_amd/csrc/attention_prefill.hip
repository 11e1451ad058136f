// attention_prefill.hip -- block-sparse attention for many query rows of one chunk (chunked
// prefill): paper Sec. 4.1, Eq. 5, over the per-row attended sets of Eq. 1 (Alg. 1 selects per
// query token, so neighbouring rows attend different blocks).
//
// Work unit: a tile of 256/G consecutive query rows of one (batch, group), i.e. 256 query-head
// rows, on one 512-thread workgroup.  Wavefront w owns query-head rows [32 w, 32 w + 32): two
// MFMA N-tiles of 16 query-heads (16/G rows each), whose online-softmax state and output
// accumulators stay in registers for the whole tile.
//   1. Each row's attended blocks become a bitmap in LDS (entries outside [0, blk(p)] are
//      dropped; a block listed twice sets one bit, so it is attended once).  Their union, in
//      ascending order, is the tile's block list.
//   2. The tile walks its block list.  Block j's 16 KiB of K and 16 KiB of V are read from HBM
//      once per tile (16-byte loads, 1 KiB contiguous per wavefront instruction) into a
//      double-buffered LDS stage, one block ahead of the math.  V is stored transposed (head dim
//      x token) so that it can be the A operand of the P V product.
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

namespace {

constexpr int kPaThreads = 512;
constexpr int kPaQh = 256;                 // query-head rows per tile
constexpr int kPaKLd = kHeadDim + 8;       // bf16 per staged K row (272 B: conflict-free 16-byte reads)
constexpr int kPaVLd = kBlock + 4;         // bf16 per staged V^T row (136 B: conflict-free 8-byte reads)
constexpr int kPaMaxWords = 8192;          // row-bitmap words (32 KiB)
constexpr int kPaMaxBlocks = 4096;         // causal blocks a tile may span
constexpr float kLog2eP = 1.4426950408889634f;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const bf16x2 h = __builtin_convertvector(f32x2{lo, hi}, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

template <int G>
__global__ __launch_bounds__(kPaThreads) void prefill_attn_kernel(AttnArgs a, int n_tiles, int n_groups) {
  constexpr int TR = kPaQh / G;  // rows per tile
  constexpr int RN = 16 / G;     // rows per N-tile
  static_assert(16 % G == 0, "an N-tile holds whole rows");
  __shared__ __align__(16) uint16_t kst[2][kBlock * kPaKLd];
  __shared__ __align__(16) uint16_t vst[2][kHeadDim * kPaVLd];
  __shared__ uint32_t rbm[kPaMaxWords];
  __shared__ uint32_t ubm[kPaMaxBlocks / 32];
  __shared__ int16_t ulist[kPaMaxBlocks];
  __shared__ int n_union;

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
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
  f32x4 acc[2][8];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int md = 0; md < 8; ++md) acc[nt][md] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float zscale = a.sm_scale * kLog2eP;

  // ---- staging roles: threads 0..255 copy K (token u/16, 16-byte part u%16 for u = lt + 256 x),
  // threads 256..511 copy V (tokens tau + 16 x, dims 8 part .. 8 part + 7; tau = lt/16).
  const int lt = tid & 255;
  const bool load_k = tid < 256;
  const uint16_t* kv = (load_k ? a.k : a.v) + bm * a.t_cap * kHeadDim;
  uint4 pre[4];
  auto issue = [&](int j) {
    const uint16_t* src = kv + (int64_t)j * kBlock * kHeadDim;
#pragma unroll
    for (int x = 0; x < 4; ++x) pre[x] = ld16(src + (lt + 256 * x) * 8);
  };
  auto stage = [&](int buf) {
    if (load_k) {
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int u = lt + 256 * x;
        *reinterpret_cast<uint4*>(&kst[buf][(u >> 4) * kPaKLd + (u & 15) * 8]) = pre[x];
      }
    } else {
      const int tau = lt >> 4, part = lt & 15;
      const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&pre[0]);
      const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&pre[1]);
      const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&pre[2]);
      const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&pre[3]);
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
        *reinterpret_cast<uint2*>(&vst[buf][(8 * part + i) * kPaVLd + 4 * tau]) = d;
      }
    }
  };

  __syncthreads();  // union list and bitmaps complete
  const int nu = n_union;
  if (nu > 0) {
    issue(ulist[0]);
    stage(0);
  }
  __syncthreads();

  for (int it = 0; it < nu; ++it) {
    const int buf = it & 1;
    const int j = ulist[it];
    if (it + 1 < nu) issue(ulist[it + 1]);

    bool act[2], nt_act[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int rli = ok_c[nt] ? rl_c[nt] : 0;  // never index past the tile's bitmaps
      act[nt] = ok_c[nt] && ((rbm[rli * W + (j >> 5)] >> (j & 31)) & 1u);
      nt_act[nt] = __ballot(act[nt]) != 0ull;
    }
    if (nt_act[0] || nt_act[1]) {
      // S^T[token 16 mt + 4 q + i][column c] for both N-tiles
      f32x4 st[2][4];
      const uint16_t* kb = &kst[buf][0];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        bf16x8 kf[4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
          kf[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(kb + (16 * mt + c) * kPaKLd + 32 * ks + 8 * q));
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          st[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (nt_act[nt]) {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) st[nt][mt] = mfma16x16x32(kf[ks], qf[nt][ks], st[nt][mt]);
          }
        }
      }
      bf16x8 pb[2][2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        if (!nt_act[nt]) continue;
        // last visible token of block j for this column (-1: the row does not list j)
        const int64_t lim64 = pc[nt] - (int64_t)j * kBlock;
        const int lim = act[nt] ? (int)(lim64 < kBlock ? lim64 : kBlock - 1) : -1;
        float z[4][4];
        float bmax = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int tok = 16 * mt + 4 * q + i;
            z[mt][i] = tok <= lim ? st[nt][mt][i] * zscale : -INFINITY;
            bmax = fmaxf(bmax, z[mt][i]);
          }
        bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
        bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
        const float m_new = fmaxf(m_run[nt], bmax);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m_run[nt] - m_use);
        float psum = 0.f;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            z[mt][i] = exp2f(z[mt][i] - m_use);
            psum += z[mt][i];
          }
        l_run[nt] = l_run[nt] * alpha + psum;
        m_run[nt] = m_new;
#pragma unroll
        for (int md = 0; md < 8; ++md) acc[nt][md] *= alpha;
        // B operand of k-step s2: slot jj holds token 16 (jj % 4) + 4 q + 2 s2 + jj / 4
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          uint4 w;
          w.x = pack_bf16(z[0][2 * s2], z[1][2 * s2]);
          w.y = pack_bf16(z[2][2 * s2], z[3][2 * s2]);
          w.z = pack_bf16(z[0][2 * s2 + 1], z[1][2 * s2 + 1]);
          w.w = pack_bf16(z[2][2 * s2 + 1], z[3][2 * s2 + 1]);
          pb[nt][s2] = as_bf16x8(w);
        }
      }
      // O^T[dim 16 md + 4 q + i][column c] += V^T P^T
      const uint16_t* vb = &vst[buf][0];
#pragma unroll
      for (int md = 0; md < 8; ++md) {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const uint16_t* src = vb + (16 * md + c) * kPaVLd + 16 * q + 8 * s2;
          const uint2 v0 = *reinterpret_cast<const uint2*>(src);
          const uint2 v1 = *reinterpret_cast<const uint2*>(src + 4);
          const bf16x8 va = as_bf16x8(make_uint4(v0.x, v0.y, v1.x, v1.y));
#pragma unroll
          for (int nt = 0; nt < 2; ++nt)
            if (nt_act[nt]) acc[nt][md] = mfma16x16x32(va, pb[nt][s2], acc[nt][md]);
        }
      }
    }
    if (it + 1 < nu) stage(buf ^ 1);
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
  hipLaunchKernelGGL(prefill_attn_kernel<G>, dim3((unsigned)((int64_t)n_groups * n_tiles)), dim3(kPaThreads), 0,
                     stream, a, n_tiles, n_groups);
  return hipGetLastError();
}

}  // namespace

bool attn_uses_tiles(int32_t group_size, int32_t n_q, int64_t q_pos0) {
  if (n_q < 16 || group_size < 1 || group_size > 16 || 16 % group_size != 0) return false;
  const int64_t tr = kPaQh / group_size;
  // the widest tile: its last row decides the bitmap width
  const int64_t rows = n_q < tr ? n_q : tr;
  const int64_t nbt = (q_pos0 + n_q - 1) / kBlock + 1;
  const int64_t words = (nbt + 31) / 32;
  return nbt <= kPaMaxBlocks && rows * words <= kPaMaxWords;
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

// indexer_kl.hip -- the indexer-training loss of Sec. 4.2 (Eq. 6-7) and its gradient with respect
// to the Forecast rows, on synthetic tensors (the Forecast projection's own weight gradient is a
// plain GEMM of this gradient with the layer input, outside this file).
//
// Per query row at position p of group m (G query heads):
//   target     each head's softmax of sm_scale q_h . K~t_i over the fine (2, 1) windows complete at
//              p (window i = mean of keys i, i + 1), summed over the group; T_w = the largest such
//              sum over the fine windows lying inside position w of the prediction grid
//              ((32, 16): tokens [16 w, 16 w + 32)).
//   predicted  P = softmax over the positions complete at p of sm_scale F . K~p_w.
//   selected   S = the k_top largest T_w (ties: lower w) among positions inside candidate blocks.
//   loss       KL of the (k+1)-bucket partitions: t_c = T_c / sum T for c in S plus the rest bucket,
//              against P_c and R = sum of P outside S.
//   gradient   dL/dz_w = P_w - t_w in S, P_w (1 - t_rest / R) outside; dF = sm_scale sum_w dz_w K~p_w.
//
// Kernels:
//   pair_compress_kernel -- the (2, 1) windows of the raw keys into the workspace: float64 sum of
//                           the pair, one rounding to bf16 (as every compressed key).
//   kl_target_kernel     -- for G in {1, 2, 4, 8, 16}: the target's shared weight of every fine
//                           window for 64 / G rows at a time (64 (row, head) columns on 32x32x16
//                           MFMA, head_tiles.hpp), into the workspace, so that every fine key
//                           fragment serves 64 / G rows.
//   kl_row_kernel        -- one 512-thread workgroup per query row.  Target: the max-pool of those
//                           weights into the positions, or for other G 16-window x 16-head
//                           MFMA tiles (A = the windows, B = the group's query rows padded to 16
//                           columns), an online maximum and sum of 2^z per head, then a second
//                           pass that sums each window's normalised head weights across the
//                           columns and max-pools it into its positions in LDS (atomic max on the
//                           float bits: all values are >= 0).  Prediction: the Forecast GEMV over
//                           the positions into LDS and its softmax.  Selection: the block-wide
//                           top-k of select_block.hpp over the candidate positions.  Then
//                           the bucket sums, the loss and the gradient GEMV.
#include <math.h>

#include "device_util.hpp"
#include "launch.hpp"
#include "head_tiles.hpp"
#include "select_block.hpp"

namespace sparda {

// Limits (checked by the entry point): 16384 positions per row and k_top <= 4096, so that the row
// kernel's per-position LDS arrays (9 bytes per position plus 2 per top-k entry) fit one CU.

__global__ __launch_bounds__(256) void pair_compress_kernel(const uint16_t* __restrict__ k, uint16_t* __restrict__ kt,
                                                            int64_t t_cap, int64_t n_win, int64_t rows) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (row, window, 16-byte chunk)
  const int64_t total = rows * n_win * 16;
  if (idx >= total) return;
  const int c = (int)(idx & 15);
  const int64_t rw = idx >> 4;
  const int64_t row = rw / n_win, i = rw - row * n_win;
  const uint16_t* src = k + (row * t_cap + i) * kHeadDim + 8 * c;
  const uint4 a = ld16(src), b = ld16(src + kHeadDim);
  const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
  uint32_t o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const double lo = ((double)bf16lo(aw[e]) + (double)bf16lo(bw[e])) * 0.5;  // exact, then one rounding
    const double hi = ((double)bf16hi(aw[e]) + (double)bf16hi(bw[e])) * 0.5;
    o[e] = (uint32_t)f64_to_bf16(lo) | ((uint32_t)f64_to_bf16(hi) << 16);
  }
  *reinterpret_cast<uint4*>(kt + (row * n_win + i) * kHeadDim + 8 * c) = make_uint4(o[0], o[1], o[2], o[3]);
}

struct KlArgs {
  const uint16_t* q;      // [B][Hq][n_q][D]
  const uint16_t* kt;     // [B][Hkv][nt][D] fine windows (workspace)
  const uint16_t* f;      // [B][Hkv][n_q][D]
  const uint16_t* kp;     // [B][Hkv][nc_cap][D] prediction windows
  float* loss;            // [B][Hkv][n_q]
  float* dF;              // [B][Hkv][n_q][D]
  float* sw;              // [B][Hkv][n_q][sw_stride] shared target weights per fine window (workspace)
  int64_t sw_stride;
  int32_t lds_pos, lds_top;  // per-position LDS entries (>= 512, a multiple of 16) and top-k list entries
  int64_t nt, nc_cap, q_pos0;
  int32_t n_kv_heads, group_size, n_q, n_init, n_local, k_top;
  WinGrid grid;           // prediction grid
  float scale_log2;       // sm_scale * log2(e)
  float sm_scale;
};

__device__ __forceinline__ float block_sum_f(float x, float* red, int wave, int lane) {
  x = row16_sum(x);
  x += __shfl_xor(x, 16, kWave);
  x += __shfl_xor(x, 32, kWave);
  __syncthreads();
  if (lane == 0) red[wave] = x;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < kDecThreads / 64; ++w) s += red[w];
  return s;
}

__device__ __forceinline__ float block_max_f(float x, float* red, int wave, int lane) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x = fmaxf(x, __shfl_xor(x, d, kWave));
  __syncthreads();
  if (lane == 0) red[wave] = x;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int w = 1; w < kDecThreads / 64; ++w) m = fmaxf(m, red[w]);
  return m;
}

// The target's shared weights of many rows on MFMA (G in {1, 2, 4, 8, 16}): a unit is 64 / G rows
// of one (batch, group) with their heads (head_tiles.hpp), scored against the fine windows
// complete at the unit's last row; each row stores its weights of the fine windows 0 .. p - 1.
template <int G>
__global__ __launch_bounds__(kMtThreads) void kl_target_kernel(KlArgs a, int n_units) {
  constexpr int U = 64 / G;
  __shared__ float red_m[kMtWaves][64], red_s[kMtWaves][64];
  const int n = threadIdx.x & 31;
  const int n_groups = (int)(gridDim.x / n_units);
  const int grp = blockIdx.x % n_groups;
  const int unit = n_units - 1 - (int)(blockIdx.x / n_groups);  // latest rows (most windows) first
  const int r0 = unit * U;
  const int nr = min(U, a.n_q - r0);
  HeadTileRows t;
  t.n_keys = (int)(a.q_pos0 + r0 + nr - 1);  // fine windows 0 .. p - 1 of the unit's last row
  t.lo = 0;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int c = 32 * nt + n;
    const int rr = min(c / G, nr - 1);
    const int64_t p = a.q_pos0 + r0 + rr;
    t.q[nt] = reinterpret_cast<const uint4*>(a.q) + (((int64_t)grp * G + c % G) * a.n_q + r0 + rr) * kMtRowU4;
    t.vis[nt] = (int)p - 1;
    t.hi[nt] = ((n % G) == 0 && c / G < nr) ? (int)p - 1 : -1;
    t.out[nt] = a.sw + ((int64_t)grp * a.n_q + r0 + rr) * a.sw_stride;
  }
  head_tile_shared_weights<G>(t, reinterpret_cast<const uint4*>(a.kt) + (int64_t)grp * a.nt * kMtRowU4,
                              a.scale_log2, red_m, red_s);
}

// kPre: the target's shared weights are in a.sw (kl_target_kernel); the row max-pools them into
// its positions.  Otherwise the row computes them itself (16-window x 16-column MFMA tiles).
template <bool kPre>
__global__ __launch_bounds__(kDecThreads) void kl_row_kernel(KlArgs a) {
  // Per-position arrays, sized by the host for the call's largest row (kl_lds_layout): the pooled
  // target (float bits for the atomic max), the predicted distribution, the top-k list and the
  // chosen flags.  A small footprint lets several rows share a CU.
  extern __shared__ __align__(16) float kl_lds[];
  float* Tp = kl_lds;
  float* Pp = kl_lds + a.lds_pos;
  int16_t* idx = reinterpret_cast<int16_t*>(Pp + a.lds_pos);
  uint8_t* chosen = reinterpret_cast<uint8_t*>(idx + a.lds_top);
  __shared__ __align__(16) uint32_t hist[kTopkLds];
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  __shared__ float red[kDecThreads / 64];
  __shared__ float red_m[kDecThreads / 64][16], red_s[kDecThreads / 64][16];
  const int64_t row = blockIdx.x;  // (b * Hkv + m) * n_q + r
  const int r = (int)(row % a.n_q);
  const int64_t bm = row / a.n_q;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, j = lane >> 4;
  const int G = a.group_size;
  const int64_t p = a.q_pos0 + r;
  const int N = grid_win_vis(a.grid, p) + 1;           // positions 0 .. N - 1 (host-checked)
  const int n_tw = (int)p;                              // fine windows 0 .. p - 1 are complete at p
  for (int w = tid; w < N; w += kDecThreads) {
    Tp[w] = 0.f;
    chosen[w] = 0;
  }
  __syncthreads();

  // ---- target
  if (kPre) {
    // T_w = the largest shared weight among the fine windows inside position w: tokens [i, i + 2)
    // within [w s, w s + l), i.e. i in [w s, w s + l - 2]; every position complete at p has them
    const float* srow = a.sw + row * a.sw_stride;
    const int gl = a.grid.l, gs = a.grid.s;
    for (int w = tid; w < N; w += kDecThreads) {
      const int i0 = w * gs, i1 = min(w * gs + gl - 2, n_tw - 1);
      float m = 0.f;
      for (int i = i0; i <= i1; ++i) m = fmaxf(m, srow[i]);
      Tp[w] = m;
    }
  } else {  // MFMA tiles of 16 fine windows x the group's heads
    bf16x8 qb[4];
    // columns past the group's heads read head 0 (a valid address) and are zeroed
    const uint16_t* qrow = a.q + ((bm * G + (n < G ? n : 0)) * a.n_q + r) * kHeadDim + 8 * j;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 v = ld16(qrow + 32 * ks);
      qb[ks] = as_bf16x8(n < G ? v : make_uint4(0u, 0u, 0u, 0u));
    }
    const uint16_t* kb = a.kt + bm * a.nt * kHeadDim + 8 * j;
    const int n_tiles = (n_tw + 15) >> 4;
    auto score = [&](int t, float (&z)[4]) {
      const int win = min(16 * t + n, n_tw - 1);
      uint4 w[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) w[ks] = ld16(kb + (int64_t)win * kHeadDim + 32 * ks);
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) c = mfma16x16x32(as_bf16x8(w[ks]), qb[ks], c);
#pragma unroll
      for (int e = 0; e < 4; ++e) z[e] = 16 * t + 4 * j + e < n_tw ? c[e] * a.scale_log2 : -INFINITY;
    };
    float m_run = -INFINITY, s_run = 0.f;
    for (int t = wave; t < n_tiles; t += kDecThreads / 64) {
      float z[4];
      score(t, z);
      const float mn = fmaxf(m_run, fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3])));
      if (mn > -INFINITY) {
        s_run = s_run * exp2f(m_run - mn) + exp2f(z[0] - mn) + exp2f(z[1] - mn) + exp2f(z[2] - mn) + exp2f(z[3] - mn);
        m_run = mn;
      }
    }
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
    const float inv = n < G ? 1.0f / S : 0.f;
    const int gl = a.grid.l, gs = a.grid.s;
    for (int t = wave; t < n_tiles; t += kDecThreads / 64) {
      float z[4];
      score(t, z);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float sh = row16_sum(n < G ? exp2f(z[e] - M) * inv : 0.f);
        const int i = 16 * t + 4 * j + e;
        if (n == e && i < n_tw) {
          // positions w with w s <= i and i + 2 <= w s + l
          const int w_hi = min(i / gs, N - 1);
          const int num = i + 2 - gl;
          const int w_lo = num <= 0 ? 0 : (num + gs - 1) / gs;
          for (int w = w_lo; w <= w_hi; ++w) atomicMax(reinterpret_cast<unsigned int*>(&Tp[w]), __float_as_uint(sh));
        }
      }
    }
  }
  __syncthreads();

  // ---- prediction: Forecast GEMV over the positions (16 lanes per position), then its softmax
  {
    const int c = lane & 15, rs = lane >> 4;
    float fv[8];
    {
      const uint4 w = ld16(a.f + (bm * a.n_q + r) * kHeadDim + 8 * c);
      fv[0] = bf16lo(w.x) * a.scale_log2; fv[1] = bf16hi(w.x) * a.scale_log2;
      fv[2] = bf16lo(w.y) * a.scale_log2; fv[3] = bf16hi(w.y) * a.scale_log2;
      fv[4] = bf16lo(w.z) * a.scale_log2; fv[5] = bf16hi(w.z) * a.scale_log2;
      fv[6] = bf16lo(w.w) * a.scale_log2; fv[7] = bf16hi(w.w) * a.scale_log2;
    }
    const uint16_t* kpb = a.kp + bm * a.nc_cap * kHeadDim + 8 * c;
    for (int base = wave * 4; base < N; base += (kDecThreads / 64) * 4) {
      const int w = base + rs;
      const uint4 k = ld16(kpb + (int64_t)min(w, N - 1) * kHeadDim);
      float d = fv[0] * bf16lo(k.x);
      d = fmaf(fv[1], bf16hi(k.x), d);
      d = fmaf(fv[2], bf16lo(k.y), d);
      d = fmaf(fv[3], bf16hi(k.y), d);
      d = fmaf(fv[4], bf16lo(k.z), d);
      d = fmaf(fv[5], bf16hi(k.z), d);
      d = fmaf(fv[6], bf16lo(k.w), d);
      d = fmaf(fv[7], bf16hi(k.w), d);
      d = row16_sum(d);
      if (c == 0 && w < N) Pp[w] = d;
    }
  }
  __syncthreads();
  float zl = -INFINITY;
  for (int w = tid; w < N; w += kDecThreads) zl = fmaxf(zl, Pp[w]);
  const float zmax = block_max_f(zl, red, wave, lane);
  float el = 0.f;
  for (int w = tid; w < N; w += kDecThreads) {
    const float e = exp2f(Pp[w] - zmax);
    Pp[w] = e;
    el += e;
  }
  const float pinv = 1.0f / block_sum_f(el, red, wave, lane);
  for (int w = tid; w < N; w += kDecThreads) Pp[w] *= pinv;

  // ---- the target's top-k among positions inside candidate blocks [n_init, blk(p) - n_local]
  const int blk = (int)(p / kBlock);
  const int tok_lo = a.n_init * kBlock, tok_hi = (blk - a.n_local + 1) * kBlock;
  const int c_lo = (tok_lo + a.grid.s - 1) / a.grid.s;
  const int c_hi = min(N - 1, tok_hi - a.grid.l >= 0 ? (tok_hi - a.grid.l) / a.grid.s : -1);
  const int C = c_hi >= c_lo ? c_hi - c_lo + 1 : 0;
  const int n_take = min(a.k_top, C);
  __syncthreads();
  if (n_take >= C) {
    for (int i = tid; i < C; i += kDecThreads) chosen[c_lo + i] = 1;
  } else if (n_take > 0) {
    block_topk_emit(Tp + c_lo, C, n_take, c_lo, idx, hist, wave_cnt, pick);
    __syncthreads();
    for (int i = tid; i < n_take; i += kDecThreads) chosen[idx[i]] = 1;
  }
  __syncthreads();

  // ---- buckets and loss
  float tt = 0.f, tr = 0.f, pr = 0.f;
  for (int w = tid; w < N; w += kDecThreads) {
    tt += Tp[w];
    if (!chosen[w]) {
      tr += Tp[w];
      pr += Pp[w];
    }
  }
  const float Ttot = block_sum_f(tt, red, wave, lane);
  const float Trest = block_sum_f(tr, red, wave, lane);
  const float R = block_sum_f(pr, red, wave, lane);
  const float tinv = 1.0f / Ttot;
  const float t_rest = Trest / Ttot;
  float kl = 0.f;
  for (int w = tid; w < N; w += kDecThreads) {
    if (chosen[w]) {
      const float tc = Tp[w] * tinv;
      if (tc > 0.f) kl += tc * __logf(tc / Pp[w]);
    }
  }
  kl = block_sum_f(kl, red, wave, lane);
  if (tid == 0) a.loss[row] = kl + (t_rest > 0.f ? t_rest * __logf(t_rest / R) : 0.f);

  // ---- gradient: dF[d] = sm_scale sum_w g_w K~p_w[d]; thread (grp, d): positions w = grp mod 4
  const float rest_f = R > 0.f ? 1.0f - t_rest / R : 0.f;
  {
    const int d = tid & 127, grp = tid >> 7;
    const uint16_t* kpb = a.kp + bm * a.nc_cap * kHeadDim + d;
    float acc = 0.f;
    for (int w = grp; w < N; w += 4) {
      const float g = chosen[w] ? Pp[w] - Tp[w] * tinv : Pp[w] * rest_f;
      const uint16_t kv = kpb[(int64_t)w * kHeadDim];
      acc = fmaf(g, __uint_as_float((uint32_t)kv << 16), acc);
    }
    __syncthreads();
    Tp[tid] = acc;  // the target scores are no longer needed
    __syncthreads();
    if (tid < 128) a.dF[row * kHeadDim + tid] = a.sm_scale * (Tp[tid] + Tp[tid + 128] + Tp[tid + 256] + Tp[tid + 384]);
  }
}

hipError_t launch_indexer_kl(const uint16_t* q, const uint16_t* k, const uint16_t* f, const uint16_t* kp,
                             uint16_t* kt_ws, float* sw_ws, float* loss, float* dF, int32_t batch, int32_t n_kv_heads,
                             int32_t group_size, int32_t n_q, int64_t q_pos0, int64_t t_cap, int64_t nc_cap,
                             int32_t n_init, int32_t n_local, int32_t k_top, WinGrid grid, float sm_scale,
                             hipStream_t stream) {
  const int64_t rows_g = (int64_t)batch * n_kv_heads;
  const int64_t nt = q_pos0 + n_q - 1;  // fine windows complete at the last row: 0 .. p - 1
  if (nt > 0) {
    const int64_t total = rows_g * nt * 16;
    hipLaunchKernelGGL(pair_compress_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, k, kt_ws,
                       t_cap, nt, rows_g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  KlArgs a;
  a.q = q;
  a.kt = kt_ws;
  a.f = f;
  a.kp = kp;
  a.loss = loss;
  a.dF = dF;
  a.nt = nt > 0 ? nt : 1;
  a.nc_cap = nc_cap;
  a.q_pos0 = q_pos0;
  a.n_kv_heads = n_kv_heads;
  a.group_size = group_size;
  a.n_q = n_q;
  a.n_init = n_init;
  a.n_local = n_local;
  a.k_top = k_top;
  a.grid = grid;
  a.sm_scale = sm_scale;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.sw = sw_ws;
  a.sw_stride = (a.nt + 3) & ~(int64_t)3;
  // the last row has the most positions; the gradient's reduction reuses 512 entries of Tp
  const int n_max = grid_win_vis(grid, q_pos0 + n_q - 1) + 1;
  a.lds_pos = n_max > 512 ? (n_max + 15) & ~15 : 512;
  a.lds_top = ((k_top < n_max ? k_top : n_max) + 8) & ~7;
  const size_t lds = (size_t)a.lds_pos * 2 * sizeof(float) + (size_t)a.lds_top * sizeof(int16_t) + (size_t)a.lds_pos;
  const int G = group_size;
  if (G == 1 || G == 2 || G == 4 || G == 8 || G == 16) {  // the target of 64 / G rows per MFMA unit
    const int n_units = (n_q + 64 / G - 1) / (64 / G);
    const dim3 grid((unsigned)(rows_g * n_units)), block(kMtThreads);
    switch (G) {
      case 1: hipLaunchKernelGGL(kl_target_kernel<1>, grid, block, 0, stream, a, n_units); break;
      case 2: hipLaunchKernelGGL(kl_target_kernel<2>, grid, block, 0, stream, a, n_units); break;
      case 4: hipLaunchKernelGGL(kl_target_kernel<4>, grid, block, 0, stream, a, n_units); break;
      case 8: hipLaunchKernelGGL(kl_target_kernel<8>, grid, block, 0, stream, a, n_units); break;
      default: hipLaunchKernelGGL(kl_target_kernel<16>, grid, block, 0, stream, a, n_units); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kl_row_kernel<true>, dim3((unsigned)(rows_g * n_q)), dim3(kDecThreads), lds, stream, a);
  } else {
    hipLaunchKernelGGL(kl_row_kernel<false>, dim3((unsigned)(rows_g * n_q)), dim3(kDecThreads), lds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace sparda

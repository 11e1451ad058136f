// select.hip -- Forecast scoring and top-k block selection (paper Sec. 4.1, Eq. 4, with the
// attended-set union of Eq. 1).
//
// Per query row at position p: forced = initial blocks U local window, candidates = the complete
// blocks in between, window scores F_row . K~_i (one Forecast head per GQA group, no softmax, no
// scale, float32 accumulation), block score s_j = the max over the windows that overlap block j
// and are complete at p (the identity for the one-key-per-block grid); the k_total - |forced|
// best candidates by (score desc, index asc) join the forced blocks; the row's set is written in
// ascending block order, -1 padded.
//
// Two paths:
//  * row-wise (decode, n_q == 1, and long multi-row cases): a bandwidth-bound GEMV kernel writes
//    the candidate scores of each row to a float32 scratch row; a second kernel runs one
//    wavefront per row that finds the exact k-th key by an 8-bit-digit radix select over a
//    wave-private LDS histogram and emits the chosen indices in ascending order with ballots.
//  * fused decode (one row per (batch, group), <= 16384 candidates): one workgroup per row keeps
//    the row's scores in LDS and runs the block-wide top-k there (select_block.hpp).
//  * fused tile (multi-row prefill with <= 512 candidates per 64-row tile): select_prefill.hip.
#include "device_util.hpp"
#include "launch.hpp"
#include "select_block.hpp"

namespace sparda {

// ---- row-wise path ----------------------------------------------------------------------

// grid.x = row * n_chunks + chunk; a chunk is 256 windows (64 per wavefront).  Lane l reads dims
// 8*(l%16)..+7 of window 4 i + l/16: each wavefront load is 1 KiB contiguous of K~.  Window
// first + x of the row goes to scratch slot x.
__global__ __launch_bounds__(256) void rowwise_score_kernel(SelectArgs a, int n_chunks) {
  const int64_t row = blockIdx.x / n_chunks;
  const int chunk = (int)(blockIdx.x % n_chunks);
  const int r = (int)(row % a.n_q);
  const int64_t bm = row / a.n_q;
  const int64_t p = a.q_pos0 + r;
  const RowGeom g = row_geom(p, a.n_init, a.n_local, a.k_total);
  if (g.n_take >= g.n_cand) return;
  int32_t wf, wl;
  row_windows(g, a.grid, p, &wf, &wl);
  const int nw = wl - wf + 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, rs = lane >> 4;
  const int first = chunk * 256 + wave * 64;
  if (first >= nw) return;
  const uint4 fw = ld16(a.f + row * kHeadDim + c * 8);
  const float f0 = bf16lo(fw.x), f1 = bf16hi(fw.x), f2 = bf16lo(fw.y), f3 = bf16hi(fw.y);
  const float f4 = bf16lo(fw.z), f5 = bf16hi(fw.z), f6 = bf16lo(fw.w), f7 = bf16hi(fw.w);
  const uint16_t* kbase = a.kc + (bm * a.nc_cap + wf) * kHeadDim + c * 8;
  uint4 kw[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int idx = min(first + 4 * i + rs, nw - 1);  // past the last window: a repeat, never stored
    kw[i] = ld16(kbase + (int64_t)idx * kHeadDim);
  }
  float* out = a.ws + row * a.ws_stride;
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
    const int idx = first + 4 * i + rs;
    if (c == 0 && idx < nw) out[idx] = d;
  }
}


// Rows with at most this many candidates keep their pooled block keys in LDS for the radix passes
// (8 KiB per wavefront); longer rows pool from the workspace on every pass.
constexpr int kRowTopkLdsKeys = 2048;

// One wavefront per row: forced blocks, padding, count, and the radix top-k over the scratch row.
__global__ __launch_bounds__(256) void rowwise_topk_kernel(SelectArgs a, int64_t n_rows) {
  __shared__ __align__(16) uint32_t hist[4][256];
  __shared__ uint32_t keys[4][kRowTopkLdsKeys];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= n_rows) return;
  const int r = (int)(row % a.n_q);
  const RowGeom g = row_geom(a.q_pos0 + r, a.n_init, a.n_local, a.k_total);
  int16_t* out = a.sel + row * a.k_total;
  emit_forced(out, g, a.k_total, lane);
  if (lane == 0) a.cnt[row] = (int16_t)(g.n_forced + g.n_take);
  const float* sc = a.ws + row * a.ws_stride;
  const int64_t p = a.q_pos0 + r;
  int32_t wf, wl;
  row_windows(g, a.grid, p, &wf, &wl);
  const int32_t wvis = grid_win_vis(a.grid, p);
  const WinGrid grid = a.grid;
  if (g.n_take < g.n_cand && g.n_cand <= kRowTopkLdsKeys) {
    // pool once: the passes and the emission then read LDS instead of the workspace
    uint32_t* kw = keys[wave];
#pragma unroll 4
    for (int i = lane; i < g.n_cand; i += kWave) kw[i] = score_key(pooled_score(sc, grid, g.cand_lo + i, wf, wvis));
    wave_lds_sync();
    wave_topk_emit([&](int i) { return kw[i]; }, g.n_cand, g.n_take, g.cand_lo, hist[wave], out + g.init_hi);
    return;
  }
  wave_topk_emit([&](int i) { return score_key(pooled_score(sc, grid, g.cand_lo + i, wf, wvis)); }, g.n_cand,
                 g.n_take, g.cand_lo, hist[wave], out + g.init_hi);
}

// ---- fused decode path ---------------------------------------------------------------------

// One workgroup per decode row (batch, group): the Forecast GEMV over all scored windows into LDS,
// the max-pool of window scores to block scores (skipped for the one-key-per-block grid), then
// the block-wide top-k (value bins, the threshold bin ranked exactly) and an ordered emission.
// Scores never leave the CU.
__global__ __launch_bounds__(kDecThreads) void decode_select_kernel(SelectArgs a) {
  __shared__ float sc[kDecodeMaxCand];
  __shared__ __align__(16) uint32_t hist[kTopkLds];
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  const int64_t row = blockIdx.x;
  decode_select_row(a, row, sc, hist, wave_cnt, pick, a.sel + row * a.k_total, a.cnt + row);
}

// Decode rows with their window scores already in the workspace (row stride ws_stride, window
// wf of the row at offset 0): one workgroup per row loads them into LDS, max-pools them to block
// scores and runs the block-wide top-k.  The second kernel of the split decode path.
__global__ __launch_bounds__(kDecThreads) void decode_topk_kernel(SelectArgs a) {
  __shared__ float sc[kDecodeMaxCand];
  __shared__ __align__(16) uint32_t hist[kTopkLds];
  __shared__ int wave_cnt[kDecThreads / 64];
  __shared__ int pick[3];
  const int64_t row = blockIdx.x;
  decode_topk_row(a, row, sc, hist, wave_cnt, pick, a.sel + row * a.k_total, a.cnt + row);
}

// Which kernels serve a select call.
enum SelectPath { kPathDecode, kPathDecodeSplit, kPathTile, kPathRowwise };

// Decode calls with fewer rows than CUs score each row with many workgroups (the row-wise score
// kernel, 256 windows each) and select with one workgroup per row; otherwise one fused workgroup
// per row.
constexpr int64_t kDecodeSplitRows = 256;
// Multi-row calls on the row-wise path with at least this many rows score on MFMA.
constexpr int32_t kTileScoreMinRows = 16;

static SelectPath select_path(int64_t rows, int32_t n_q, int64_t q_pos0, int32_t n_init, int32_t n_local,
                              WinGrid grid) {
  const int64_t p = q_pos0 + n_q - 1;
  const RowGeom g = row_geom(p, n_init, n_local, 1 << 30);
  int32_t wf, wl;
  row_windows(g, grid, p, &wf, &wl);
  const int64_t nw = wl >= wf ? wl - wf + 1 : 0;
  if (n_q == 1) {  // window scores and (for a windowed grid) block scores share the LDS score array
    const int64_t need = grid_is_blocks(grid) ? g.n_cand : nw + g.n_cand;
    if (need > kDecodeMaxCand) return kPathRowwise;
    return rows < kDecodeSplitRows && nw >= 1024 ? kPathDecodeSplit : kPathDecode;
  }
  // multi-row: the fused tile kernel serves both grids up to kSelTileMaxCand candidates per row
  const bool tile_grid = grid_is_blocks(grid) || (grid.l == 32 && grid.s == 16);
  return tile_grid && g.n_cand <= kSelTileMaxCand ? kPathTile : kPathRowwise;
}

int select_decode_path(int64_t rows, int32_t n_q, int64_t q_pos0, int32_t n_init, int32_t n_local, WinGrid grid) {
  const SelectPath path = select_path(rows, n_q, q_pos0, n_init, n_local, grid);
  return path == kPathDecode ? 0 : path == kPathDecodeSplit ? 1 : -1;
}

hipError_t launch_decode_split_scores(const SelectArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads;
  const RowGeom g = row_geom(a.q_pos0, a.n_init, a.n_local, a.k_total);
  int32_t wf, wl;
  row_windows(g, a.grid, a.q_pos0, &wf, &wl);
  if (g.n_cand <= 0 || wl < wf) return hipSuccess;
  const int n_chunks = (wl - wf + 1 + 255) / 256;
  hipLaunchKernelGGL(rowwise_score_kernel, dim3((unsigned)(rows * n_chunks)), dim3(256), 0, stream, a, n_chunks);
  return hipGetLastError();
}

bool select_needs_scratch(int64_t rows, int32_t n_q, int64_t q_pos0, int32_t n_init, int32_t n_local, WinGrid grid) {
  const SelectPath path = select_path(rows, n_q, q_pos0, n_init, n_local, grid);
  return path == kPathRowwise || path == kPathDecodeSplit;
}

hipError_t launch_rowwise_topk(const SelectArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads * a.n_q;
  hipLaunchKernelGGL(rowwise_topk_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, a, rows);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.batch * a.n_kv_heads * a.n_q;
  const SelectPath path = select_path(rows, a.n_q, a.q_pos0, a.n_init, a.n_local, a.grid);
  if (path == kPathDecode) {
    hipLaunchKernelGGL(decode_select_kernel, dim3((unsigned)rows), dim3(kDecThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (path == kPathTile) return launch_prefill_select(a, stream);
  const int64_t pl = a.q_pos0 + a.n_q - 1;
  const RowGeom gl = row_geom(pl, a.n_init, a.n_local, a.k_total);
  int32_t wf, wl;
  row_windows(gl, a.grid, pl, &wf, &wl);
  if (gl.n_cand > 0 && wl >= wf && a.n_q >= kTileScoreMinRows) {
    // many rows: 64-row units score on MFMA, each key fragment shared by the unit's rows
    hipError_t e = launch_tile_scores(a, stream);
    if (e != hipSuccess) return e;
  } else if (gl.n_cand > 0 && wl >= wf) {  // the last row scores the most windows
    const int n_chunks = (wl - wf + 1 + 255) / 256;
    hipLaunchKernelGGL(rowwise_score_kernel, dim3((unsigned)(rows * n_chunks)), dim3(256), 0, stream, a, n_chunks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (path == kPathDecodeSplit)
    hipLaunchKernelGGL(decode_topk_kernel, dim3((unsigned)rows), dim3(kDecThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(rowwise_topk_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, a, rows);
  return hipGetLastError();
}

}  // namespace sparda

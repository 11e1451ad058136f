// launch.hpp -- host-side launchers of the SparDA kernels (private to the library).
// Arguments have been validated by the C ABI layer before any launcher runs; each launcher only
// computes a grid, enqueues kernels on `stream` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sparda {

// Geometry of one query row at position p (Eq. 1 / Eq. 4): forced and candidate blocks.
struct RowGeom {
  int blk;       // p / 64
  int init_hi;   // initial blocks [0, init_hi)
  int local_lo;  // local blocks [local_lo, blk] (local_lo >= init_hi)
  int n_forced;  // init_hi + blk - local_lo + 1
  int cand_lo;   // candidates [cand_lo, cand_lo + n_cand)
  int n_cand;
  int n_take;    // candidates chosen: min(k_total - n_forced, n_cand)
};

__host__ __device__ inline RowGeom row_geom(int64_t p, int n_init, int n_local, int k_total) {
  RowGeom g;
  g.blk = (int)(p / 64);
  g.init_hi = n_init < g.blk + 1 ? n_init : g.blk + 1;
  int lo = g.blk - n_local + 1;
  if (lo < 0) lo = 0;
  if (lo < g.init_hi) lo = g.init_hi;
  g.local_lo = lo;
  g.n_forced = g.init_hi + (g.blk - lo + 1);
  g.cand_lo = n_init;
  const int hi = g.blk - n_local;
  g.n_cand = hi >= n_init ? hi - n_init + 1 : 0;
  const int budget = k_total - g.n_forced;
  g.n_take = budget < g.n_cand ? budget : g.n_cand;
  return g;
}

// The compressed-key grid (Sec. 3, Eq. 2): window i holds the mean of tokens [i s, i s + l).
// A block's score is the largest score among the windows that overlap it and are complete at
// the query's position (the max-pool of the InfLLM-V2 selector).  With l = s = 64 every block is
// one window and the pool is the identity.
struct WinGrid {
  int32_t l, s;  // window length and stride, in tokens; l <= 64, s divides 64
};

// First and last window overlapping block j (the last one not yet clamped to visibility).
__host__ __device__ inline int32_t grid_win_lo(const WinGrid& w, int32_t j) {
  const int32_t t = j * 64 - w.l;
  return t < 0 ? 0 : t / w.s + 1;
}
__host__ __device__ inline int32_t grid_win_hi(const WinGrid& w, int32_t j) { return ((j + 1) * 64 - 1) / w.s; }
// Last window complete at position p (-1 if none).
__host__ __device__ inline int32_t grid_win_vis(const WinGrid& w, int64_t p) {
  return p + 1 >= w.l ? (int32_t)((p + 1 - w.l) / w.s) : -1;
}
__host__ __device__ inline bool grid_is_blocks(const WinGrid& w) { return w.l == 64 && w.s == 64; }

struct SelectArgs {
  const uint16_t* f;
  const uint16_t* kc;
  int16_t* sel;
  int16_t* cnt;
  float* ws;           // score scratch for the row-wise path
  int64_t ws_stride;   // floats per row in ws
  int32_t batch, n_kv_heads, n_q;
  int64_t q_pos0, nc_cap;
  int32_t n_init, n_local, k_total;
  WinGrid grid;        // compressed-key grid of kc (nc_cap counts its windows)
  // The multi-head selector only (select_multihead.hip):
  const uint16_t* q;   // bf16 [B][Hq][n_q][D] attention queries, Hq = n_kv_heads * group_size
  float scale_log2;    // softmax temperature times log2(e): scores are taken in the exp2 domain
  int32_t group_size;
};

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int16_t* sel;
  const int16_t* cnt;
  uint16_t* o;
  float* ws;           // split partials
  int32_t batch, n_kv_heads, group_size, n_q;
  int64_t q_pos0, t_cap;
  int32_t kv_mode, k_total;
  float sm_scale;
  int32_t n_splits;        // splits of the selected-block list per row
  int32_t blocks_per_split;
};

// Tiles of the fused multi-row selection kernel.
constexpr int kSelTileRows = 64;
constexpr int kSelTileMaxCand = 512;
// Candidates a decode row may have for the fused decode kernel (scores held in 64 KiB of LDS).
constexpr int kDecodeMaxCand = 16384;

hipError_t launch_compress(const uint16_t* k, uint16_t* kc, int32_t rows, int64_t t_cap, int64_t nc_cap,
                           WinGrid grid, int32_t w_begin, int32_t w_end, hipStream_t stream);

// Windows a row at position p scores: [first, last] (empty when last < first).
__host__ __device__ inline void row_windows(const RowGeom& g, const WinGrid& w, int64_t p, int32_t* first,
                                           int32_t* last) {
  *first = grid_win_lo(w, g.cand_lo);
  const int32_t hi = grid_win_hi(w, g.cand_lo + g.n_cand - 1), vis = grid_win_vis(w, p);
  *last = g.n_cand > 0 ? (hi < vis ? hi : vis) : *first - 1;
}

// True when the call keeps its window scores in workspace scratch: the row-wise path, and decode
// calls with fewer rows than CUs (scored by many workgroups per row).
bool select_needs_scratch(int64_t rows, int32_t n_q, int64_t q_pos0, int32_t n_init, int32_t n_local, WinGrid grid);
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);
// Which decode path a select call takes: 0 the fused kernel (one workgroup per row, scores in
// LDS), 1 the split path (window scores by many workgroups per row into the workspace, then one
// workgroup per row selects), -1 neither (multi-row or too many windows).
int select_decode_path(int64_t rows, int32_t n_q, int64_t q_pos0, int32_t n_init, int32_t n_local, WinGrid grid);
// The split decode path's scoring launch alone (its selection runs in decode_topk_row).
hipError_t launch_decode_split_scores(const SelectArgs& a, hipStream_t stream);
// Multi-row tiles of 64 rows with at most kSelTileMaxCand candidates (select_prefill.hip).
hipError_t launch_prefill_select(const SelectArgs& a, hipStream_t stream);

// Each query row's largest Forecast score over its candidate blocks, (64, 64) grid
// (score_max.hip).  Units are the rows of one (batch, group) inside one 64-token block.
struct ScoreMaxArgs {
  const uint16_t* f;   // bf16 [n_groups][n_q][128]
  const uint16_t* kc;  // bf16 [n_groups][nc_cap][128]
  float* row_max;      // [n_groups][n_q]
  int64_t nc_cap, q_pos0;
  int32_t n_q, n_groups;  // n_groups = batch * n_kv_heads
  int32_t blk0, n_units;  // blocks of the first and following rows: [blk0, blk0 + n_units)
  int32_t n_init, n_local;
};
hipError_t launch_score_rowmax(const ScoreMaxArgs& a, hipStream_t stream);
// Window scores of multi-row calls into the row-wise workspace on MFMA (score_max.hip): units of
// the rows inside one 64-token block, the windows of each unit's last row.
hipError_t launch_tile_scores(const SelectArgs& a, hipStream_t stream);

// Row-wise top-k over pooled window scores already in a.ws (row stride a.ws_stride, window wf of
// the row at offset 0), for the multi-head selector's row-wise path (select.hip).
hipError_t launch_rowwise_topk(const SelectArgs& a, hipStream_t stream);
// The InfLLM-V2 multi-head selector (select_multihead.hip).  Workspace floats of a call (0 on the
// fused decode path); *stride gets the floats per row.
size_t multihead_ws_floats(int64_t rows, int32_t group_size, int32_t n_q, int64_t q_pos0, int32_t n_init,
                           int32_t n_local, int32_t k_total, WinGrid grid, int64_t* stride);
hipError_t launch_multihead_select(const SelectArgs& a, hipStream_t stream);

// Split count and blocks per split the attention launcher uses for `rows` query rows.
void attn_plan(int64_t rows, int32_t k_total, int32_t* n_splits, int32_t* blocks_per_split);
hipError_t launch_sparse_attn(const AttnArgs& a, hipStream_t stream);
// One decode step: the select call s, then the attention call a over the sets it writes.  Where
// the select takes a decode path (fused, or split: its scoring launch first), k_total <= 1024
// and the caches are full, one kernel per (row, attention split) selects and attends
// (decode_step_kernel for G <= 5, decode_step_wide_kernel for 6 <= G <= 16; plus the split
// combine); otherwise the two calls.
hipError_t launch_decode_step(const SelectArgs& s, const AttnArgs& a, hipStream_t stream);
// True when a multi-row call takes the tiled kernel (attention_prefill.hip), which needs no
// workspace: at least 16 rows, 16 % G == 0, and the tile's row bitmaps fit in LDS.
bool attn_uses_tiles(int32_t group_size, int32_t n_q, int64_t q_pos0);
hipError_t launch_prefill_attn(const AttnArgs& a, hipStream_t stream);

// The indexer-training loss (indexer_kl.hip); kt_ws holds (q_pos0 + n_q - 1) fine windows per row.
hipError_t launch_indexer_kl(const uint16_t* q, const uint16_t* k, const uint16_t* f, const uint16_t* kp,
                             uint16_t* kt_ws, float* sw_ws, float* loss, float* dF, int32_t batch, int32_t n_kv_heads,
                             int32_t group_size, int32_t n_q, int64_t q_pos0, int64_t t_cap, int64_t nc_cap,
                             int32_t n_init, int32_t n_local, int32_t k_top, WinGrid grid, float sm_scale,
                             hipStream_t stream);
hipError_t launch_plan_staging(const int16_t* sel, const int16_t* cnt, int64_t p, int16_t* slot_blk, int16_t* slot_len,
                               int16_t* fetch, int16_t* staged, int16_t* stage_cnt, int32_t* n_fetch, int64_t rows,
                               int32_t k_total, hipStream_t stream);
// New K/V rows [B][Hkv][n_new][D] (device) into the mapped host pools at positions
// [pos0, pos0 + n_new) (gather.hip).
hipError_t launch_writeback(const uint16_t* k_new, const uint16_t* v_new, uint16_t* host_k, uint16_t* host_v,
                            int64_t rows, int32_t n_new, int64_t pos0, int64_t t_cap, int32_t n_workgroups,
                            hipStream_t stream);
// The decoded token's K/V rows [B][Hkv][D] into every staging slot that holds block p / 64, at row
// p % 64 (gather.hip).
hipError_t launch_stage_append(const uint16_t* k_new, const uint16_t* v_new, const int16_t* sel, const int16_t* cnt,
                               int64_t p, uint16_t* stage_k, uint16_t* stage_v, int64_t rows, int32_t k_total,
                               hipStream_t stream);
hipError_t launch_gather(const uint16_t* host_k, const uint16_t* host_v, const int16_t* sel, const int16_t* cnt,
                         uint16_t* stage_k, uint16_t* stage_v, int64_t rows, int64_t t_cap, int32_t k_total,
                         int32_t n_workgroups, hipStream_t stream);

}  // namespace sparda

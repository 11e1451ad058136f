/*
 * sparda.h -- C ABI of the MI355X (gfx950) SparDA selection + block-sparse attention library.
 *
 * SparDA (Sparse Decoupled Attention) adds a Forecast projection F to every layer.  The
 * Forecast row of layer l, one head per GQA group, scores the mean-pooled block keys K~ of layer
 * l+1; the top-k blocks, merged with the initial and local blocks, are the only KV blocks that
 * layer l+1 attends to (paper Sec. 4.1, Eq. 3-5; the attended-set structure is Eq. 1 of Sec. 3).
 * This library implements that data path on one GPU:
 *
 *   sparda_compress_keys    K -> K~               (Sec. 3, Eq. 2)
 *   sparda_forecast_select  F, K~ -> block sets   (Sec. 4.1, Eq. 4 with Eq. 1)
 *   sparda_forecast_score_max F, K~ -> each row's largest candidate score (the scoring
 *                           contraction alone, a measurement of Eq. 4 without the top-k)
 *   sparda_sparse_attn      Q, K, V, sets -> O    (Sec. 4.1, Eq. 5 with Eq. 1)
 *   sparda_sparse_attn_noalloc  the same without a workspace argument (a static scratch array),
 *                           for callers that cannot allocate
 *   sparda_decode_step      F, K~, Q, K, V -> block sets and O: one decode step of a layer, the
 *                           select and the attention in one launch where they fit one workgroup
 *                           per row (Sec. 4.1, Eq. 4 then Eq. 5, with Eq. 1)
 *   sparda_multihead_select Q, K~ -> block sets   (the InfLLM-V2 selector of Sec. 3 that the
 *                           Forecast indexer replaces; a baseline)
 *   sparda_gather_blocks    host KV pool -> HBM staging of the selected blocks, meant for a side
 *                           stream so that layer l+1's fetch overlaps layer l (Sec. 4.3, Alg. 2)
 *   sparda_stage_append_kv  the decoded token -> the staged copy of its own block (Alg. 2's append,
 *                           for offloaded layers whose blocks were gathered before the token existed)
 *   sparda_writeback_kv     new K/V rows -> the pinned host pools (the asynchronous write-back of
 *                           Sec. 5.3, Efficiency Results), for a side stream
 *   sparda_plan_staging     step-to-step reuse of the staged blocks: which blocks the next gather
 *                           must fetch (the NOSI engine of App. C)
 *   sparda_indexer_kl       Q, K, F, K~ -> the indexer-training loss and its gradient w.r.t. F
 *                           (Sec. 4.2, Eq. 6-7)
 *
 * Conventions shared by every call:
 *   - Every function returns an int status: SPARDA_OK (0) or a negative SPARDA_ERR_* code.  No
 *     call throws, aborts or prints.  sparda_last_error_detail() gives a human-readable reason
 *     for the last failure of the calling thread.
 *   - Tensors are bf16 (passed as void*, 2 bytes per element, IEEE bfloat16 bits), dense and
 *     row-major in the layouts given per argument.  Block indices are int16.
 *   - Device pointers must be 16-byte aligned device (HBM) memory owned by the caller.  The
 *     library allocates nothing and keeps no state beyond a thread-local error string and, for
 *     sparda_sparse_attn_noalloc, one static scratch array per device with its looked-up address:
 *     every buffer, workspace and stream belongs to the caller and must stay alive until the work
 *     enqueued on the stream has completed.
 *   - Every compute call only enqueues work on the given stream and returns; argument errors are
 *     reported synchronously before anything is enqueued (nothing is written on error); a failed
 *     launch returns SPARDA_ERR_HIP; device faults surface at the caller's next synchronisation.
 *   - Ordering between streams (e.g. a gather on a side stream and the attention that reads its
 *     staging buffer) is the caller's: record an event after the gather and make the compute
 *     stream wait on it.
 *   - v1 limits: head_dim 128, block 64, compression grid (64, 64) -- one key per block -- or the
 *     paper's (32, 16) (App. C),
 *     group_size 1..16, block indices < 32768.  Other values return SPARDA_ERR_UNSUPPORTED.
 *
 * Notation: B batch, Hkv KV heads (= Forecast heads = GQA groups), G query heads per group,
 * Hq = Hkv * G, D head_dim, L block size (64), n_q query rows per (batch, group), p = q_pos0 + r
 * the position of row r, blk(p) = p / L.  Query head h belongs to group h / G.
 */
#ifndef SPARDA_H
#define SPARDA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum sparda_status {
  SPARDA_OK = 0,
  SPARDA_ERR_INVALID_ARG = -1,     /* null/misaligned pointer, inconsistent sizes, bad range   */
  SPARDA_ERR_UNSUPPORTED = -2,     /* valid but outside the v1 limits listed above             */
  SPARDA_ERR_WORKSPACE = -3,       /* workspace smaller than sparda_workspace_size() reports   */
  SPARDA_ERR_HOST_NOT_MAPPED = -4, /* gather source is not device-accessible pinned host memory */
  SPARDA_ERR_HIP = -5              /* a HIP runtime call or kernel launch failed                */
};

/* Problem description shared by all calls. */
typedef struct sparda_shape {
  uint32_t struct_size;  /* = sizeof(sparda_shape); lets the ABI grow                          */
  int32_t batch;         /* B >= 1                                                              */
  int32_t n_kv_heads;    /* Hkv >= 1: KV heads, one Forecast head each                          */
  int32_t group_size;    /* G in 1..16: query heads per KV head (GQA group)                     */
  int32_t head_dim;      /* D: 128                                                              */
  int32_t block_size;    /* L: 64 tokens per block                                              */
  int32_t cmp_kernel;    /* compression window length l_C: 64 (one key per block) or 32        */
  int32_t cmp_stride;    /* compression stride s_C: 64, or 16 with l_C = 32                    */
  int32_t n_init;        /* initial blocks always attended (>= 0)                               */
  int32_t n_local;       /* local blocks always attended, the query's own block included (>= 1) */
  int32_t k_total;       /* attended-set size per query row, forced blocks included;            */
                         /* n_init + n_local <= k_total <= 32767                                */
  int64_t t_cap;         /* token capacity (T stride) of the K/V caches; a multiple of L        */
  int64_t nc_cap;        /* window capacity (stride) of the K~ cache: compressed keys per row   */
} sparda_shape;

/* Workspace owners for sparda_workspace_size(). */
enum sparda_op {
  SPARDA_OP_FORECAST_SELECT = 1,
  SPARDA_OP_SPARSE_ATTN = 2,
  SPARDA_OP_MULTIHEAD_SELECT = 3,
  SPARDA_OP_INDEXER_KL = 4,
  SPARDA_OP_DECODE_STEP = 5
};

/*
 * sparda_compress_keys -- mean-pooled compressed keys (Sec. 3, Eq. 2): window i of the grid
 * (l_C, s_C) holds the keys of tokens [i s_C, i s_C + l_C); with l_C = s_C = L window i is block i.
 *   k_cache  in : bf16 [B][Hkv][t_cap][D] device.
 *   t_ctx       : tokens currently valid in k_cache (t_ctx <= t_cap).
 *   win_begin, win_end : compress windows i in [win_begin, win_end); every one must be complete,
 *                 i.e. (win_end - 1) s_C + l_C <= t_ctx, and win_end <= nc_cap.  In decode, call
 *                 it with the windows completed by the newest tokens (the incremental K~ update
 *                 of Alg. 2: one window per L tokens on the (64, 64) grid, one per 16 on
 *                 (32, 16)); win_begin == win_end is a no-op.
 *   k_cmp   out : bf16 [B][Hkv][nc_cap][D] device; only rows [win_begin, win_end) are written.
 *   K~_i = round_to_nearest_even_bf16( (1/l_C) * sum of the l_C keys of window i ), the sum being
 *   exact for bf16 inputs (float64 accumulation), so the result does not depend on order.
 */
int sparda_compress_keys(const sparda_shape* shape, const void* k_cache, int64_t t_ctx, int32_t win_begin,
                         int32_t win_end, void* k_cmp, hipStream_t stream);

/*
 * sparda_forecast_select -- attended block set of every query row (Sec. 4.1, Eq. 4; Eq. 1).
 *   f      in  : bf16 [B][Hkv][n_q][D] device, the Forecast rows (one head per group).  For a
 *                one-layer-ahead selection these are layer l's Forecast rows and k_cmp is layer
 *                l+1's K~ (Eq. 4); for layer 0 they are the current-layer Forecast.
 *   n_q        : rows per (batch, group), >= 1.  n_q == 1 is the decode form.
 *   q_pos0     : position of row 0; row r is at p = q_pos0 + r; p < t_cap.
 *   k_cmp  in  : bf16 [B][Hkv][nc_cap][D] device; every window that overlaps a candidate block
 *                of the last row and is complete at its position must be valid and < nc_cap.
 *   sel    out : int16 [B][Hkv][n_q][k_total] device: ascending block indices, -1 padded.
 *   cnt    out : int16 [B][Hkv][n_q] device: valid entries of each row = min(k_total, blk(p)+1).
 *   ws, ws_bytes: device workspace of at least sparda_workspace_size(SPARDA_OP_FORECAST_SELECT).
 * Per row: forced = blocks [0, n_init) U [blk(p) - n_local + 1, blk(p)] (clipped to >= 0);
 * candidates = [n_init, blk(p) - n_local]; every window i scores F_row . K~_i (float32
 * accumulation, no softmax, no scale) and candidate j scores s_j = the largest score of the windows
 * that overlap block j and are complete at p (i s_C + l_C <= p + 1): the max-pool to block scores
 * of the InfLLM-V2 selector (Sec. 3), the identity on the (64, 64) grid.  The k_total - |forced|
 * best candidates by (score descending, block index ascending) are added to the forced blocks.
 * All G query heads of a group share the set.
 */
int sparda_forecast_select(const sparda_shape* shape, const void* f, int32_t n_q, int64_t q_pos0,
                           const void* k_cmp, int16_t* sel, int16_t* cnt, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/*
 * sparda_forecast_score_max -- the scoring contraction of sparda_forecast_select alone (Sec. 4.1,
 * Eq. 4): every candidate block of every query row is scored and each row's largest score is
 * written.  It measures the dense F . K~ contraction apart from the per-row top-k (the scores
 * are reduced on chip; nothing else is written).  (64, 64) grid only.
 *   f, n_q, q_pos0, k_cmp : as for sparda_forecast_select.
 *   row_max out : float32 [B][Hkv][n_q] device (4-byte aligned): max over the row's candidates
 *                [n_init, blk(p) - n_local] of F_row . K~_j (float32 accumulation), -inf for a
 *                row without candidates.
 * Errors: SPARDA_ERR_UNSUPPORTED for the (32, 16) grid; SPARDA_ERR_INVALID_ARG for null or
 * misaligned pointers, rows outside t_cap, or a candidate at or beyond nc_cap.
 */
int sparda_forecast_score_max(const sparda_shape* shape, const void* f, int32_t n_q, int64_t q_pos0,
                              const void* k_cmp, float* row_max, hipStream_t stream);

/*
 * sparda_multihead_select -- the same attended sets chosen by the InfLLM-V2 multi-head selector
 * that the Forecast indexer replaces (Sec. 3, three-stage block representation; its per-head
 * score is the softmax of the indexer-training target, Sec. 4.2).  A baseline for comparing
 * selection cost and choices; it selects from the attention queries of the same layer.
 *   q      in  : bf16 [B][Hq][n_q][D] device, Hq = n_kv_heads * group_size; heads
 *                m G .. m G + G - 1 belong to group m.
 *   n_q, q_pos0: as for sparda_forecast_select.
 *   k_cmp  in  : bf16 [B][Hkv][nc_cap][D] device; every window complete at the last row's
 *                position (i s_C + l_C <= p + 1) must be valid and < nc_cap, since each head's
 *                softmax runs over all of them, the initial and local blocks' windows included.
 *   sm_scale   : softmax temperature, normally 1/sqrt(D); finite and > 0.
 *   sel, cnt out: as for sparda_forecast_select.
 *   ws, ws_bytes: device workspace of at least sparda_workspace_size(SPARDA_OP_MULTIHEAD_SELECT)
 *                (0 bytes for decode with G in {1, 2, 4, 8} up to about 38K windows times G).
 * Per row: for every head h of the group, z_hi = sm_scale q_h . K~_i over the complete windows i,
 * a_hi = softmax_i(z_hi) (float32, exp2 domain, each head's exact maximum subtracted); window i's
 * shared score is sum_h a_hi; candidate j scores the largest shared score of the windows that
 * overlap block j and are complete at p; forced blocks, ordering and ties as for
 * sparda_forecast_select.
 */
int sparda_multihead_select(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0,
                            const void* k_cmp, float sm_scale, int16_t* sel, int16_t* cnt, void* ws,
                            size_t ws_bytes, hipStream_t stream);

/*
 * sparda_sparse_attn -- block-sparse attention over the attended sets (Sec. 4.1, Eq. 5; Eq. 1).
 *   q      in  : bf16 [B][Hq][n_q][D] device.
 *   n_q, q_pos0: as for select (row r is at position p = q_pos0 + r).
 *   k, v   in  : kv_mode 0 -- bf16 [B][Hkv][t_cap][D] device, the full caches (token t in row t).
 *                kv_mode 1 -- bf16 [B][Hkv][k_total][L][D] device staging filled by
 *                sparda_gather_blocks: slot s holds the L tokens of block sel[s].  Decode only
 *                (n_q == 1).
 *   sel, cnt in: as produced by sparda_forecast_select (any order of the first cnt entries is
 *                accepted; entries outside [0, blk(p)] are skipped; the attended tokens are the
 *                union of the listed blocks, so a block listed twice is attended once).
 *   sm_scale   : logit scale, normally 1/sqrt(D).
 *   o      out : bf16 [B][Hq][n_q][D] device.  A row that attends no token gets zeros.
 *   ws, ws_bytes: device workspace of at least sparda_workspace_size(SPARDA_OP_SPARSE_ATTN).
 * o = softmax(sm_scale * q K_S^T) V_S over the tokens t <= p of the attended blocks S, with bf16
 * inputs, float32 accumulation and online softmax.
 */
int sparda_sparse_attn(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0, const void* k,
                       const void* v, int32_t kv_mode, const int16_t* sel, const int16_t* cnt, float sm_scale,
                       void* o, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * sparda_decode_step -- one decode step of a layer (n_q == 1, full K/V caches): the Forecast
 * selection of every (batch, group) row (Sec. 4.1, Eq. 4 with Eq. 1) followed by the block-sparse
 * attention over the selected sets (Eq. 5).  The results are those of
 *     sparda_forecast_select(shape, f, 1, q_pos, k_cmp, sel, cnt, ws, ws_bytes, stream);
 *     sparda_sparse_attn(shape, q, 1, q_pos, k, v, 0, sel, cnt, sm_scale, o, ws, ws_bytes, stream);
 * bit for bit.  Where the selection takes a decode path (one workgroup per row, or its
 * scoring spread over workgroups below 256 rows) and k_total <= 1024, one kernel does both
 * for each (row, attention split): rows that finish their selection early already stream their
 * K and V while others select, and with splits every split's workgroup computes the row's
 * selection itself; otherwise it enqueues the two calls.
 *   f, k_cmp   : as for sparda_forecast_select with n_q = 1; q_pos is the row's position.
 *   q, k, v    : as for sparda_sparse_attn with n_q = 1 and kv_mode 0.
 *   sm_scale   : logit scale, finite.
 *   sel, cnt out: the sets, as sparda_forecast_select writes them.
 *   o      out : bf16 [B][Hq][1][D] device.
 *   ws, ws_bytes: device workspace of at least sparda_workspace_size(SPARDA_OP_DECODE_STEP, n_q = 1):
 *                the selection's window scores, then (256-byte aligned) the attention's split
 *                partials, side by side (0 bytes when neither is needed).
 * Errors: those of the two calls, all reported before anything is enqueued.
 */
int sparda_decode_step(const sparda_shape* shape, const void* f, int64_t q_pos, const void* k_cmp, const void* q,
                       const void* k, const void* v, float sm_scale, int16_t* sel, int16_t* cnt, void* o, void* ws,
                       size_t ws_bytes, hipStream_t stream);

/*
 * sparda_sparse_attn_noalloc -- sparda_sparse_attn without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, layouts, kernels and results as sparda_sparse_attn;
 * the split partials of calls with fewer rows than the chip has CUs go to a scratch array of
 * SPARDA_NOALLOC_SCRATCH_BYTES that the library holds in every device's memory (a static device
 * array, one copy per GPU, kept until the process ends).  The call allocates nothing.
 *   - The first call on a device looks the array's address up (hipGetSymbolAddress) with that
 *     device current; the stream must belong to the current device, as for any HIP launch.
 *   - Every call on one GPU shares that GPU's array: calls whose work overlaps on that GPU (two
 *     streams, two threads) race on it and must be ordered by the caller.  The array keeps the
 *     last call's partials; nothing in it needs to start at zero.
 *   - A call whose partials exceed the array returns SPARDA_ERR_WORKSPACE.  The array holds
 *     511 rows x splits x 16 heads x (D + 2) floats, which covers every call the v1 limits allow
 *     (partials exist only below 256 rows, with at most ceil(256 / rows) splits per row).
 */
#define SPARDA_NOALLOC_SCRATCH_BYTES ((size_t)4718592) /* 4.5 MiB */
int sparda_sparse_attn_noalloc(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0, const void* k,
                               const void* v, int32_t kv_mode, const int16_t* sel, const int16_t* cnt,
                               float sm_scale, void* o, hipStream_t stream);

/*
 * sparda_indexer_kl -- the indexer-training loss of Sec. 4.2 (Eq. 6-7) per query row, and its
 * gradient with respect to the Forecast row (the Forecast projection is the only trained part;
 * its weight gradient is this gradient times the layer input, a plain GEMM).
 *   shape     : the prediction grid is shape's (cmp_kernel, cmp_stride), normally (32, 16); the
 *               target uses fine (2, 1) windows (the training table of App. B).
 *   q     in  : bf16 [B][Hq][n_q][D] device, the target layer's attention queries.
 *   k     in  : bf16 [B][Hkv][t_cap][D] device, the target layer's keys (tokens up to the last
 *               row's position are read).
 *   f     in  : bf16 [B][Hkv][n_q][D] device, the Forecast rows of the previous layer.
 *   k_cmp in  : bf16 [B][Hkv][nc_cap][D] device, the target layer's keys on the prediction grid;
 *               every window complete at the last row must be < nc_cap.
 *   n_q, q_pos0: rows and the position of row 0; every row must have a complete window
 *               (q_pos0 >= cmp_kernel - 1); at most 16384 windows per row.
 *   sm_scale  : 1 / tau of both softmaxes (finite, > 0).
 *   k_top     : size of the target's selected set, 0 .. 4096.
 *   loss  out : float [B][Hkv][n_q] device.
 *   d_f   out : float [B][Hkv][n_q][D] device, d loss / d F.
 *   ws, ws_bytes: device workspace of sparda_workspace_size(SPARDA_OP_INDEXER_KL) bytes (the fine
 *               windows, then every row's target weight of each fine window).
 * Per row at position p: positions w = the prediction windows complete at p; the target T_w =
 * max over the fine windows inside w (tokens [i, i + 2) within [w s, w s + l)) of the sum over the
 * group's heads of softmax_i(sm_scale q_h . K~fine_i) (fine windows complete at p); the
 * prediction P = softmax_w(sm_scale F . K~_w); S = the k_top largest T_w (ties: lower w) among
 * positions whose tokens lie in candidate blocks [n_init, blk(p) - n_local]; loss =
 * sum_{c in S} t_c log(t_c / P_c) + t_rest log(t_rest / R) with t = T / sum T, t_rest and R the
 * masses outside S; d F = sm_scale sum_w g_w K~_w with g_w = P_w - t_w in S and
 * P_w (1 - t_rest / R) outside.  float32 arithmetic (exp2 domain), bf16 inputs.
 */
int sparda_indexer_kl(const sparda_shape* shape, const void* q, const void* k, const void* f, const void* k_cmp,
                      int32_t n_q, int64_t q_pos0, float sm_scale, int32_t k_top, float* loss, float* d_f,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * sparda_plan_staging -- step-to-step reuse of a layer's staging buffer (the NOSI inference engine
 * of the paper's efficiency setup, App. C: each layer caches the blocks its previous decode step
 * attended, so a step fetches only the newly selected ones).  Decode form, one call per layer and
 * step, before that layer's gather.
 *   sel, cnt   in : the step's selection, int16 [B][Hkv][k_total] and [B][Hkv] device (as
 *                   sparda_forecast_select produces for n_q == 1: distinct blocks).
 *   q_pos         : the query's position p; 0 <= p < t_cap.
 *   slot_blk, slot_len in/out : int16 [B][Hkv][k_total] device, the staging state: slot s holds the
 *                   first slot_len[s] tokens of block slot_blk[s] (-1: empty).  Initialise slot_blk
 *                   to -1 (and slot_len to 0) once; the call updates both.
 *   fetch     out : int16 [B][Hkv][k_total] device, the block to copy into slot s this step, -1
 *                   when the slot needs no copy: pass it to sparda_gather_blocks with stage_cnt.
 *   sel_staged out: int16 [B][Hkv][k_total] device, the block slot s holds for this step's
 *                   attention, -1 when the step does not attend it: pass it to sparda_sparse_attn
 *                   (kv_mode 1) with stage_cnt.
 *   stage_cnt out : int16 [B][Hkv] device, k_total for every row.
 *   n_fetch   out : int32 [B][Hkv] device, blocks fetched per row (the copy volume).
 * A staged block is kept when it is an entry of the new set and covers every token of the block
 * up to p (need(j) = min(L, p + 1 - j L) tokens; tokens never change once written); slots are
 * examined in ascending order, each claiming the first unclaimed matching entry.  The other
 * entries are fetched, in entry order, into the remaining slots in ascending order; slots the
 * step does not use are emptied.  k_total <= 1024 (SPARDA_ERR_UNSUPPORTED otherwise).
 */
int sparda_plan_staging(const sparda_shape* shape, const int16_t* sel, const int16_t* cnt, int64_t q_pos,
                        int16_t* slot_blk, int16_t* slot_len, int16_t* fetch, int16_t* sel_staged,
                        int16_t* stage_cnt, int32_t* n_fetch, hipStream_t stream);

/*
 * sparda_gather_blocks -- copy the selected blocks of a host-resident KV pool into HBM staging
 * (Sec. 4.3 persistent prefetch; Alg. 2 "launch prefetch of B_{l+1}").
 *   host_k, host_v in : bf16 [B][Hkv][t_cap][D] pinned host memory mapped into the device
 *                       address space (e.g. hipHostMalloc); SPARDA_ERR_HOST_NOT_MAPPED otherwise.
 *                       The allocation holding each pointer must extend B Hkv t_cap D 2 bytes
 *                       from it (looked up with hipMemGetAddressRange); SPARDA_ERR_INVALID_ARG
 *                       otherwise, so a short pool is refused before any PCIe access.
 *   sel, cnt       in : device, decode-form selection: int16 [B][Hkv][k_total] and [B][Hkv].
 *   stage_k, stage_v out : bf16 [B][Hkv][k_total][L][D] device; slot s < cnt receives block
 *                       sel[s]; other slots are untouched; entries with (sel+1)*L > t_cap are
 *                       skipped.
 *   n_workgroups      : size of the persistent grid (the CU budget the copy may occupy), >= 1;
 *                       the grid loops over all (batch, group, slot) copy tasks.
 *   stream            : normally a side stream distinct from the compute stream.
 */
int sparda_gather_blocks(const sparda_shape* shape, const void* host_k, const void* host_v, const int16_t* sel,
                         const int16_t* cnt, void* stage_k, void* stage_v, int32_t n_workgroups,
                         hipStream_t stream);

/*
 * sparda_stage_append_kv -- appends the decoded token to the staged copy of its own block (Alg. 2
 * appends each step's K/V to the cache; in an offloaded layer the attended blocks were gathered
 * before the token existed, because layer l's prefetch is launched during layer l-1).
 *   k_new, v_new in : bf16 [B][Hkv][D] device (16-byte aligned), the token at position q_pos.
 *   q_pos           : the token's position, 0 <= q_pos < t_cap.
 *   sel, cnt     in : device, the staging layout the attention will read: int16 [B][Hkv][k_total]
 *                     and [B][Hkv] (the gather's sel/cnt, or the staging plan's sel_staged/stage_cnt).
 *   stage_k, stage_v in/out: bf16 [B][Hkv][k_total][L][D] device staging.
 * Every slot s < cnt with sel[s] == q_pos / L receives the row at q_pos mod L; nothing else is
 * written.  Call it on the compute stream after the gather into that staging has completed and
 * before the attention.
 */
int sparda_stage_append_kv(const sparda_shape* shape, const void* k_new, const void* v_new, int64_t q_pos,
                           const int16_t* sel, const int16_t* cnt, void* stage_k, void* stage_v, hipStream_t stream);

/*
 * sparda_writeback_kv -- stores newly created K/V rows into the pinned host pools that the
 * offloaded layers gather from: the asynchronous CPU write-back of new KV entries after they are
 * used for attention (Sec. 5.3, prefill-throughput paragraph; in decode, the token Alg. 2 appends
 * each step).  Meant for a side
 * stream, like the gather.
 *   k_new, v_new in : bf16 [B][Hkv][n_new][D] device (16-byte aligned).
 *   n_new, pos0     : the rows land at positions [pos0, pos0 + n_new) of every (batch, group)
 *                     pool row; n_new >= 1, pos0 >= 0, pos0 + n_new <= t_cap.
 *   host_k, host_v out: bf16 [B][Hkv][t_cap][D] pinned host memory mapped for the device, each
 *                     allocation extending B Hkv t_cap D 2 bytes from the pointer (as for
 *                     sparda_gather_blocks: SPARDA_ERR_HOST_NOT_MAPPED, SPARDA_ERR_INVALID_ARG).
 *   n_workgroups    : persistent workgroups writing over PCIe (the CU budget), >= 1.
 * The copy is bitwise; positions outside the range are not touched.  Ordering against gathers
 * or host reads of the same positions is the caller's (record an event, synchronise).
 */
int sparda_writeback_kv(const sparda_shape* shape, const void* k_new, const void* v_new, int32_t n_new, int64_t pos0,
                        void* host_k, void* host_v, int32_t n_workgroups, hipStream_t stream);

/*
 * sparda_workspace_size -- device workspace bytes that call `op` (a sparda_op) needs for n_q
 * rows starting at position q_pos0 (the same n_q and q_pos0 as the call).
 *   Returns SPARDA_OK and writes *bytes (0 is possible); argument errors as for the call itself.
 *   The workspace is scratch: its contents are not needed between calls.
 */
int sparda_workspace_size(const sparda_shape* shape, int32_t op, int32_t n_q, int64_t q_pos0, size_t* bytes);

/* Static text for a status code (never null). */
const char* sparda_status_string(int status);

/* Reason for the calling thread's last failed call ("" if none). */
const char* sparda_last_error_detail(void);

#ifdef __cplusplus
}
#endif

#endif /* SPARDA_H */

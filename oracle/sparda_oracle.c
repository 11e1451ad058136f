/*
 * sparda_oracle.c -- plain CPU oracle for SparDA's selection + block-sparse attention path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file exists to check the GPU library, never to stand in for
 * it: only the test suite, the smoke check and the benchmark's CPU-baseline leg load it.  It
 * shares no source, header, table or helper with the HIP path.
 *
 * Every function is the plain definition of what the method computes, written with loops in
 * float64 (bf16 inputs are exact in float64).  Nothing is blocked, fused or reordered.
 *
 *   compress   Key compression, paper Sec. 3 (InfLLM-V2 recap), Eq. 2: one compressed key per
 *              window of l_C keys with stride s_C, the mean of the window (window i covers
 *              tokens [i s_C, i s_C + l_C)).  Grids with windows no longer than a block and a
 *              stride dividing the block are accepted: (64, 64), one key per block, and the
 *              paper's (32, 16), among others.
 *   select     Sec. 4.1, Eq. 4 with the attended-set union of Eq. 1: the Forecast row of a GQA
 *              group scores every compressed key by a plain dot product (one Forecast head per
 *              group, no softmax, no scale -- "Forecast indexer" paragraph of Sec. 4.1); a
 *              max-pool turns the compressed-grid scores into block scores (the final stage of
 *              the InfLLM-V2 selector that Sec. 3 recaps and Sec. 4.1 reuses): a block's score is
 *              the largest score of the windows that overlap it and are complete at the query's
 *              position.  The top-k block scores, excluding the initial and local blocks, are
 *              merged with the initial and local blocks.  Ties in score are broken by the lower
 *              block index.  With window = stride = block the max-pool is the identity.
 *   multihead  The InfLLM-V2 selector that SparDA replaces (Sec. 3, "three-stage block
 *              representation", whose per-head score the indexer-training target of Sec. 4.2 writes out as
 *              its target): every one of the G query heads of a group scores the compressed keys,
 *              a softmax with the attention temperature turns each head's scores into a
 *              distribution over the keys complete at the query's position, the G distributions
 *              are summed into one shared score per key, and the same max-pool, top-k and union
 *              as above follow.
 *   attend     Sec. 3, Eq. 1 and Sec. 4.1, Eq. 5: softmax attention of the query over exactly the
 *              keys/values of the attended blocks, causal within the query's own block.
 *   gather     Sec. 4.3 and Alg. 2 (prefetch of the selected blocks): staging slot s holds the 64
 *              keys/values of block sel[s].
 *   kl         The indexer-training loss (Sec. 4.2, Eq. 6-7, with the fine-grained target of the
 *              same section and the windows of the training table in App. B): a target
 *              distribution from the attention queries over fine (2, 1) compressed keys,
 *              max-pooled to the (32, 16) prediction grid; the Forecast softmax over that grid;
 *              the KL divergence of their (k+1)-bucket partitions by the target's top-k set, and
 *              its gradient with respect to the Forecast row.
 *   plan       Step-to-step reuse of the staged blocks (the NOSI engine of the efficiency setup,
 *              App. C: each layer keeps the blocks its previous decode step attended, and a step
 *              fetches only the newly selected ones): which staging slots keep their block and
 *              which blocks are fetched into which slots.
 *
 * Readings of the paper that these definitions take (k counts the forced blocks, the local
 * window is block-granular and contains the query's own block, score ties go to the lower
 * index, out-of-range selected entries are skipped, a block listed twice is attended once)
 * are listed with their reasons in the design notes of the repository.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define REF_OK 0
#define REF_ERR_INVALID_ARG (-1)
#define REF_ERR_UNSUPPORTED (-2)

/* The oracle's own description of a problem.  Field meanings:
 *   batch, n_kv_heads, group_size (query heads per KV head), head_dim,
 *   block_size (tokens per block), cmp_kernel / cmp_stride (compression window),
 *   n_init (initial blocks always attended), n_local (local blocks always attended, counting the
 *   query's own block), k_total (attended-set size, forced blocks included),
 *   t_cap (token capacity = T stride of the K/V caches), nc_cap (window capacity of K~). */
typedef struct {
  int32_t batch, n_kv_heads, group_size, head_dim;
  int32_t block_size, cmp_kernel, cmp_stride;
  int32_t n_init, n_local, k_total;
  int64_t t_cap, nc_cap;
} ref_shape;

/* Threads of the OpenMP loops over independent rows (the CPU baseline times the oracle on one
 * thread and on every host core).  Returns the count in effect; n < 1 leaves it unchanged. */
int sparda_ref_set_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

/* ---- bf16 <-> float64 ------------------------------------------------------------------ */

double sparda_ref_bf16_to_f64(uint16_t h) {
  uint32_t u = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Round a float64 straight to the nearest bf16, ties to even (no intermediate float32 step, so
 * no double rounding).  bf16 has 8 significant bits, 8 exponent bits (bias 127). */
uint16_t sparda_ref_f64_to_bf16(double x) {
  uint16_t sign = signbit(x) ? 0x8000u : 0u;
  double a = fabs(x);
  if (isnan(x)) return (uint16_t)(sign | 0x7FC0u);
  if (a == 0.0) return sign;
  if (isinf(x)) return (uint16_t)(sign | 0x7F80u);
  int e;
  double m = frexp(a, &e);             /* a = m * 2^e, 0.5 <= m < 1 */
  double q = nearbyint(ldexp(m, 8));   /* 8 significant bits, default mode = ties to even */
  if (q == 256.0) { q = 128.0; e += 1; }
  int biased = e - 1 + 127;            /* a ~= (q/128) * 2^(e-1) */
  if (biased >= 255) return (uint16_t)(sign | 0x7F80u);
  if (biased <= 0) {
    /* subnormal bf16: the grid is 2^-133 (= 2^-126 * 2^-7); q == 128 lands on the smallest
     * normal, whose encoding is 0x0080, so the same formula covers it. */
    double qs = nearbyint(ldexp(a, 133));
    return (uint16_t)(sign | (uint16_t)qs);
  }
  return (uint16_t)(sign | (uint16_t)(biased << 7) | (uint16_t)((int)q - 128));
}

/* ---- shape checks --------------------------------------------------------------------- */

static int check_shape(const ref_shape* s) {
  if (!s) return REF_ERR_INVALID_ARG;
  if (s->batch < 1 || s->n_kv_heads < 1 || s->group_size < 1 || s->head_dim < 1) return REF_ERR_INVALID_ARG;
  if (s->block_size < 1 || s->n_init < 0 || s->n_local < 1) return REF_ERR_INVALID_ARG;
  if (s->k_total < s->n_init + s->n_local) return REF_ERR_INVALID_ARG;
  if (s->t_cap < 1 || s->nc_cap < 0) return REF_ERR_INVALID_ARG;
  /* every complete block must hold a complete window: windows no longer than a block, stride
   * dividing the block */
  if (s->cmp_stride < 1 || s->cmp_kernel < s->cmp_stride || s->cmp_kernel > s->block_size ||
      s->block_size % s->cmp_stride != 0)
    return REF_ERR_UNSUPPORTED;
  return REF_OK;
}

/* ---- Eq. 2: mean-pooled compressed keys ------------------------------------------------- */

/* k: bf16 [B][Hkv][t_cap][D];  k_cmp: bf16 [B][Hkv][nc_cap][D].
 * Writes K~_i for windows i in [w_begin, w_end); each window [i s_C, i s_C + l_C) must be
 * complete inside t_ctx. */
int sparda_ref_compress_keys(const ref_shape* s, const uint16_t* k, int64_t t_ctx, int32_t w_begin,
                             int32_t w_end, uint16_t* k_cmp) {
  int rc = check_shape(s);
  if (rc) return rc;
  const int64_t lw = s->cmp_kernel, sw = s->cmp_stride, D = s->head_dim;
  if (w_begin < 0 || w_end < w_begin || (int64_t)w_end > s->nc_cap) return REF_ERR_INVALID_ARG;
  if (w_end > w_begin && ((int64_t)(w_end - 1) * sw + lw > t_ctx || t_ctx > s->t_cap)) return REF_ERR_INVALID_ARG;
  const int64_t nrows = (int64_t)s->batch * s->n_kv_heads;
#pragma omp parallel for schedule(static)
  for (int64_t bm = 0; bm < nrows; ++bm) {
    const uint16_t* kh = k + bm * s->t_cap * D;
    uint16_t* ch = k_cmp + bm * s->nc_cap * D;
    for (int64_t i = w_begin; i < w_end; ++i) {
      for (int64_t d = 0; d < D; ++d) {
        double sum = 0.0;
        for (int64_t t = i * sw; t < i * sw + lw; ++t) sum += sparda_ref_bf16_to_f64(kh[t * D + d]);
        ch[i * D + d] = sparda_ref_f64_to_bf16(sum / (double)lw);
      }
    }
  }
  return REF_OK;
}

/* ---- Eq. 1 / Eq. 4: forced blocks, candidates, top-k ------------------------------------- */

typedef struct {
  double score;
  int32_t block;
} scored_block;

/* Order: higher score first, then lower block index first. */
static int by_score_then_index(const void* pa, const void* pb) {
  const scored_block* a = (const scored_block*)pa;
  const scored_block* b = (const scored_block*)pb;
  if (a->score > b->score) return -1;
  if (a->score < b->score) return 1;
  return (a->block > b->block) - (a->block < b->block);
}

/* The score of compressed-key window i for one query row. */
typedef double (*window_score_fn)(const void* ctx, int64_t i);

/* Eq. 4: the Forecast row of the group dotted with window i's compressed key. */
typedef struct {
  const uint16_t* frow;
  const uint16_t* kc;
  int64_t D;
} forecast_ctx;

static double forecast_window_score(const void* vctx, int64_t i) {
  const forecast_ctx* c = (const forecast_ctx*)vctx;
  const int64_t D = c->D;
  const uint16_t* frow = c->frow;
  const uint16_t* kc = c->kc;
  double dot = 0.0;
  for (int64_t d = 0; d < D; ++d) dot += sparda_ref_bf16_to_f64(frow[d]) * sparda_ref_bf16_to_f64(kc[i * D + d]);
  return dot;
}

/* The windows whose scores block j max-pools at a query whose last complete window is w_vis:
 * every window overlapping the block's tokens [j L, (j + 1) L), i s_C < (j + 1) L and
 * i s_C + l_C > j L, that is complete at the query (Sec. 3; the footprint and visibility
 * readings).  The range [*i_lo, *i_hi] is empty when *i_hi < *i_lo. */
static void block_windows(const ref_shape* s, int64_t j, int64_t w_vis, int64_t* i_lo, int64_t* i_hi) {
  const int64_t L = s->block_size, lw = s->cmp_kernel, sw = s->cmp_stride;
  int64_t lo = (j * L - lw) / sw + 1;
  if (j * L - lw < 0) lo = 0;
  int64_t hi = ((j + 1) * L - 1) / sw;
  if (hi > w_vis) hi = w_vis;
  *i_lo = lo;
  *i_hi = hi;
}

/* Selection of one row at position p from window scores (Eq. 1 with the max-pool and top-k of
 * the InfLLM-V2 selector): the outputs are those of sparda_ref_select_row. */
static int select_pooled(const ref_shape* s, int64_t p, window_score_fn score, const void* ctx, int16_t* sel_row,
                         int16_t* cnt, double* scores, int32_t* wins) {
  const int64_t L = s->block_size, lw = s->cmp_kernel, sw = s->cmp_stride;
  const int64_t blk = p / L;

  /* forced(p): the initial blocks and the local window [blk - n_local + 1, blk]. */
  const int64_t init_hi = (s->n_init < blk + 1) ? s->n_init : blk + 1;  /* init = [0, init_hi) */
  int64_t local_lo = blk - s->n_local + 1;
  if (local_lo < 0) local_lo = 0;
  if (local_lo < init_hi) local_lo = init_hi;                            /* drop duplicates */
  const int64_t n_forced = init_hi + (blk - local_lo + 1);

  /* candidates: complete blocks that are neither initial nor local. */
  const int64_t cand_lo = s->n_init, cand_hi = blk - s->n_local;        /* inclusive */
  const int64_t n_cand = (cand_hi >= cand_lo) ? cand_hi - cand_lo + 1 : 0;
  const int64_t n_sel_budget = s->k_total - n_forced;
  if (n_sel_budget < 0) return REF_ERR_INVALID_ARG;
  const int64_t n_take = n_sel_budget < n_cand ? n_sel_budget : n_cand;
  /* windows complete at position p: i s_C + l_C <= p + 1 */
  const int64_t w_vis = (p + 1 - lw) >= 0 ? (p + 1 - lw) / sw : -1;     /* last visible window */

  const int64_t n_blk_cap = (s->t_cap + L - 1) / L;
  if (scores)
    for (int64_t j = 0; j < n_blk_cap; ++j) scores[j] = NAN;
  if (wins)
    for (int64_t j = 0; j < n_blk_cap; ++j) wins[j] = -1;

  scored_block* list = (scored_block*)malloc(sizeof(scored_block) * (size_t)(n_cand > 0 ? n_cand : 1));
  if (!list) return REF_ERR_INVALID_ARG;
  for (int64_t c = 0; c < n_cand; ++c) {
    const int64_t j = cand_lo + c;
    int64_t i_lo, i_hi;
    block_windows(s, j, w_vis, &i_lo, &i_hi);
    if (i_hi >= s->nc_cap) { free(list); return REF_ERR_INVALID_ARG; }
    double best = -INFINITY;
    int64_t best_i = -1;
    for (int64_t i = i_lo; i <= i_hi; ++i) {
      const double x = score(ctx, i);
      if (x > best) { best = x; best_i = i; }
    }
    list[c].score = best;
    list[c].block = (int32_t)j;
    if (scores) scores[j] = best;
    if (wins) wins[j] = (int32_t)best_i;
  }
  qsort(list, (size_t)n_cand, sizeof(scored_block), by_score_then_index);

  /* Emit forced U chosen in ascending order.  A membership table over [0, blk] keeps this a
   * plain set union rather than a merge. */
  unsigned char* in_set = (unsigned char*)calloc((size_t)(blk + 1), 1);
  if (!in_set) { free(list); return REF_ERR_INVALID_ARG; }
  for (int64_t j = 0; j < init_hi; ++j) in_set[j] = 1;
  for (int64_t j = local_lo; j <= blk; ++j) in_set[j] = 1;
  for (int64_t c = 0; c < n_take; ++c) in_set[list[c].block] = 1;
  int64_t n = 0;
  for (int64_t j = 0; j <= blk; ++j)
    if (in_set[j]) sel_row[n++] = (int16_t)j;
  for (int64_t i = n; i < s->k_total; ++i) sel_row[i] = -1;
  *cnt = (int16_t)n;
  free(in_set);
  free(list);
  return REF_OK;
}

/* One query row (batch b, group m, row r at position p = q_pos0 + r).
 *   f: bf16 [B][Hkv][n_q][D]; k_cmp: bf16 [B][Hkv][nc_cap][D] (compressed-key windows)
 *   sel_row: k_total entries, ascending block indices, -1 padded; cnt: number of valid entries.
 *   scores (optional, one double per block of the capacity, ceil(t_cap / block) of them): the
 *   max-pooled Forecast score of every candidate block, NaN for a block that is not a candidate.
 *   wins (optional, same length): the lowest window index reaching that score, -1 elsewhere. */
int sparda_ref_select_row(const ref_shape* s, const uint16_t* f, int32_t n_q, int64_t q_pos0,
                          const uint16_t* k_cmp, int32_t b, int32_t m, int32_t r, int16_t* sel_row,
                          int16_t* cnt, double* scores, int32_t* wins) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (b < 0 || b >= s->batch || m < 0 || m >= s->n_kv_heads || r < 0 || r >= n_q) return REF_ERR_INVALID_ARG;
  const int64_t D = s->head_dim;
  const int64_t p = q_pos0 + r;
  if (p < 0 || p >= s->t_cap) return REF_ERR_INVALID_ARG;
  forecast_ctx ctx;
  ctx.frow = f + (((int64_t)b * s->n_kv_heads + m) * n_q + r) * D;
  ctx.kc = k_cmp + ((int64_t)b * s->n_kv_heads + m) * s->nc_cap * D;
  ctx.D = D;
  return select_pooled(s, p, forecast_window_score, &ctx, sel_row, cnt, scores, wins);
}

/* The InfLLM-V2 selector's shared score of window i: the sum over the group's heads of each
 * head's softmax weight on window i, precomputed for every window complete at the query. */
static double shared_window_score(const void* vctx, int64_t i) { return ((const double*)vctx)[i]; }

/* One query row of the multi-head selector (batch b, group m, row r at p = q_pos0 + r).
 *   q: bf16 [B][Hq][n_q][D], heads m G .. m G + G - 1 belong to group m; k_cmp as above, holding
 *   every window complete at p (nc_cap > the last of them, else INVALID_ARG).
 *   For head h: z_i = sm_scale q_h . K~_i over the windows complete at p, a_i = softmax(z)_i;
 *   window i's shared score is the sum of a_i over the G heads.  Block scores are the max-pool of
 *   the shared scores, and the selection is that of sparda_ref_select_row with them (scores /
 *   wins report them the same way). */
int sparda_ref_multihead_select_row(const ref_shape* s, const uint16_t* q, int32_t n_q, int64_t q_pos0,
                                    const uint16_t* k_cmp, double sm_scale, int32_t b, int32_t m, int32_t r,
                                    int16_t* sel_row, int16_t* cnt, double* scores, int32_t* wins) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (b < 0 || b >= s->batch || m < 0 || m >= s->n_kv_heads || r < 0 || r >= n_q) return REF_ERR_INVALID_ARG;
  if (!(sm_scale > 0.0) || !isfinite(sm_scale)) return REF_ERR_INVALID_ARG;
  const int64_t D = s->head_dim, G = s->group_size, lw = s->cmp_kernel, sw = s->cmp_stride;
  const int64_t p = q_pos0 + r;
  if (p < 0 || p >= s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t n_vis = (p + 1 - lw) >= 0 ? (p + 1 - lw) / sw + 1 : 0;  /* windows 0 .. n_vis - 1 */
  if (n_vis > s->nc_cap) return REF_ERR_INVALID_ARG;
  const uint16_t* keys = k_cmp + ((int64_t)b * s->n_kv_heads + m) * s->nc_cap * D;
  double* shared = (double*)calloc((size_t)(n_vis > 0 ? n_vis : 1), sizeof(double));
  double* z = (double*)malloc(sizeof(double) * (size_t)(n_vis > 0 ? n_vis : 1));
  if (!shared || !z) { free(shared); free(z); return REF_ERR_INVALID_ARG; }
  for (int64_t h = m * G; h < (m + 1) * G; ++h) {
    const uint16_t* qrow = q + (((int64_t)b * s->n_kv_heads * G + h) * n_q + r) * D;
    double zmax = -INFINITY;
    for (int64_t i = 0; i < n_vis; ++i) {
      double acc = 0.0;
      for (int64_t e = 0; e < D; ++e) acc += sparda_ref_bf16_to_f64(qrow[e]) * sparda_ref_bf16_to_f64(keys[i * D + e]);
      z[i] = sm_scale * acc;
      if (z[i] > zmax) zmax = z[i];
    }
    double denom = 0.0;
    for (int64_t i = 0; i < n_vis; ++i) denom += exp(z[i] - zmax);
    for (int64_t i = 0; i < n_vis; ++i) shared[i] += exp(z[i] - zmax) / denom;
  }
  free(z);
  rc = select_pooled(s, p, shared_window_score, shared, sel_row, cnt, scores, wins);
  free(shared);
  return rc;
}

/* All rows.  sel: int16 [B][Hkv][n_q][k_total]; cnt: int16 [B][Hkv][n_q]. */
int sparda_ref_forecast_select(const ref_shape* s, const uint16_t* f, int32_t n_q, int64_t q_pos0,
                               const uint16_t* k_cmp, int16_t* sel, int16_t* cnt) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (n_q < 1) return REF_ERR_INVALID_ARG;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  int err = REF_OK;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = 0; i < rows; ++i) {
    const int32_t r = (int32_t)(i % n_q);
    const int32_t m = (int32_t)((i / n_q) % s->n_kv_heads);
    const int32_t b = (int32_t)(i / ((int64_t)n_q * s->n_kv_heads));
    int e = sparda_ref_select_row(s, f, n_q, q_pos0, k_cmp, b, m, r, sel + i * s->k_total, cnt + i, NULL, NULL);
    if (e) {
#pragma omp critical
      err = e;
    }
  }
  return err;
}

/* Each row's largest candidate score: the Eq. 4 scores of sparda_ref_forecast_select's
 * candidates [n_init, blk(p) - n_local], max-pooled per block as there, reduced to their maximum
 * (-inf when the row has no candidate).  It is the scoring of the selection without its top-k.
 * row_max: double [B][Hkv][n_q]. */
int sparda_ref_forecast_score_max(const ref_shape* s, const uint16_t* f, int32_t n_q, int64_t q_pos0,
                                  const uint16_t* k_cmp, double* row_max) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (n_q < 1 || q_pos0 < 0 || q_pos0 + n_q > s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t L = s->block_size, lw = s->cmp_kernel, sw = s->cmp_stride, D = s->head_dim;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  int err = REF_OK;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t row = 0; row < rows; ++row) {
    const int64_t bm = row / n_q, p = q_pos0 + row % n_q;
    forecast_ctx ctx;
    ctx.frow = f + row * D;
    ctx.kc = k_cmp + bm * s->nc_cap * D;
    ctx.D = D;
    const int64_t w_vis = (p + 1 - lw) >= 0 ? (p + 1 - lw) / sw : -1;
    double best = -INFINITY;
    for (int64_t j = s->n_init; j <= p / L - s->n_local; ++j) {
      int64_t i_lo, i_hi;
      block_windows(s, j, w_vis, &i_lo, &i_hi);
      if (i_hi >= s->nc_cap) {
#pragma omp critical
        err = REF_ERR_INVALID_ARG;
        break;
      }
      for (int64_t i = i_lo; i <= i_hi; ++i) {
        const double x = forecast_window_score(&ctx, i);
        if (x > best) best = x;
      }
    }
    row_max[row] = best;
  }
  return err;
}

/* All rows of the multi-head selector.  sel: int16 [B][Hkv][n_q][k_total]; cnt: int16 [B][Hkv][n_q]. */
int sparda_ref_multihead_select(const ref_shape* s, const uint16_t* q, int32_t n_q, int64_t q_pos0,
                                const uint16_t* k_cmp, double sm_scale, int16_t* sel, int16_t* cnt) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (n_q < 1) return REF_ERR_INVALID_ARG;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  int err = REF_OK;
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = 0; i < rows; ++i) {
    const int32_t r = (int32_t)(i % n_q);
    const int32_t m = (int32_t)((i / n_q) % s->n_kv_heads);
    const int32_t b = (int32_t)(i / ((int64_t)n_q * s->n_kv_heads));
    int e = sparda_ref_multihead_select_row(s, q, n_q, q_pos0, k_cmp, sm_scale, b, m, r, sel + i * s->k_total,
                                            cnt + i, NULL, NULL);
    if (e) {
#pragma omp critical
      err = e;
    }
  }
  return err;
}

/* ---- Eq. 1 / Eq. 5: attention over the attended blocks ---------------------------------- */

/* One (batch b, query head h, row r).  q: bf16 [B][Hq][n_q][D].
 * kv_mode 0: k, v are full caches bf16 [B][Hkv][t_cap][D], token t at row t.
 * kv_mode 1: k, v are staging buffers bf16 [B][Hkv][k_total][block][D] for a single query row
 *            (n_q == 1); slot s holds the tokens of block sel[s].
 * sel/cnt as produced by select; an entry outside [0, blk(p)] is skipped.  Tokens after p are
 * never attended.  out: D doubles; all zeros when no token is attended. */
int sparda_ref_attend_row(const ref_shape* s, const uint16_t* q, int32_t n_q, int64_t q_pos0,
                          const uint16_t* k, const uint16_t* v, int32_t kv_mode, const int16_t* sel,
                          const int16_t* cnt, double sm_scale, int32_t b, int32_t h, int32_t r, double* out) {
  int rc = check_shape(s);
  if (rc) return rc;
  const int64_t D = s->head_dim, L = s->block_size, G = s->group_size;
  const int64_t Hq = (int64_t)s->n_kv_heads * G;
  if (b < 0 || b >= s->batch || h < 0 || h >= Hq || r < 0 || r >= n_q) return REF_ERR_INVALID_ARG;
  if (kv_mode != 0 && kv_mode != 1) return REF_ERR_INVALID_ARG;
  if (kv_mode == 1 && n_q != 1) return REF_ERR_INVALID_ARG;
  const int64_t p = q_pos0 + r;
  if (p < 0 || p >= s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t blk = p / L;
  const int64_t m = h / G;  /* consecutive query heads share a KV head */
  const int64_t row = ((int64_t)b * s->n_kv_heads + m) * n_q + r;
  const int16_t* srow = sel + row * s->k_total;
  int64_t n_sel = cnt[row];
  if (n_sel > s->k_total) n_sel = s->k_total;

  const uint16_t* qrow = q + (((int64_t)b * Hq + h) * n_q + r) * D;
  /* Collect the attended tokens as (pointer to key row, pointer to value row). */
  const int64_t max_tok = n_sel * L;
  const uint16_t** krows = (const uint16_t**)malloc(sizeof(void*) * (size_t)(max_tok > 0 ? max_tok : 1));
  const uint16_t** vrows = (const uint16_t**)malloc(sizeof(void*) * (size_t)(max_tok > 0 ? max_tok : 1));
  double* z = (double*)malloc(sizeof(double) * (size_t)(max_tok > 0 ? max_tok : 1));
  if (!krows || !vrows || !z) { free(krows); free(vrows); free(z); return REF_ERR_INVALID_ARG; }
  int64_t n_tok = 0;
  for (int64_t sidx = 0; sidx < n_sel; ++sidx) {
    const int64_t j = srow[sidx];
    if (j < 0 || j > blk) continue;
    /* The attended tokens are a union over the set's blocks (Eq. 1, Eq. 5): a block listed
     * twice contributes its tokens once, through its first entry. */
    int seen = 0;
    for (int64_t e = 0; e < sidx; ++e) seen |= (srow[e] == j);
    if (seen) continue;
    for (int64_t i = 0; i < L; ++i) {
      const int64_t t = j * L + i;
      if (t > p) break;
      if (kv_mode == 0) {
        const int64_t base = (((int64_t)b * s->n_kv_heads + m) * s->t_cap + t) * D;
        krows[n_tok] = k + base;
        vrows[n_tok] = v + base;
      } else {
        const int64_t base = ((((int64_t)b * s->n_kv_heads + m) * s->k_total + sidx) * L + i) * D;
        krows[n_tok] = k + base;
        vrows[n_tok] = v + base;
      }
      ++n_tok;
    }
  }
  for (int64_t d = 0; d < D; ++d) out[d] = 0.0;
  if (n_tok > 0) {
    double zmax = -INFINITY;
    for (int64_t t = 0; t < n_tok; ++t) {
      double dot = 0.0;
      for (int64_t d = 0; d < D; ++d) dot += sparda_ref_bf16_to_f64(qrow[d]) * sparda_ref_bf16_to_f64(krows[t][d]);
      z[t] = sm_scale * dot;
      if (z[t] > zmax) zmax = z[t];
    }
    double denom = 0.0;
    for (int64_t t = 0; t < n_tok; ++t) {
      z[t] = exp(z[t] - zmax);
      denom += z[t];
    }
    for (int64_t t = 0; t < n_tok; ++t) {
      const double w = z[t] / denom;
      for (int64_t d = 0; d < D; ++d) out[d] += w * sparda_ref_bf16_to_f64(vrows[t][d]);
    }
  }
  free(krows);
  free(vrows);
  free(z);
  return REF_OK;
}

/* All (b, h, r).  o: float64 [B][Hq][n_q][D]. */
int sparda_ref_sparse_attn(const ref_shape* s, const uint16_t* q, int32_t n_q, int64_t q_pos0, const uint16_t* k,
                           const uint16_t* v, int32_t kv_mode, const int16_t* sel, const int16_t* cnt,
                           double sm_scale, double* o) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (n_q < 1) return REF_ERR_INVALID_ARG;
  const int64_t Hq = (int64_t)s->n_kv_heads * s->group_size;
  const int64_t rows = (int64_t)s->batch * Hq * n_q;
  int err = REF_OK;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t i = 0; i < rows; ++i) {
    const int32_t r = (int32_t)(i % n_q);
    const int32_t h = (int32_t)((i / n_q) % Hq);
    const int32_t b = (int32_t)(i / ((int64_t)n_q * Hq));
    int e = sparda_ref_attend_row(s, q, n_q, q_pos0, k, v, kv_mode, sel, cnt, sm_scale, b, h, r,
                                  o + i * s->head_dim);
    if (e) {
#pragma omp critical
      err = e;
    }
  }
  return err;
}

/* ---- Sec. 4.3 / Alg. 2: copy selected blocks into staging ------------------------------- */

/* host_k/host_v: bf16 [B][Hkv][t_cap][D]; sel/cnt from a single-row select ([B][Hkv][k_total],
 * [B][Hkv]); stage_k/stage_v: bf16 [B][Hkv][k_total][block][D].  Slot s < cnt receives the whole
 * block sel[s]; other slots and entries whose block lies outside the cache are left untouched. */
int sparda_ref_gather_blocks(const ref_shape* s, const uint16_t* host_k, const uint16_t* host_v,
                             const int16_t* sel, const int16_t* cnt, uint16_t* stage_k, uint16_t* stage_v) {
  int rc = check_shape(s);
  if (rc) return rc;
  const int64_t D = s->head_dim, L = s->block_size;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads;
  for (int64_t bm = 0; bm < rows; ++bm) {
    int64_t n = cnt[bm];
    if (n > s->k_total) n = s->k_total;
    for (int64_t sidx = 0; sidx < n; ++sidx) {
      const int64_t j = sel[bm * s->k_total + sidx];
      if (j < 0 || (j + 1) * L > s->t_cap) continue;
      const size_t bytes = (size_t)(L * D) * sizeof(uint16_t);
      memcpy(stage_k + (bm * s->k_total + sidx) * L * D, host_k + (bm * s->t_cap + j * L) * D, bytes);
      memcpy(stage_v + (bm * s->k_total + sidx) * L * D, host_v + (bm * s->t_cap + j * L) * D, bytes);
    }
  }
  return REF_OK;
}

/* Sec. 5.3 (Efficiency Results, prefill throughput): the write-back of newly created KV rows
 * into the host pools.  k_new, v_new: bf16 [B][Hkv][n_new][D]; the rows land at positions pos0 .. pos0 + n_new - 1 of the pools
 * host_k, host_v: bf16 [B][Hkv][t_cap][D]; nothing else is written. */
int sparda_ref_writeback_kv(const ref_shape* s, const uint16_t* k_new, const uint16_t* v_new, int32_t n_new,
                            int64_t pos0, uint16_t* host_k, uint16_t* host_v) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (n_new < 1 || pos0 < 0 || pos0 + n_new > s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t D = s->head_dim;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads;
  for (int64_t bm = 0; bm < rows; ++bm)
    for (int64_t t = 0; t < n_new; ++t) {
      memcpy(host_k + (bm * s->t_cap + pos0 + t) * D, k_new + (bm * n_new + t) * D, (size_t)D * sizeof(uint16_t));
      memcpy(host_v + (bm * s->t_cap + pos0 + t) * D, v_new + (bm * n_new + t) * D, (size_t)D * sizeof(uint16_t));
    }
  return REF_OK;
}

/* Alg. 2 (decode step): the token decoded at position q_pos is appended to the KV cache.  In an
 * offloaded layer the attended blocks were copied to staging before the token existed (the
 * prefetch of B_l is launched during layer l-1), so the token's K/V row is written into every
 * staging slot s < cnt whose block sel[s] is the token's own block q_pos / L, at row q_pos mod L.
 * k_new, v_new: bf16 [B][Hkv][D]; sel, cnt: decode-form [B][Hkv][k_total] and [B][Hkv];
 * stage_k, stage_v: bf16 [B][Hkv][k_total][L][D].  Nothing else is written. */
int sparda_ref_stage_append_kv(const ref_shape* s, const uint16_t* k_new, const uint16_t* v_new, int64_t q_pos,
                               const int16_t* sel, const int16_t* cnt, uint16_t* stage_k, uint16_t* stage_v) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (q_pos < 0 || q_pos >= s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t D = s->head_dim, L = s->block_size, K = s->k_total;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads;
  const int64_t j = q_pos / L, t = q_pos % L;
  for (int64_t bm = 0; bm < rows; ++bm) {
    int64_t n = cnt[bm];
    if (n > K) n = K;
    for (int64_t slot = 0; slot < n; ++slot) {
      if (sel[bm * K + slot] != j) continue;
      memcpy(stage_k + ((bm * K + slot) * L + t) * D, k_new + bm * D, (size_t)D * sizeof(uint16_t));
      memcpy(stage_v + ((bm * K + slot) * L + t) * D, v_new + bm * D, (size_t)D * sizeof(uint16_t));
    }
  }
  return REF_OK;
}

/* ---- App. C (NOSI step reuse): staging plan of one decode step ------------------------------- */

/* A layer's staging buffer is a cache of k_total slots per (batch, group) row.  Slot s holds the
 * first slot_len[s] tokens of block slot_blk[s] (-1: empty), as fetched by an earlier step.  Tokens
 * never change once written, so a staged block still serves the query at position p exactly when
 * its staged prefix covers every token of the block up to p: need(j) = min(L, p + 1 - j L).
 *
 * For the new attended set S (sel/cnt of a single-row select at position q_pos):
 *   kept    -- slots holding a block of S with slot_len >= need: unchanged, no copy;
 *   missing -- the blocks of S that no kept slot holds, in ascending block order;
 *   free    -- every other slot, in ascending slot order; the r-th missing block goes to the r-th
 *              free slot (fetch[s] = block, slot_blk = block, slot_len = need) and the free slots
 *              left over are emptied (slot_blk = -1, slot_len = 0);
 *   sel_staged[s] = the block slot s holds for this step's attention, -1 when it holds none of S.
 * Only blocks attended by the previous step are ever kept: a slot that S does not use is emptied.
 * fetch[s] = -1 for every slot that needs no copy; n_fetch[row] = number of missing blocks.
 * Arrays are [B][Hkv][k_total] int16 ([B][Hkv] int32 for n_fetch); slot_blk / slot_len are read
 * and updated in place.  Start from slot_blk = -1 everywhere. */
int sparda_ref_plan_staging(const ref_shape* s, const int16_t* sel, const int16_t* cnt, int64_t q_pos,
                            int16_t* slot_blk, int16_t* slot_len, int16_t* fetch, int16_t* sel_staged,
                            int32_t* n_fetch) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (q_pos < 0 || q_pos >= s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t L = s->block_size, K = s->k_total;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads;
  unsigned char* kept = (unsigned char*)malloc((size_t)K);
  unsigned char* held = (unsigned char*)malloc((size_t)K);
  if (!kept || !held) { free(kept); free(held); return REF_ERR_INVALID_ARG; }
  for (int64_t row = 0; row < rows; ++row) {
    const int16_t* srow = sel + row * K;
    int16_t* blk = slot_blk + row * K;
    int16_t* len = slot_len + row * K;
    int16_t* fet = fetch + row * K;
    int16_t* att = sel_staged + row * K;
    int64_t n = cnt[row];
    if (n < 0 || n > K) { free(kept); free(held); return REF_ERR_INVALID_ARG; }
    /* kept slots, and which entries of S they hold */
    for (int64_t i = 0; i < K; ++i) held[i] = 0;
    for (int64_t t = 0; t < K; ++t) {
      kept[t] = 0;
      if (blk[t] < 0) continue;
      const int64_t j = blk[t];
      int64_t need = q_pos + 1 - j * L;
      if (need > L) need = L;
      for (int64_t i = 0; i < n; ++i) {
        if (srow[i] == j && !held[i] && len[t] >= need) {
          kept[t] = 1;
          held[i] = 1;
          break;
        }
      }
    }
    /* missing blocks in ascending order (S is ascending) into free slots in ascending order */
    int64_t next_free = 0, fetched = 0;
    for (int64_t t = 0; t < K; ++t) {
      fet[t] = -1;
      att[t] = kept[t] ? blk[t] : -1;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (held[i] || srow[i] < 0) continue;
      while (next_free < K && kept[next_free]) ++next_free;
      if (next_free >= K) { free(kept); free(held); return REF_ERR_INVALID_ARG; }
      const int64_t j = srow[i];
      int64_t need = q_pos + 1 - j * L;
      if (need > L) need = L;
      fet[next_free] = (int16_t)j;
      att[next_free] = (int16_t)j;
      blk[next_free] = (int16_t)j;
      len[next_free] = (int16_t)need;
      kept[next_free] = 1; /* taken */
      ++next_free;
      ++fetched;
    }
    for (int64_t t = 0; t < K; ++t) {
      if (att[t] < 0) {
        blk[t] = -1;
        len[t] = 0;
      }
    }
    n_fetch[row] = (int32_t)fetched;
  }
  free(kept);
  free(held);
  return REF_OK;
}

/* ---- Sec. 4.2, Eq. 6-7: the indexer-training loss of one query row --------------------------- */

/* One query row (batch b, group m, row r at position p = q_pos0 + r).
 *   s          : shape; cmp_kernel / cmp_stride give the prediction grid (l_P, s_P), normally
 *                (32, 16); group_size G heads per group; n_init / n_local the forced blocks.
 *   q          : bf16 [B][Hq][n_q][D] attention queries of the target layer.
 *   kc_tgt     : bf16 [B][Hkv][nt_cap][D] target compressed keys on the grid (lt, st), normally
 *                (2, 1): window i covers tokens [i st, i st + lt).
 *   f          : bf16 [B][Hkv][n_q][D] Forecast rows (of the previous layer).
 *   kc_pred    : bf16 [B][Hkv][nc_cap][D] prediction compressed keys on the grid (l_P, s_P).
 *   sm_scale   : 1 / tau for both softmaxes.
 *   k_top      : size of the target's selected set.
 * Definitions:
 *   positions  w = 0 .. N-1: the prediction windows complete at p (w s_P + l_P <= p + 1).
 *   target     for each head h of the group, a_h = softmax over the target windows complete at p
 *              of sm_scale q_h . K~tgt_i; the shared score is sum_h a_h,i; T_w = the largest shared
 *              score of the target windows lying inside position w's tokens (i st >= w s_P and
 *              i st + lt <= w s_P + l_P).
 *   predicted  P = softmax over w < N of sm_scale F . K~pred_w.
 *   selected   S = the k_top largest T_w (ties: lower w) among the positions whose tokens lie in
 *              candidate blocks [n_init, blk(p) - n_local] (init and local blocks excluded).
 *   buckets    t_c = T_c / sum_w T_w for c in S and t_rest = the rest of the target mass;
 *              P_c for c in S and R = 1 - sum_S P_c (the predicted rest).
 *   loss       KL(t || p) = sum_c t_c log(t_c / P_c) + t_rest log(t_rest / R), 0 log 0 = 0.
 *   gradient   d loss / d z_w (z_w = sm_scale F . K~pred_w): P_w - t_w for w in S and
 *              P_w (1 - t_rest / R) for the other positions; dF = sm_scale sum_w grad_w K~pred_w.
 * Outputs: *loss, dF[D] (optional), sel[k_top] (optional: the selected positions ascending, -1
 * padded) and *n_sel. */
int sparda_ref_indexer_kl_row(const ref_shape* s, const uint16_t* q, const uint16_t* kc_tgt, int64_t nt_cap,
                              int32_t lt, int32_t st, const uint16_t* f, const uint16_t* kc_pred, int32_t n_q,
                              int64_t q_pos0, double sm_scale, int32_t k_top, int32_t b, int32_t m, int32_t r,
                              double* loss, double* dF, int32_t* sel, int32_t* n_sel) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (b < 0 || b >= s->batch || m < 0 || m >= s->n_kv_heads || r < 0 || r >= n_q || k_top < 0) return REF_ERR_INVALID_ARG;
  if (lt < 1 || st < 1 || !(sm_scale > 0.0)) return REF_ERR_INVALID_ARG;
  const int64_t D = s->head_dim, G = s->group_size, L = s->block_size, lp = s->cmp_kernel, sp_ = s->cmp_stride;
  const int64_t p = q_pos0 + r;
  if (p < 0 || p >= s->t_cap) return REF_ERR_INVALID_ARG;
  const int64_t n_pos = (p + 1 - lp) >= 0 ? (p + 1 - lp) / sp_ + 1 : 0;  /* positions 0 .. n_pos - 1 */
  const int64_t n_tw = (p + 1 - lt) >= 0 ? (p + 1 - lt) / st + 1 : 0;    /* target windows complete at p */
  if (n_pos > s->nc_cap || n_tw > nt_cap) return REF_ERR_INVALID_ARG;
  const int64_t bm = (int64_t)b * s->n_kv_heads + m;
  const uint16_t* kt = kc_tgt + bm * nt_cap * D;
  const uint16_t* kp = kc_pred + bm * s->nc_cap * D;
  const uint16_t* frow = f + (bm * n_q + r) * D;
  double* shared = (double*)calloc((size_t)(n_tw > 0 ? n_tw : 1), sizeof(double));
  double* z = (double*)malloc(sizeof(double) * (size_t)((n_tw > n_pos ? n_tw : n_pos) + 1));
  double* T = (double*)malloc(sizeof(double) * (size_t)(n_pos + 1));
  double* P = (double*)malloc(sizeof(double) * (size_t)(n_pos + 1));
  scored_block* list = (scored_block*)malloc(sizeof(scored_block) * (size_t)(n_pos + 1));
  unsigned char* in_s = (unsigned char*)calloc((size_t)(n_pos + 1), 1);
  if (!shared || !z || !T || !P || !list || !in_s) {
    free(shared); free(z); free(T); free(P); free(list); free(in_s);
    return REF_ERR_INVALID_ARG;
  }
  /* target: per-head softmax over the fine windows, summed over the group */
  for (int64_t hg = 0; hg < G; ++hg) {
    const uint16_t* qh = q + (((int64_t)b * s->n_kv_heads * G + m * G + hg) * n_q + r) * D;
    double zmax = -INFINITY;
    for (int64_t i = 0; i < n_tw; ++i) {
      double acc = 0.0;
      for (int64_t e = 0; e < D; ++e) acc += sparda_ref_bf16_to_f64(qh[e]) * sparda_ref_bf16_to_f64(kt[i * D + e]);
      z[i] = acc * sm_scale;
      if (z[i] > zmax) zmax = z[i];
    }
    double den = 0.0;
    for (int64_t i = 0; i < n_tw; ++i) den += exp(z[i] - zmax);
    for (int64_t i = 0; i < n_tw; ++i) shared[i] += exp(z[i] - zmax) / den;
  }
  /* max-pool of the shared scores to the prediction positions */
  double t_total = 0.0;
  for (int64_t w = 0; w < n_pos; ++w) {
    double best = 0.0;  /* shared scores are > 0; a position with no inside window pools to 0 */
    for (int64_t i = 0; i < n_tw; ++i)
      if (i * st >= w * sp_ && i * st + lt <= w * sp_ + lp && shared[i] > best) best = shared[i];
    T[w] = best;
    t_total += best;
  }
  /* prediction: softmax of the Forecast scores over the positions */
  double zmax = -INFINITY;
  for (int64_t w = 0; w < n_pos; ++w) {
    double acc = 0.0;
    for (int64_t e = 0; e < D; ++e) acc += sparda_ref_bf16_to_f64(frow[e]) * sparda_ref_bf16_to_f64(kp[w * D + e]);
    z[w] = sm_scale * acc;
    if (z[w] > zmax) zmax = z[w];
  }
  double pden = 0.0;
  for (int64_t w = 0; w < n_pos; ++w) pden += exp(z[w] - zmax);
  for (int64_t w = 0; w < n_pos; ++w) P[w] = exp(z[w] - zmax) / pden;
  /* the target's top-k among positions inside candidate blocks */
  const int64_t blk = p / L, cand_tok_lo = (int64_t)s->n_init * L, cand_tok_hi = (blk - s->n_local + 1) * L;
  int64_t n_c = 0;
  for (int64_t w = 0; w < n_pos; ++w) {
    if (w * sp_ >= cand_tok_lo && w * sp_ + lp <= cand_tok_hi) {
      list[n_c].score = T[w];
      list[n_c].block = (int32_t)w;
      ++n_c;
    }
  }
  qsort(list, (size_t)n_c, sizeof(scored_block), by_score_then_index);
  const int64_t n_take = k_top < n_c ? k_top : n_c;
  for (int64_t c = 0; c < n_take; ++c) in_s[list[c].block] = 1;
  /* buckets, loss and gradient */
  double t_rest = 0.0, R = 0.0, kl = 0.0;
  for (int64_t w = 0; w < n_pos; ++w) {
    if (in_s[w]) {
      const double tc = T[w] / t_total;
      if (tc > 0.0) kl += tc * log(tc / P[w]);
    } else {
      t_rest += T[w] / t_total;
      R += P[w];
    }
  }
  if (t_rest > 0.0) kl += t_rest * log(t_rest / R);
  *loss = n_pos > 0 ? kl : 0.0;
  if (dF) {
    for (int64_t e = 0; e < D; ++e) dF[e] = 0.0;
    for (int64_t w = 0; w < n_pos; ++w) {
      const double g = in_s[w] ? P[w] - T[w] / t_total : (R > 0.0 ? P[w] * (1.0 - t_rest / R) : 0.0);
      for (int64_t e = 0; e < D; ++e) dF[e] += sm_scale * g * sparda_ref_bf16_to_f64(kp[w * D + e]);
    }
  }
  if (sel) {
    int64_t n = 0;
    for (int64_t w = 0; w < n_pos; ++w)
      if (in_s[w]) sel[n++] = (int32_t)w;
    for (int64_t i = n; i < k_top; ++i) sel[i] = -1;
  }
  if (n_sel) *n_sel = (int32_t)n_take;
  free(shared); free(z); free(T); free(P); free(list); free(in_s);
  return REF_OK;
}

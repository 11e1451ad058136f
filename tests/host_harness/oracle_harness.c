/* oracle_harness.c -- runs every function of the CPU oracle (oracle/sparda_oracle.c) on small
 * seeded inputs held in buffers of exactly the documented sizes, so that AddressSanitizer and
 * UndefinedBehaviorSanitizer see any access outside them: both compression grids, ragged context
 * lengths and chunks, sets larger than the candidate range, a multi-step staging plan, the
 * multi-head selector, the score row maximum and the indexer-training loss.  Exit status 0 when
 * every call returned its documented status. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t batch, n_kv_heads, group_size, head_dim;
  int32_t block_size, cmp_kernel, cmp_stride;
  int32_t n_init, n_local, k_total;
  int64_t t_cap, nc_cap;
} ref_shape;

int sparda_ref_compress_keys(const ref_shape*, const uint16_t*, int64_t, int32_t, int32_t, uint16_t*);
int sparda_ref_select_row(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, int32_t, int32_t,
                          int32_t, int16_t*, int16_t*, double*, int32_t*);
int sparda_ref_multihead_select_row(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, double,
                                    int32_t, int32_t, int32_t, int16_t*, int16_t*, double*, int32_t*);
int sparda_ref_forecast_select(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, int16_t*,
                               int16_t*);
int sparda_ref_forecast_score_max(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, double*);
int sparda_ref_multihead_select(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, double,
                                int16_t*, int16_t*);
int sparda_ref_attend_row(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, const uint16_t*,
                          int32_t, const int16_t*, const int16_t*, double, int32_t, int32_t, int32_t, double*);
int sparda_ref_sparse_attn(const ref_shape*, const uint16_t*, int32_t, int64_t, const uint16_t*, const uint16_t*,
                           int32_t, const int16_t*, const int16_t*, double, double*);
int sparda_ref_gather_blocks(const ref_shape*, const uint16_t*, const uint16_t*, const int16_t*, const int16_t*,
                             uint16_t*, uint16_t*);
int sparda_ref_writeback_kv(const ref_shape*, const uint16_t*, const uint16_t*, int32_t, int64_t, uint16_t*,
                            uint16_t*);
int sparda_ref_plan_staging(const ref_shape*, const int16_t*, const int16_t*, int64_t, int16_t*, int16_t*, int16_t*,
                            int16_t*, int32_t*);
int sparda_ref_indexer_kl_row(const ref_shape*, const uint16_t*, const uint16_t*, int64_t, int32_t, int32_t,
                              const uint16_t*, const uint16_t*, int32_t, int64_t, double, int32_t, int32_t, int32_t,
                              int32_t, double*, double*, int32_t*, int32_t*);

static int g_fail = 0;
#define EXPECT(call, want)                                                                  \
  do {                                                                                      \
    int rc_ = (call);                                                                       \
    if (rc_ != (want)) {                                                                    \
      fprintf(stderr, "line %d: %s returned %d, expected %d\n", __LINE__, #call, rc_, want); \
      ++g_fail;                                                                             \
    }                                                                                       \
  } while (0)

static uint64_t g_rng = 88172645463325252ull;
static uint16_t rnd_bf16(void) { /* xorshift64 -> a finite bf16 in about [-4, 4] */
  g_rng ^= g_rng << 13;
  g_rng ^= g_rng >> 7;
  g_rng ^= g_rng << 17;
  const uint16_t sign = (uint16_t)((g_rng >> 20) & 1u) << 15;
  const uint16_t expo = (uint16_t)(120 + (g_rng >> 8) % 9) << 7;
  return (uint16_t)(sign | expo | (uint16_t)(g_rng & 0x7f));
}
static uint16_t* bf16_buf(size_t n) {
  uint16_t* p = (uint16_t*)malloc(n * sizeof(uint16_t));
  for (size_t i = 0; i < n; ++i) p[i] = rnd_bf16();
  return p;
}

static ref_shape shape(int B, int H, int G, int k, int64_t t_cap, int64_t nc_cap, int lw, int sw, int n_init,
                       int n_local) {
  ref_shape s = {B, H, G, 128, 64, lw, sw, n_init, n_local, k, t_cap, nc_cap};
  return s;
}

/* One configuration end to end: compress, select (whole and per row), score maximum, multi-head
 * select, attention (whole and per row, cache and staging), gather, write-back. */
static void run(int B, int H, int G, int k, int64_t T, int64_t t_cap, int n_q, int lw, int sw, int n_init,
                int n_local) {
  const int64_t D = 128, nw = T >= lw ? (T - lw) / sw + 1 : 0, nc_cap = nw > 0 ? nw : 1;
  const ref_shape s = shape(B, H, G, k, t_cap, nc_cap, lw, sw, n_init, n_local);
  const int64_t q_pos0 = T - n_q;
  const size_t rows = (size_t)B * H * n_q;
  uint16_t* kk = bf16_buf((size_t)B * H * t_cap * D);
  uint16_t* vv = bf16_buf((size_t)B * H * t_cap * D);
  uint16_t* f = bf16_buf(rows * D);
  uint16_t* q = bf16_buf(rows * G * D);
  uint16_t* kc = (uint16_t*)malloc((size_t)B * H * nc_cap * D * sizeof(uint16_t));
  int16_t* sel = (int16_t*)malloc(rows * k * sizeof(int16_t));
  int16_t* cnt = (int16_t*)malloc(rows * sizeof(int16_t));
  double* o = (double*)malloc(rows * G * D * sizeof(double));
  double* rmax = (double*)malloc(rows * sizeof(double));
  const int64_t n_blk = (t_cap + 63) / 64;
  double* scores = (double*)malloc(n_blk * sizeof(double));
  int32_t* wins = (int32_t*)malloc(n_blk * sizeof(int32_t));
  int16_t* row = (int16_t*)malloc(k * sizeof(int16_t));
  int16_t rc_cnt;
  double out[128];
  EXPECT(sparda_ref_compress_keys(&s, kk, T, 0, (int32_t)nw, kc), 0);
  EXPECT(sparda_ref_forecast_select(&s, f, n_q, q_pos0, kc, sel, cnt), 0);
  EXPECT(sparda_ref_select_row(&s, f, n_q, q_pos0, kc, B - 1, H - 1, n_q - 1, row, &rc_cnt, scores, wins), 0);
  if (lw == 64 && sw == 64) EXPECT(sparda_ref_forecast_score_max(&s, f, n_q, q_pos0, kc, rmax), 0);
  EXPECT(sparda_ref_multihead_select(&s, q, n_q, q_pos0, kc, 0.0883883476, sel, cnt), 0);
  EXPECT(sparda_ref_multihead_select_row(&s, q, n_q, q_pos0, kc, 0.0883883476, 0, 0, 0, row, &rc_cnt, scores, wins),
         0);
  EXPECT(sparda_ref_forecast_select(&s, f, n_q, q_pos0, kc, sel, cnt), 0);
  EXPECT(sparda_ref_sparse_attn(&s, q, n_q, q_pos0, kk, vv, 0, sel, cnt, 0.0883883476, o), 0);
  EXPECT(sparda_ref_attend_row(&s, q, n_q, q_pos0, kk, vv, 0, sel, cnt, 0.0883883476, B - 1, H * G - 1, n_q - 1,
                               out),
         0);
  if (n_q == 1) { /* staging form: gather the sets, attend from staging, write back a token */
    uint16_t* sk = (uint16_t*)malloc((size_t)B * H * k * 64 * D * sizeof(uint16_t));
    uint16_t* sv = (uint16_t*)malloc((size_t)B * H * k * 64 * D * sizeof(uint16_t));
    memset(sk, 0, (size_t)B * H * k * 64 * D * sizeof(uint16_t));
    memset(sv, 0, (size_t)B * H * k * 64 * D * sizeof(uint16_t));
    EXPECT(sparda_ref_gather_blocks(&s, kk, vv, sel, cnt, sk, sv), 0);
    EXPECT(sparda_ref_sparse_attn(&s, q, 1, q_pos0, sk, sv, 1, sel, cnt, 0.0883883476, o), 0);
    uint16_t* kn = bf16_buf((size_t)B * H * 3 * D);
    uint16_t* vn = bf16_buf((size_t)B * H * 3 * D);
    EXPECT(sparda_ref_writeback_kv(&s, kn, vn, 3, t_cap - 3, kk, vv), 0);
    EXPECT(sparda_ref_writeback_kv(&s, kn, vn, 3, t_cap - 2, kk, vv), -1);
    free(kn);
    free(vn);
    free(sk);
    free(sv);
  }
  free(kk); free(vv); free(f); free(q); free(kc); free(sel); free(cnt); free(o); free(rmax); free(scores);
  free(wins); free(row);
}

/* The staging plan over consecutive decode positions with sets that drift. */
static void plan_steps(void) {
  const int B = 2, H = 3, K = 12;
  const ref_shape s = shape(B, H, 4, K, 8192, 128, 64, 64, 1, 2);
  const size_t n = (size_t)B * H * K;
  int16_t* sel = (int16_t*)malloc(n * sizeof(int16_t));
  int16_t* cnt = (int16_t*)malloc((size_t)B * H * sizeof(int16_t));
  int16_t* blk = (int16_t*)malloc(n * sizeof(int16_t));
  int16_t* len = (int16_t*)malloc(n * sizeof(int16_t));
  int16_t* fetch = (int16_t*)malloc(n * sizeof(int16_t));
  int16_t* staged = (int16_t*)malloc(n * sizeof(int16_t));
  int32_t* nf = (int32_t*)malloc((size_t)B * H * sizeof(int32_t));
  for (size_t i = 0; i < n; ++i) {
    blk[i] = -1;
    len[i] = 0;
  }
  for (int step = 0; step < 200; ++step) {
    const int64_t p = 4000 + step;
    for (int r = 0; r < B * H; ++r) {
      const int c = 3 + (int)((g_rng >> 5) % (K - 2));
      cnt[r] = (int16_t)c;
      for (int e = 0; e < K; ++e) {
        g_rng ^= g_rng << 13;
        g_rng ^= g_rng >> 7;
        g_rng ^= g_rng << 17;
        sel[r * K + e] = e < c ? (int16_t)((g_rng >> 11) % (p / 64 + 1)) : -1;
      }
    }
    EXPECT(sparda_ref_plan_staging(&s, sel, cnt, p, blk, len, fetch, staged, nf), 0);
  }
  free(sel); free(cnt); free(blk); free(len); free(fetch); free(staged); free(nf);
}

/* The indexer-training loss of rows of a ragged chunk on both prediction grids. */
static void indexer_kl(int lw, int sw, int G, int k_top) {
  const int B = 1, H = 2, n_q = 7;
  const int64_t T = 1500, D = 128, nw = (T - lw) / sw + 1, nt = T - 1;
  const ref_shape s = shape(B, H, G, 8, 1536, nw, lw, sw, 1, 2);
  const ref_shape sf = shape(B, H, G, 8, 1536, nt, 2, 1, 1, 2);
  uint16_t* kk = bf16_buf((size_t)B * H * 1536 * D);
  uint16_t* q = bf16_buf((size_t)B * H * G * n_q * D);
  uint16_t* f = bf16_buf((size_t)B * H * n_q * D);
  uint16_t* kcp = (uint16_t*)malloc((size_t)B * H * nw * D * sizeof(uint16_t));
  uint16_t* kct = (uint16_t*)malloc((size_t)B * H * nt * D * sizeof(uint16_t));
  EXPECT(sparda_ref_compress_keys(&s, kk, T, 0, (int32_t)nw, kcp), 0);
  EXPECT(sparda_ref_compress_keys(&sf, kk, T, 0, (int32_t)nt, kct), 0);
  double loss, dF[128];
  int32_t* selp = (int32_t*)malloc((size_t)(k_top > 0 ? k_top : 1) * sizeof(int32_t));
  int32_t n_sel;
  for (int r = 0; r < n_q; ++r)
    EXPECT(sparda_ref_indexer_kl_row(&s, q, kct, nt, 2, 1, f, kcp, n_q, T - n_q, 0.0883883476, k_top, 0, 1, r, &loss,
                                     dF, selp, &n_sel),
           0);
  free(kk); free(q); free(f); free(kcp); free(kct); free(selp);
}

int main(void) {
  run(1, 2, 4, 16, 4096, 4096, 1, 64, 64, 1, 2);     /* decode, 4K */
  run(2, 3, 4, 16, 5000, 5056, 1, 64, 64, 1, 2);     /* decode, ragged context in a larger cache */
  run(1, 2, 4, 16, 3000, 3008, 300, 64, 64, 1, 2);   /* ragged prefill chunk */
  run(1, 1, 16, 96, 9000, 9024, 1, 32, 16, 1, 32);   /* the paper's grid and window */
  run(1, 2, 3, 64, 2000, 2048, 100, 32, 16, 0, 1);   /* no initial block, one local block */
  run(2, 1, 4, 200, 4096, 4096, 1, 64, 64, 1, 2);    /* a set larger than the context */
  run(1, 1, 2, 3, 64, 64, 64, 64, 64, 1, 2);         /* one block only */
  plan_steps();
  indexer_kl(32, 16, 4, 8);
  indexer_kl(64, 64, 16, 0);
  indexer_kl(32, 16, 2, 4096);
  printf("oracle harness: %d failed expectations\n", g_fail);
  return g_fail ? 1 : 0;
}

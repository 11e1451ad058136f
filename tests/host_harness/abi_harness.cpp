// abi_harness.cpp -- drives every entry point of include/sparda.h through its host code, built
// host-only against the stub runtime of hip_stub.cpp, under AddressSanitizer and
// UndefinedBehaviorSanitizer.  Device pointers are distinct aligned addresses that the host code
// never dereferences; pinned host pools are ranges registered with the stub.  The calls follow the
// benchmark's workloads (decode at 4K/32K/128K, the 32K prefill, the paper's head layout, the
// offloaded 32-layer decode at B64, 128K with its gathers, reuse plans and write-backs) and the
// documented error paths.  Exit status 0 when every call returned what the header promises and
// every launch had a valid configuration.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "sparda.h"

extern "C" {
void stub_register_host(const void* p, size_t bytes);
void stub_clear_host(void);
long stub_launches(void);
long stub_bad_launches(void);
}

namespace {

int g_failures = 0;

void expect(int got, int want, const char* what, int line) {
  if (got != want) {
    std::fprintf(stderr, "line %d: %s returned %d (%s), expected %d: %s\n", line, what, got, sparda_status_string(got),
                 want, sparda_last_error_detail());
    ++g_failures;
  } else if (want != SPARDA_OK && std::strlen(sparda_last_error_detail()) == 0) {
    std::fprintf(stderr, "line %d: %s failed without a detail text\n", line, what);
    ++g_failures;
  }
}
#define EXPECT(call, want) expect((call), (want), #call, __LINE__)

// Distinct 256-byte aligned stand-ins for device buffers (never dereferenced on the host).
uintptr_t g_next = (uintptr_t)1 << 44;
void* dev(size_t bytes) {
  void* p = reinterpret_cast<void*>(g_next);
  g_next += (bytes + 4095) & ~(size_t)4095;
  return p;
}
template <class T>
T* devp(size_t bytes) {
  return static_cast<T*>(dev(bytes));
}

sparda_shape shape(int B, int H, int G, int k, int64_t t_cap, int64_t nc_cap, int n_init = 1, int n_local = 2,
                   int lw = 64, int sw = 64) {
  sparda_shape s;
  std::memset(&s, 0, sizeof s);
  s.struct_size = sizeof(sparda_shape);
  s.batch = B;
  s.n_kv_heads = H;
  s.group_size = G;
  s.head_dim = 128;
  s.block_size = 64;
  s.cmp_kernel = lw;
  s.cmp_stride = sw;
  s.n_init = n_init;
  s.n_local = n_local;
  s.k_total = k;
  s.t_cap = t_cap;
  s.nc_cap = nc_cap;
  return s;
}

size_t ws_of(const sparda_shape& s, int op, int n_q, int64_t q_pos0) {
  size_t n = 0;
  EXPECT(sparda_workspace_size(&s, op, n_q, q_pos0, &n), SPARDA_OK);
  return n;
}

const float kScale = 0.08838834764831845f;

// One layer's select + attention (decode or multi-row), with workspaces sized by the library.
void layer(const sparda_shape& s, int n_q, int64_t q_pos0) {
  const size_t rows = (size_t)s.batch * s.n_kv_heads * n_q;
  void* f = dev(rows * 256);
  void* kc = dev((size_t)s.batch * s.n_kv_heads * s.nc_cap * 256);
  void* q = dev(rows * s.group_size * 256);
  void* k = dev((size_t)s.batch * s.n_kv_heads * s.t_cap * 256);
  void* v = dev((size_t)s.batch * s.n_kv_heads * s.t_cap * 256);
  int16_t* sel = devp<int16_t>(rows * s.k_total * 2);
  int16_t* cnt = devp<int16_t>(rows * 2);
  void* o = dev(rows * s.group_size * 256);
  const size_t ws_s = ws_of(s, SPARDA_OP_FORECAST_SELECT, n_q, q_pos0);
  const size_t ws_a = ws_of(s, SPARDA_OP_SPARSE_ATTN, n_q, q_pos0);
  const int64_t pl = q_pos0 + n_q;
  const int32_t nw = pl >= s.cmp_kernel ? (int32_t)((pl - s.cmp_kernel) / s.cmp_stride + 1) : 0;
  EXPECT(sparda_compress_keys(&s, k, pl, 0, nw, kc, nullptr), SPARDA_OK);
  EXPECT(sparda_forecast_select(&s, f, n_q, q_pos0, kc, sel, cnt, ws_s ? dev(ws_s) : nullptr, ws_s, nullptr),
         SPARDA_OK);
  EXPECT(sparda_sparse_attn(&s, q, n_q, q_pos0, k, v, 0, sel, cnt, kScale, o, ws_a ? dev(ws_a) : nullptr, ws_a,
                            nullptr),
         SPARDA_OK);
  EXPECT(sparda_sparse_attn_noalloc(&s, q, n_q, q_pos0, k, v, 0, sel, cnt, kScale, o, nullptr), SPARDA_OK);
  if (ws_s > 16)  // a workspace one float short is refused
    EXPECT(sparda_forecast_select(&s, f, n_q, q_pos0, kc, sel, cnt, dev(ws_s), ws_s - 4, nullptr),
           SPARDA_ERR_WORKSPACE);
  if (ws_a > 16)
    EXPECT(sparda_sparse_attn(&s, q, n_q, q_pos0, k, v, 0, sel, cnt, kScale, o, dev(ws_a), ws_a - 4, nullptr),
           SPARDA_ERR_WORKSPACE);
  if (s.cmp_kernel == 64 && n_q > 1) {
    float* row_max = devp<float>(rows * 4);
    EXPECT(sparda_forecast_score_max(&s, f, n_q, q_pos0, kc, row_max, nullptr), SPARDA_OK);
  }
  const size_t ws_m = ws_of(s, SPARDA_OP_MULTIHEAD_SELECT, n_q, q_pos0);
  EXPECT(sparda_multihead_select(&s, q, n_q, q_pos0, kc, kScale, sel, cnt, ws_m ? dev(ws_m) : nullptr, ws_m, nullptr),
         SPARDA_OK);
}

// The offloaded decode of the benchmark: 32 layers at B64, 128K, k = 64, two pools shared by the
// offloaded layers, the one-layer-ahead select, the reuse plan, the gather and the staged
// attention per layer, and the write-back of the decoded token, over a few steps.
void offloaded_pipeline() {
  const int B = 64, H = 8, G = 4, K = 64, L = 32;
  const int64_t T = 131072, nb = T / 64;
  sparda_shape s = shape(B, H, G, K, T, nb);
  const size_t pool = (size_t)B * H * T * 256;  // 16 GiB per pool: registered, never touched
  const uintptr_t host_base = (uintptr_t)1 << 46;
  void* hk[2];
  void* hv[2];
  for (int i = 0; i < 2; ++i) {
    hk[i] = reinterpret_cast<void*>(host_base + (2 * i) * pool);
    hv[i] = reinterpret_cast<void*>(host_base + (2 * i + 1) * pool);
    stub_register_host(hk[i], pool);
    stub_register_host(hv[i], pool);
  }
  const size_t rows = (size_t)B * H;
  void* stage_k = dev(rows * K * 64 * 256);
  void* stage_v = dev(rows * K * 64 * 256);
  int16_t* sel = devp<int16_t>(rows * K * 2);
  int16_t* cnt = devp<int16_t>(rows * 2);
  int16_t* blk = devp<int16_t>(rows * K * 2);
  int16_t* len = devp<int16_t>(rows * K * 2);
  int16_t* fetch = devp<int16_t>(rows * K * 2);
  int16_t* staged = devp<int16_t>(rows * K * 2);
  int16_t* scnt = devp<int16_t>(rows * 2);
  int32_t* nfetch = devp<int32_t>(rows * 4);
  void* f = dev(rows * 256);
  void* q = dev(rows * G * 256);
  void* o = dev(rows * G * 256);
  void* kc = dev(rows * nb * 256);
  void* k_new = dev(rows * 256);
  void* v_new = dev(rows * 256);
  for (int step = 0; step < 3; ++step) {
    const int64_t p = T - 3 + step;
    const size_t ws_s = ws_of(s, SPARDA_OP_FORECAST_SELECT, 1, p);
    const size_t ws_a = ws_of(s, SPARDA_OP_SPARSE_ATTN, 1, p);
    for (int l = 0; l < L; ++l) {
      EXPECT(sparda_forecast_select(&s, f, 1, p, kc, sel, cnt, ws_s ? dev(ws_s) : nullptr, ws_s, nullptr), SPARDA_OK);
      if (l == 0) continue;
      EXPECT(sparda_plan_staging(&s, sel, cnt, p, blk, len, fetch, staged, scnt, nfetch, nullptr), SPARDA_OK);
      for (int nwg : {8, 16, 64, 256})
        EXPECT(sparda_gather_blocks(&s, hk[(l - 1) % 2], hv[(l - 1) % 2], fetch, scnt, stage_k, stage_v, nwg, nullptr),
               SPARDA_OK);
      EXPECT(sparda_gather_blocks(&s, hk[(l - 1) % 2], hv[(l - 1) % 2], sel, cnt, stage_k, stage_v, 8, nullptr),
             SPARDA_OK);
      EXPECT(sparda_stage_append_kv(&s, k_new, v_new, p, staged, scnt, stage_k, stage_v, nullptr), SPARDA_OK);
      EXPECT(sparda_sparse_attn(&s, q, 1, p, stage_k, stage_v, 1, staged, scnt, kScale, o,
                                ws_a ? dev(ws_a) : nullptr, ws_a, nullptr),
             SPARDA_OK);
      EXPECT(sparda_writeback_kv(&s, k_new, v_new, 1, p, hk[(l - 1) % 2], hv[(l - 1) % 2], 8, nullptr), SPARDA_OK);
    }
  }
  // a pool one 16-byte piece short, an offset pointer whose allocation ends too early, and an
  // unregistered pointer are refused before any launch
  const long before = stub_launches();
  void* short_pool = reinterpret_cast<void*>(host_base + 4 * pool);
  stub_register_host(short_pool, pool - 16);
  EXPECT(sparda_gather_blocks(&s, short_pool, hv[0], sel, cnt, stage_k, stage_v, 8, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_gather_blocks(&s, hk[0], short_pool, sel, cnt, stage_k, stage_v, 8, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_writeback_kv(&s, k_new, v_new, 1, T - 1, short_pool, hv[0], 8, nullptr), SPARDA_ERR_INVALID_ARG);
  void* inside = reinterpret_cast<char*>(hk[0]) + 4096;
  EXPECT(sparda_gather_blocks(&s, inside, hv[0], sel, cnt, stage_k, stage_v, 8, nullptr), SPARDA_ERR_INVALID_ARG);
  void* unknown = reinterpret_cast<void*>((uintptr_t)1 << 47);
  EXPECT(sparda_gather_blocks(&s, unknown, hv[0], sel, cnt, stage_k, stage_v, 8, nullptr), SPARDA_ERR_HOST_NOT_MAPPED);
  EXPECT(sparda_writeback_kv(&s, k_new, v_new, 1, T - 1, hk[0], unknown, 8, nullptr), SPARDA_ERR_HOST_NOT_MAPPED);
  if (stub_launches() != before) {
    std::fprintf(stderr, "a refused gather or write-back launched a kernel\n");
    ++g_failures;
  }
  stub_clear_host();
}

void argument_errors() {
  sparda_shape s = shape(2, 8, 4, 16, 4096, 64);
  void* p = dev(1 << 20);
  int16_t* i16 = devp<int16_t>(1 << 16);
  size_t n = 0;
  EXPECT(sparda_workspace_size(nullptr, SPARDA_OP_SPARSE_ATTN, 1, 4095, &n), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_workspace_size(&s, 99, 1, 4095, &n), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_workspace_size(&s, SPARDA_OP_SPARSE_ATTN, 1, 4095, nullptr), SPARDA_ERR_INVALID_ARG);
  sparda_shape bad = s;
  bad.struct_size = 4;
  EXPECT(sparda_compress_keys(&bad, p, 4096, 0, 64, p, nullptr), SPARDA_ERR_INVALID_ARG);
  bad = s;
  bad.head_dim = 64;
  EXPECT(sparda_compress_keys(&bad, p, 4096, 0, 64, p, nullptr), SPARDA_ERR_UNSUPPORTED);
  bad = s;
  bad.group_size = 17;
  EXPECT(sparda_sparse_attn(&bad, p, 1, 4095, p, p, 0, i16, i16, kScale, p, p, 1 << 20, nullptr),
         SPARDA_ERR_UNSUPPORTED);
  bad = s;
  bad.k_total = 2;
  EXPECT(sparda_forecast_select(&bad, p, 1, 4095, p, i16, i16, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  bad = s;
  bad.t_cap = 100;
  EXPECT(sparda_forecast_select(&bad, p, 1, 99, p, i16, i16, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_compress_keys(&s, p, 4096, 0, 65, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_compress_keys(&s, p, 4000, 62, 63, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_compress_keys(&s, reinterpret_cast<char*>(p) + 2, 4096, 0, 64, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_forecast_select(&s, p, 0, 4095, p, i16, i16, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_forecast_select(&s, p, 2, 4095, p, i16, i16, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_forecast_select(&s, nullptr, 1, 4095, p, i16, i16, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_sparse_attn(&s, p, 1, 4095, p, p, 2, i16, i16, kScale, p, p, 1 << 20, nullptr),
         SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_sparse_attn(&s, p, 2, 4094, p, p, 1, i16, i16, kScale, p, p, 1 << 20, nullptr),
         SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_sparse_attn(&s, p, 1, 4095, p, p, 0, i16, i16, NAN, p, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_sparse_attn(&s, p, 1, 4095, p, p, 0, i16, i16, kScale, p, nullptr, 0, nullptr), SPARDA_ERR_WORKSPACE);
  EXPECT(sparda_sparse_attn_noalloc(&s, p, 1, 4095, p, p, 2, i16, i16, kScale, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_multihead_select(&s, p, 1, 4095, p, -1.f, i16, i16, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_gather_blocks(&s, p, p, i16, i16, p, p, 0, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_writeback_kv(&s, p, p, 0, 0, p, p, 8, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_writeback_kv(&s, p, p, 2, 4095, p, p, 8, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_stage_append_kv(&s, p, p, 4096, i16, i16, p, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_stage_append_kv(&s, p, p, -1, i16, i16, p, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_stage_append_kv(&s, p, nullptr, 10, i16, i16, p, p, nullptr), SPARDA_ERR_INVALID_ARG);
  EXPECT(sparda_plan_staging(&s, i16, i16, 4096, i16, i16, i16, i16, i16, reinterpret_cast<int32_t*>(p), nullptr),
         SPARDA_ERR_INVALID_ARG);
  float* fl = devp<float>(1 << 20);
  EXPECT(sparda_indexer_kl(&s, p, p, p, p, 1, 4095, kScale, 8, fl, fl, nullptr, 0, nullptr), SPARDA_ERR_WORKSPACE);
  EXPECT(sparda_indexer_kl(&s, p, p, p, p, 1, 4095, kScale, -1, fl, fl, p, 1 << 20, nullptr), SPARDA_ERR_INVALID_ARG);
  for (int st = 0; st >= -6; --st)
    if (std::strlen(sparda_status_string(st)) == 0) ++g_failures;
}

}  // namespace

int main() {
  // decode at the benchmark's context lengths, and a ragged one
  layer(shape(1, 8, 4, 16, 4096, 64), 1, 4095);
  layer(shape(8, 8, 4, 64, 32768, 512), 1, 32767);
  layer(shape(32, 8, 4, 64, 131072, 2048), 1, 131071);
  layer(shape(3, 2, 3, 12, 5056, 79), 1, 5000);
  // the 32K prefill, a ragged chunk, and a chunk past 512 candidates (the row-wise path)
  layer(shape(1, 8, 4, 64, 32768, 512), 32768, 0);
  layer(shape(2, 3, 4, 64, 5056, 79), 700, 4300);
  layer(shape(1, 2, 4, 64, 70016, 1094), 130, 69870);
  // the paper's layout on the (32, 16) grid: decode at 128K (split select) and the 32K prefill
  layer(shape(32, 2, 16, 96, 131072, 8191, 1, 32, 32, 16), 1, 131071);
  layer(shape(1, 2, 16, 96, 32768, 2047, 1, 32, 32, 16), 32768, 0);
  // the indexer-training loss on a 256-row chunk at 64K
  {
    sparda_shape s = shape(1, 8, 4, 64, 65536, 4095, 1, 2, 32, 16);
    const size_t ws = ws_of(s, SPARDA_OP_INDEXER_KL, 256, 65280);
    EXPECT(sparda_indexer_kl(&s, dev(1 << 24), dev((size_t)8 * 65536 * 256), dev(1 << 20), dev((size_t)8 * 4095 * 256),
                             256, 65280, kScale, 64, devp<float>(1 << 14), devp<float>(1 << 22), dev(ws), ws, nullptr),
           SPARDA_OK);
  }
  offloaded_pipeline();
  argument_errors();
  const long bad = stub_bad_launches();
  std::printf("abi harness: %ld launches checked, %ld with an invalid configuration, %d failed expectations\n",
              stub_launches(), bad, g_failures);
  return (g_failures == 0 && bad == 0 && stub_launches() > 100) ? 0 : 1;
}

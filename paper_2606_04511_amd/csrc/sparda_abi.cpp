// sparda_abi.cpp -- the extern "C" entry points declared in include/sparda.h.
//
// Every entry point validates its arguments on the host (no HIP call happens before validation
// has passed, so argument errors are reported without a GPU), sizes its workspace, and hands
// the launch to the kernel files.  The library keeps no state except a thread-local error text.
#include "sparda.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "launch.hpp"

namespace {

thread_local std::string g_detail;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_detail = buf;
  return status;
}

int ok() {
  g_detail.clear();
  return SPARDA_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

constexpr int64_t kMaxBlocks = 32768;  // block indices are int16

int check_shape(const sparda_shape* s) {
  if (!s) return fail(SPARDA_ERR_INVALID_ARG, "shape is null");
  if (s->struct_size != sizeof(sparda_shape))
    return fail(SPARDA_ERR_INVALID_ARG, "shape.struct_size is %u, expected %zu", s->struct_size, sizeof(sparda_shape));
  if (s->batch < 1 || s->n_kv_heads < 1 || s->group_size < 1)
    return fail(SPARDA_ERR_INVALID_ARG, "batch, n_kv_heads and group_size must be >= 1");
  if (s->group_size > 16) return fail(SPARDA_ERR_UNSUPPORTED, "group_size %d > 16", s->group_size);
  if (s->head_dim != 128) return fail(SPARDA_ERR_UNSUPPORTED, "head_dim %d (only 128)", s->head_dim);
  if (s->block_size != 64) return fail(SPARDA_ERR_UNSUPPORTED, "block_size %d (only 64)", s->block_size);
  if (!((s->cmp_kernel == 64 && s->cmp_stride == 64) || (s->cmp_kernel == 32 && s->cmp_stride == 16)))
    return fail(SPARDA_ERR_UNSUPPORTED, "compression window (%d, %d) (only (64, 64) and (32, 16))", s->cmp_kernel,
                s->cmp_stride);
  if (s->n_init < 0 || s->n_local < 1) return fail(SPARDA_ERR_INVALID_ARG, "n_init >= 0 and n_local >= 1 required");
  if ((int64_t)s->k_total < (int64_t)s->n_init + s->n_local)
    return fail(SPARDA_ERR_INVALID_ARG, "k_total %d < n_init + n_local", s->k_total);
  if (s->k_total >= kMaxBlocks) return fail(SPARDA_ERR_UNSUPPORTED, "k_total %d too large", s->k_total);
  if (s->t_cap < 64 || s->t_cap % 64 != 0)
    return fail(SPARDA_ERR_INVALID_ARG, "t_cap %lld must be a positive multiple of 64", (long long)s->t_cap);
  if (s->t_cap / 64 > kMaxBlocks)
    return fail(SPARDA_ERR_UNSUPPORTED, "t_cap %lld exceeds 32768 blocks", (long long)s->t_cap);
  if (s->nc_cap < 0 || s->nc_cap > kMaxBlocks * (64 / s->cmp_stride))
    return fail(SPARDA_ERR_INVALID_ARG, "nc_cap out of range");
  if ((int64_t)s->batch * s->n_kv_heads > 65535)
    return fail(SPARDA_ERR_UNSUPPORTED, "batch * n_kv_heads > 65535");
  return SPARDA_OK;
}

int check_dev(const void* p, const char* name, uintptr_t align) {
  if (!p) return fail(SPARDA_ERR_INVALID_ARG, "%s is null", name);
  if (!aligned(p, align)) return fail(SPARDA_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, (size_t)align);
  return SPARDA_OK;
}

int check_rows(const sparda_shape* s, int32_t n_q, int64_t q_pos0) {
  if (n_q < 1) return fail(SPARDA_ERR_INVALID_ARG, "n_q %d < 1", n_q);
  if (q_pos0 < 0 || q_pos0 + n_q > s->t_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "positions [%lld, %lld) outside t_cap %lld", (long long)q_pos0,
                (long long)(q_pos0 + n_q), (long long)s->t_cap);
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  if (rows > (int64_t)1 << 30) return fail(SPARDA_ERR_UNSUPPORTED, "too many query rows");
  return SPARDA_OK;
}

sparda::WinGrid grid_of(const sparda_shape* s) { return sparda::WinGrid{s->cmp_kernel, s->cmp_stride}; }

// Workspace of sparda_forecast_select: window scores of the row-wise path (none for the fused
// kernels).  The last row scores the most windows.
size_t select_ws(const sparda_shape* s, int32_t n_q, int64_t q_pos0, int64_t* stride) {
  const int64_t pl = q_pos0 + n_q - 1;
  const sparda::RowGeom g = sparda::row_geom(pl, s->n_init, s->n_local, s->k_total);
  int32_t wf, wl;
  sparda::row_windows(g, grid_of(s), pl, &wf, &wl);
  const int64_t nw = wl >= wf ? (int64_t)(wl - wf + 1) : 0;
  *stride = (nw + 3) & ~(int64_t)3;
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  if (!sparda::select_needs_scratch(rows, n_q, q_pos0, s->n_init, s->n_local, grid_of(s))) return 0;
  if (g.n_cand == 0) return 0;
  return (size_t)rows * (size_t)*stride * sizeof(float);
}

// Workspace of sparda_multihead_select: every head's window scores plus the shared scores on the
// row-wise path (none on the fused decode kernel).
size_t multihead_ws(const sparda_shape* s, int32_t n_q, int64_t q_pos0, int64_t* stride) {
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  return sparda::multihead_ws_floats(rows, s->group_size, n_q, q_pos0, s->n_init, s->n_local, s->k_total,
                                     grid_of(s), stride) *
         sizeof(float);
}

// Workspace of sparda_indexer_kl: the fine (2, 1) windows complete at the last row (bf16), then
// every row's target weight of each of them (float, rows padded to 4).
size_t kl_keys_bytes(const sparda_shape* s, int32_t n_q, int64_t q_pos0) {
  const int64_t nt = q_pos0 + n_q - 1;
  return (size_t)s->batch * s->n_kv_heads * (size_t)(nt > 0 ? nt : 1) * s->head_dim * sizeof(uint16_t);
}
size_t kl_ws(const sparda_shape* s, int32_t n_q, int64_t q_pos0) {
  const int64_t nt = q_pos0 + n_q - 1;
  const int64_t stride = ((nt > 0 ? nt : 1) + 3) & ~(int64_t)3;
  return kl_keys_bytes(s, n_q, q_pos0) + (size_t)s->batch * s->n_kv_heads * n_q * (size_t)stride * sizeof(float);
}

size_t attn_ws(const sparda_shape* s, int32_t n_q, int64_t q_pos0, int32_t* n_splits, int32_t* bps);

// Workspace of a decode step: the selection's window scores, then (from a 256-byte aligned
// offset) the attention's split partials.  The two live side by side because the fused kernel's
// workgroups still read scores while others write partials.  *attn_off gets the offset.
size_t step_ws(const sparda_shape* s, int64_t q_pos, size_t* attn_off) {
  int64_t stride;
  int32_t ns, bps;
  const size_t a = (select_ws(s, 1, q_pos, &stride) + 255) & ~(size_t)255, b = attn_ws(s, 1, q_pos, &ns, &bps);
  if (attn_off) *attn_off = a;
  return b > 0 ? a + b : a;
}

size_t attn_ws(const sparda_shape* s, int32_t n_q, int64_t q_pos0, int32_t* n_splits, int32_t* bps) {
  if (sparda::attn_uses_tiles(s->group_size, n_q, q_pos0)) {  // tiled multi-row kernel: no partials
    *n_splits = 1;
    *bps = s->k_total;
    return 0;
  }
  const int64_t rows = (int64_t)s->batch * s->n_kv_heads * n_q;
  sparda::attn_plan(rows, s->k_total, n_splits, bps);
  if (*n_splits <= 1) return 0;
  return (size_t)rows * (size_t)*n_splits * (size_t)s->group_size * (size_t)(s->head_dim + 2) * sizeof(float);
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(SPARDA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

// Scratch of sparda_sparse_attn_noalloc: the split partials of attention calls with fewer rows
// than CUs.  Partials exist only below 256 rows, with at most ceil(256 / rows) splits per row,
// so rows x splits <= 511 and 511 x 16 heads x (128 + 2) floats = 4.25 MB covers every call.
// One copy per GPU, for the life of the process.  Host code never uses the array's name as an
// address: the device address comes from hipGetSymbolAddress, once per device.
static_assert(SPARDA_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size is a multiple of its alignment");
static_assert(SPARDA_NOALLOC_SCRATCH_BYTES >= (size_t)511 * 16 * (128 + 2) * sizeof(float),
              "scratch covers the largest split partials");

}  // namespace

static __device__ __align__(256) unsigned char scratch[SPARDA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up on the first call on that device.
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPARDA_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(SPARDA_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(SPARDA_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SPARDA_OK;
}

// sparda_sparse_attn and its no-allocation variant (static_ws: the partials go to `scratch`).
// Validates an attention call and fills its kernel arguments; nothing is enqueued.
int attn_prepare(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0, const void* k, const void* v,
                 int32_t kv_mode, const int16_t* sel, const int16_t* cnt, float sm_scale, void* o, void* ws,
                 size_t ws_bytes, bool static_ws, sparda::AttnArgs* out) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(q, "q", 16)) || (rc = check_dev(k, "k", 16)) || (rc = check_dev(v, "v", 16)) ||
      (rc = check_dev(sel, "sel", 2)) || (rc = check_dev(cnt, "cnt", 2)) || (rc = check_dev(o, "o", 16)))
    return rc;
  if ((rc = check_rows(shape, n_q, q_pos0))) return rc;
  if (kv_mode != 0 && kv_mode != 1) return fail(SPARDA_ERR_INVALID_ARG, "kv_mode %d", kv_mode);
  if (kv_mode == 1 && n_q != 1) return fail(SPARDA_ERR_INVALID_ARG, "staging mode needs n_q == 1");
  if (!std::isfinite(sm_scale)) return fail(SPARDA_ERR_INVALID_ARG, "sm_scale is not finite");
  int32_t ns = 1, bps = shape->k_total;
  const size_t need = attn_ws(shape, n_q, q_pos0, &ns, &bps);
  if (static_ws) {
    if (need > SPARDA_NOALLOC_SCRATCH_BYTES)
      return fail(SPARDA_ERR_WORKSPACE, "split partials of %zu bytes exceed the %zu-byte static scratch", need,
                  (size_t)SPARDA_NOALLOC_SCRATCH_BYTES);
    ws = nullptr;
    if (need > 0 && (rc = scratch_address(&ws))) return rc;
  } else if (need > 0) {
    if (!ws || !aligned(ws, 16)) return fail(SPARDA_ERR_WORKSPACE, "workspace of %zu bytes required", need);
    if (ws_bytes < need) return fail(SPARDA_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  }
  sparda::AttnArgs& a = *out;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.sel = sel;
  a.cnt = cnt;
  a.o = static_cast<uint16_t*>(o);
  a.ws = static_cast<float*>(ws);
  a.batch = shape->batch;
  a.n_kv_heads = shape->n_kv_heads;
  a.group_size = shape->group_size;
  a.n_q = n_q;
  a.q_pos0 = q_pos0;
  a.t_cap = shape->t_cap;
  a.kv_mode = kv_mode;
  a.k_total = shape->k_total;
  a.sm_scale = sm_scale;
  a.n_splits = ns;
  a.blocks_per_split = bps;
  return ok();
}

int attn_call(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0, const void* k, const void* v,
              int32_t kv_mode, const int16_t* sel, const int16_t* cnt, float sm_scale, void* o, void* ws,
              size_t ws_bytes, bool static_ws, hipStream_t stream) {
  sparda::AttnArgs a;
  const int rc = attn_prepare(shape, q, n_q, q_pos0, k, v, kv_mode, sel, cnt, sm_scale, o, ws, ws_bytes, static_ws, &a);
  if (rc) return rc;
  return hip_status(sparda::launch_sparse_attn(a, stream), "attention launch");

}

// Validates a select call and fills its kernel arguments; nothing is enqueued.
int select_prepare(const sparda_shape* shape, const void* f, int32_t n_q, int64_t q_pos0, const void* k_cmp,
                   int16_t* sel, int16_t* cnt, void* ws, size_t ws_bytes, sparda::SelectArgs* out) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(f, "f", 16)) || (rc = check_dev(k_cmp, "k_cmp", 16)) || (rc = check_dev(sel, "sel", 2)) ||
      (rc = check_dev(cnt, "cnt", 2)))
    return rc;
  if ((rc = check_rows(shape, n_q, q_pos0))) return rc;
  const int64_t pl = q_pos0 + n_q - 1;
  const sparda::RowGeom gl = sparda::row_geom(pl, shape->n_init, shape->n_local, shape->k_total);
  int32_t wf, wl;
  sparda::row_windows(gl, grid_of(shape), pl, &wf, &wl);
  if (gl.n_cand > 0 && (int64_t)wl >= shape->nc_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "compressed key %d (for block %d) beyond nc_cap %lld", wl,
                gl.cand_lo + gl.n_cand - 1, (long long)shape->nc_cap);
  int64_t stride = 0;
  const size_t need = select_ws(shape, n_q, q_pos0, &stride);
  if (need > 0) {
    if (!ws || !aligned(ws, 16)) return fail(SPARDA_ERR_WORKSPACE, "workspace of %zu bytes required", need);
    if (ws_bytes < need) return fail(SPARDA_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  }
  sparda::SelectArgs& a = *out;
  a.f = static_cast<const uint16_t*>(f);
  a.kc = static_cast<const uint16_t*>(k_cmp);
  a.sel = sel;
  a.cnt = cnt;
  a.ws = static_cast<float*>(ws);
  a.ws_stride = stride;
  a.batch = shape->batch;
  a.n_kv_heads = shape->n_kv_heads;
  a.n_q = n_q;
  a.q_pos0 = q_pos0;
  a.nc_cap = shape->nc_cap;
  a.n_init = shape->n_init;
  a.n_local = shape->n_local;
  a.k_total = shape->k_total;
  a.grid = grid_of(shape);
  return ok();
}

}  // namespace

extern "C" {

const char* sparda_status_string(int status) {
  switch (status) {
    case SPARDA_OK: return "SPARDA_OK";
    case SPARDA_ERR_INVALID_ARG: return "SPARDA_ERR_INVALID_ARG";
    case SPARDA_ERR_UNSUPPORTED: return "SPARDA_ERR_UNSUPPORTED";
    case SPARDA_ERR_WORKSPACE: return "SPARDA_ERR_WORKSPACE";
    case SPARDA_ERR_HOST_NOT_MAPPED: return "SPARDA_ERR_HOST_NOT_MAPPED";
    case SPARDA_ERR_HIP: return "SPARDA_ERR_HIP";
    default: return "SPARDA_ERR_UNKNOWN";
  }
}

const char* sparda_last_error_detail(void) { return g_detail.c_str(); }

int sparda_workspace_size(const sparda_shape* shape, int32_t op, int32_t n_q, int64_t q_pos0, size_t* bytes) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (!bytes) return fail(SPARDA_ERR_INVALID_ARG, "bytes is null");
  if ((rc = check_rows(shape, n_q, q_pos0))) return rc;
  if (op == SPARDA_OP_FORECAST_SELECT) {
    int64_t stride;
    *bytes = select_ws(shape, n_q, q_pos0, &stride);
  } else if (op == SPARDA_OP_SPARSE_ATTN) {
    int32_t ns, bps;
    *bytes = attn_ws(shape, n_q, q_pos0, &ns, &bps);
  } else if (op == SPARDA_OP_MULTIHEAD_SELECT) {
    int64_t stride;
    *bytes = multihead_ws(shape, n_q, q_pos0, &stride);
  } else if (op == SPARDA_OP_INDEXER_KL) {
    *bytes = kl_ws(shape, n_q, q_pos0);
  } else if (op == SPARDA_OP_DECODE_STEP) {
    if (n_q != 1) return fail(SPARDA_ERR_INVALID_ARG, "a decode step has n_q == 1");
    *bytes = step_ws(shape, q_pos0, nullptr);
  } else {
    return fail(SPARDA_ERR_INVALID_ARG, "unknown op %d", op);
  }
  return ok();
}

int sparda_compress_keys(const sparda_shape* shape, const void* k_cache, int64_t t_ctx, int32_t win_begin,
                         int32_t win_end, void* k_cmp, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(k_cache, "k_cache", 16)) || (rc = check_dev(k_cmp, "k_cmp", 16))) return rc;
  if (t_ctx < 0 || t_ctx > shape->t_cap) return fail(SPARDA_ERR_INVALID_ARG, "t_ctx outside [0, t_cap]");
  if (win_begin < 0 || win_end < win_begin) return fail(SPARDA_ERR_INVALID_ARG, "bad window range");
  if (win_end > shape->nc_cap) return fail(SPARDA_ERR_INVALID_ARG, "win_end %d > nc_cap", win_end);
  if (win_end == win_begin) return ok();
  if ((int64_t)(win_end - 1) * shape->cmp_stride + shape->cmp_kernel > t_ctx)
    return fail(SPARDA_ERR_INVALID_ARG, "window %d is not complete", win_end - 1);
  return hip_status(sparda::launch_compress(static_cast<const uint16_t*>(k_cache), static_cast<uint16_t*>(k_cmp),
                                            shape->batch * shape->n_kv_heads, shape->t_cap, shape->nc_cap,
                                            grid_of(shape), win_begin, win_end, stream),
                    "compress launch");
}

int sparda_forecast_select(const sparda_shape* shape, const void* f, int32_t n_q, int64_t q_pos0,
                           const void* k_cmp, int16_t* sel, int16_t* cnt, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  sparda::SelectArgs a;
  const int rc = select_prepare(shape, f, n_q, q_pos0, k_cmp, sel, cnt, ws, ws_bytes, &a);
  if (rc) return rc;
  return hip_status(sparda::launch_select(a, stream), "select launch");
}

int sparda_decode_step(const sparda_shape* shape, const void* f, int64_t q_pos, const void* k_cmp, const void* q,
                       const void* k, const void* v, float sm_scale, int16_t* sel, int16_t* cnt, void* o, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  sparda::SelectArgs sa;
  sparda::AttnArgs aa;
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_rows(shape, 1, q_pos))) return rc;
  size_t off = 0;
  const size_t need = step_ws(shape, q_pos, &off);
  // each half checks its arguments and its part of the workspace, then the whole is checked
  if ((rc = select_prepare(shape, f, 1, q_pos, k_cmp, sel, cnt, ws, off, &sa))) return rc;
  void* ws_att = (ws && need > off) ? static_cast<char*>(ws) + off : nullptr;
  if ((rc = attn_prepare(shape, q, 1, q_pos, k, v, 0, sel, cnt, sm_scale, o, ws_att, need - off, false, &aa)))
    return rc;
  if (need > 0 && ws_bytes < need) return fail(SPARDA_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  return hip_status(sparda::launch_decode_step(sa, aa, stream), "decode step launch");

}

int sparda_forecast_score_max(const sparda_shape* shape, const void* f, int32_t n_q, int64_t q_pos0,
                              const void* k_cmp, float* row_max, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(f, "f", 16)) || (rc = check_dev(k_cmp, "k_cmp", 16)) || (rc = check_dev(row_max, "row_max", 4)))
    return rc;
  if ((rc = check_rows(shape, n_q, q_pos0))) return rc;
  if (shape->cmp_kernel != 64 || shape->cmp_stride != 64)
    return fail(SPARDA_ERR_UNSUPPORTED, "the score-only contraction covers the (64, 64) grid only");
  const int64_t pl = q_pos0 + n_q - 1;
  const sparda::RowGeom gl = sparda::row_geom(pl, shape->n_init, shape->n_local, shape->k_total);
  if (gl.n_cand > 0 && (int64_t)(gl.cand_lo + gl.n_cand - 1) >= shape->nc_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "compressed key %d beyond nc_cap %lld", gl.cand_lo + gl.n_cand - 1,
                (long long)shape->nc_cap);
  sparda::ScoreMaxArgs a;
  a.f = static_cast<const uint16_t*>(f);
  a.kc = static_cast<const uint16_t*>(k_cmp);
  a.row_max = row_max;
  a.nc_cap = shape->nc_cap;
  a.q_pos0 = q_pos0;
  a.n_q = n_q;
  a.n_groups = shape->batch * shape->n_kv_heads;
  a.blk0 = (int32_t)(q_pos0 / 64);
  a.n_units = (int32_t)(pl / 64) - a.blk0 + 1;
  a.n_init = shape->n_init;
  a.n_local = shape->n_local;
  return hip_status(sparda::launch_score_rowmax(a, stream), "score-max launch");
}

int sparda_multihead_select(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0,
                            const void* k_cmp, float sm_scale, int16_t* sel, int16_t* cnt, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(q, "q", 16)) || (rc = check_dev(k_cmp, "k_cmp", 16)) || (rc = check_dev(sel, "sel", 2)) ||
      (rc = check_dev(cnt, "cnt", 2)))
    return rc;
  if ((rc = check_rows(shape, n_q, q_pos0))) return rc;
  if (!(sm_scale > 0.0f) || !std::isfinite(sm_scale))
    return fail(SPARDA_ERR_INVALID_ARG, "sm_scale must be finite and > 0");
  const int64_t pl = q_pos0 + n_q - 1;
  const int64_t last = sparda::grid_win_vis(grid_of(shape), pl);  // every head's softmax reads 0 .. last
  if (last >= shape->nc_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "compressed key %lld (complete at position %lld) beyond nc_cap %lld",
                (long long)last, (long long)pl, (long long)shape->nc_cap);
  int64_t stride = 0;
  const size_t need = multihead_ws(shape, n_q, q_pos0, &stride);
  if (need > 0) {
    if (!ws || !aligned(ws, 16)) return fail(SPARDA_ERR_WORKSPACE, "workspace of %zu bytes required", need);
    if (ws_bytes < need) return fail(SPARDA_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  }
  sparda::SelectArgs a{};
  a.kc = static_cast<const uint16_t*>(k_cmp);
  a.sel = sel;
  a.cnt = cnt;
  a.ws = static_cast<float*>(ws);
  a.ws_stride = stride;
  a.batch = shape->batch;
  a.n_kv_heads = shape->n_kv_heads;
  a.n_q = n_q;
  a.q_pos0 = q_pos0;
  a.nc_cap = shape->nc_cap;
  a.n_init = shape->n_init;
  a.n_local = shape->n_local;
  a.k_total = shape->k_total;
  a.grid = grid_of(shape);
  a.q = static_cast<const uint16_t*>(q);
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.group_size = shape->group_size;
  return hip_status(sparda::launch_multihead_select(a, stream), "multihead select launch");
}

int sparda_sparse_attn(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0, const void* k,
                       const void* v, int32_t kv_mode, const int16_t* sel, const int16_t* cnt, float sm_scale,
                       void* o, void* ws, size_t ws_bytes, hipStream_t stream) {
  return attn_call(shape, q, n_q, q_pos0, k, v, kv_mode, sel, cnt, sm_scale, o, ws, ws_bytes, false, stream);
}

int sparda_sparse_attn_noalloc(const sparda_shape* shape, const void* q, int32_t n_q, int64_t q_pos0, const void* k,
                               const void* v, int32_t kv_mode, const int16_t* sel, const int16_t* cnt,
                               float sm_scale, void* o, hipStream_t stream) {
  return attn_call(shape, q, n_q, q_pos0, k, v, kv_mode, sel, cnt, sm_scale, o, nullptr, 0, true, stream);
}

int sparda_indexer_kl(const sparda_shape* shape, const void* q, const void* k, const void* f, const void* k_cmp,
                      int32_t n_q, int64_t q_pos0, float sm_scale, int32_t k_top, float* loss, float* d_f,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(q, "q", 16)) || (rc = check_dev(k, "k", 16)) || (rc = check_dev(f, "f", 16)) ||
      (rc = check_dev(k_cmp, "k_cmp", 16)) || (rc = check_dev(loss, "loss", 4)) || (rc = check_dev(d_f, "d_f", 4)))
    return rc;
  if ((rc = check_rows(shape, n_q, q_pos0))) return rc;
  if (!(sm_scale > 0.0f) || !std::isfinite(sm_scale))
    return fail(SPARDA_ERR_INVALID_ARG, "sm_scale must be finite and > 0");
  if (k_top < 0 || k_top > 4096) return fail(SPARDA_ERR_INVALID_ARG, "k_top %d outside [0, 4096]", k_top);
  if (q_pos0 < shape->cmp_kernel - 1)
    return fail(SPARDA_ERR_INVALID_ARG, "row 0 (position %lld) has no complete window", (long long)q_pos0);
  const int64_t pl = q_pos0 + n_q - 1;
  const int64_t last = sparda::grid_win_vis(grid_of(shape), pl);
  if (last >= shape->nc_cap || last + 1 > 16384)
    return fail(SPARDA_ERR_INVALID_ARG, "window %lld of the last row beyond nc_cap %lld or 16384 per row",
                (long long)last, (long long)shape->nc_cap);
  const size_t need = kl_ws(shape, n_q, q_pos0);
  if (!ws || !aligned(ws, 16)) return fail(SPARDA_ERR_WORKSPACE, "workspace of %zu bytes required", need);
  if (ws_bytes < need) return fail(SPARDA_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  return hip_status(sparda::launch_indexer_kl(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                              static_cast<const uint16_t*>(f), static_cast<const uint16_t*>(k_cmp),
                                              static_cast<uint16_t*>(ws),
                                              reinterpret_cast<float*>(static_cast<char*>(ws) +
                                                                       kl_keys_bytes(shape, n_q, q_pos0)),
                                              loss, d_f, shape->batch, shape->n_kv_heads,
                                              shape->group_size, n_q, q_pos0, shape->t_cap, shape->nc_cap,
                                              shape->n_init, shape->n_local, k_top, grid_of(shape), sm_scale, stream),
                    "indexer kl launch");
}

int sparda_plan_staging(const sparda_shape* shape, const int16_t* sel, const int16_t* cnt, int64_t q_pos,
                        int16_t* slot_blk, int16_t* slot_len, int16_t* fetch, int16_t* sel_staged,
                        int16_t* stage_cnt, int32_t* n_fetch, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(sel, "sel", 2)) || (rc = check_dev(cnt, "cnt", 2)) || (rc = check_dev(slot_blk, "slot_blk", 2)) ||
      (rc = check_dev(slot_len, "slot_len", 2)) || (rc = check_dev(fetch, "fetch", 2)) ||
      (rc = check_dev(sel_staged, "sel_staged", 2)) || (rc = check_dev(stage_cnt, "stage_cnt", 2)) ||
      (rc = check_dev(n_fetch, "n_fetch", 4)))
    return rc;
  if (q_pos < 0 || q_pos >= shape->t_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "q_pos %lld outside [0, t_cap)", (long long)q_pos);
  if (shape->k_total > 1024) return fail(SPARDA_ERR_UNSUPPORTED, "k_total %d > 1024 for the staging plan", shape->k_total);
  return hip_status(sparda::launch_plan_staging(sel, cnt, q_pos, slot_blk, slot_len, fetch, sel_staged, stage_cnt, n_fetch,
                                                (int64_t)shape->batch * shape->n_kv_heads, shape->k_total, stream),
                    "plan launch");
}

// The device address of a pinned host pool mapped for the device.  Fails with
// SPARDA_ERR_HOST_NOT_MAPPED unless `host` is device-mapped pinned host memory, and with
// SPARDA_ERR_INVALID_ARG unless the allocation holding it extends at least `need` bytes from it
// (the largest offset a gather or write-back over the pool layout can touch).
static int mapped_pool(const void* host, const char* name, size_t need, void** dev) {
  hipPointerAttribute_t attr;
  hipError_t e = hipPointerGetAttributes(&attr, host);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // clear the error state of this query
    return fail(SPARDA_ERR_HOST_NOT_MAPPED, "%s is not a registered HIP allocation (%s)", name, hipGetErrorString(e));
  }
  if (attr.type != hipMemoryTypeHost || attr.devicePointer == nullptr)
    return fail(SPARDA_ERR_HOST_NOT_MAPPED, "%s is not device-mapped pinned host memory", name);
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  e = hipMemGetAddressRange(&base, &size, attr.devicePointer);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(SPARDA_ERR_HOST_NOT_MAPPED, "%s: the extent of its allocation is unknown (%s)", name,
                hipGetErrorString(e));
  }
  const uintptr_t p = reinterpret_cast<uintptr_t>(attr.devicePointer), b = reinterpret_cast<uintptr_t>(base);
  if (p < b || p - b > size || size - (p - b) < need)
    return fail(SPARDA_ERR_INVALID_ARG, "%s: %zu bytes of its allocation lie past the pointer, the pool layout "
                "[B][Hkv][t_cap][D] needs %zu", name, p < b ? (size_t)0 : size - (size_t)(p - b), need);
  *dev = attr.devicePointer;
  return SPARDA_OK;
}

// Bytes of one host pool: bf16 [B][Hkv][t_cap][D].
static size_t pool_bytes(const sparda_shape* s) {
  return (size_t)s->batch * s->n_kv_heads * (size_t)s->t_cap * s->head_dim * sizeof(uint16_t);
}

int sparda_writeback_kv(const sparda_shape* shape, const void* k_new, const void* v_new, int32_t n_new, int64_t pos0,
                        void* host_k, void* host_v, int32_t n_workgroups, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(k_new, "k_new", 16)) || (rc = check_dev(v_new, "v_new", 16)) ||
      (rc = check_dev(host_k, "host_k", 16)) || (rc = check_dev(host_v, "host_v", 16)))
    return rc;
  if (n_new < 1) return fail(SPARDA_ERR_INVALID_ARG, "n_new %d < 1", n_new);
  if (pos0 < 0 || pos0 + n_new > shape->t_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "positions [%lld, %lld) outside t_cap %lld", (long long)pos0,
                (long long)(pos0 + n_new), (long long)shape->t_cap);
  if (n_workgroups < 1) return fail(SPARDA_ERR_INVALID_ARG, "n_workgroups %d < 1", n_workgroups);
  void* dk = nullptr;
  void* dv = nullptr;
  if ((rc = mapped_pool(host_k, "host_k", pool_bytes(shape), &dk)) ||
      (rc = mapped_pool(host_v, "host_v", pool_bytes(shape), &dv)))
    return rc;
  return hip_status(sparda::launch_writeback(static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                                             static_cast<uint16_t*>(dk), static_cast<uint16_t*>(dv),
                                             (int64_t)shape->batch * shape->n_kv_heads, n_new, pos0, shape->t_cap,
                                             n_workgroups, stream),
                    "write-back launch");
}

int sparda_stage_append_kv(const sparda_shape* shape, const void* k_new, const void* v_new, int64_t q_pos,
                           const int16_t* sel, const int16_t* cnt, void* stage_k, void* stage_v, hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(k_new, "k_new", 16)) || (rc = check_dev(v_new, "v_new", 16)) || (rc = check_dev(sel, "sel", 2)) ||
      (rc = check_dev(cnt, "cnt", 2)) || (rc = check_dev(stage_k, "stage_k", 16)) ||
      (rc = check_dev(stage_v, "stage_v", 16)))
    return rc;
  if (q_pos < 0 || q_pos >= shape->t_cap)
    return fail(SPARDA_ERR_INVALID_ARG, "q_pos %lld outside [0, t_cap)", (long long)q_pos);
  return hip_status(sparda::launch_stage_append(static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                                                sel, cnt, q_pos, static_cast<uint16_t*>(stage_k),
                                                static_cast<uint16_t*>(stage_v),
                                                (int64_t)shape->batch * shape->n_kv_heads, shape->k_total, stream),
                    "stage append launch");
}

int sparda_gather_blocks(const sparda_shape* shape, const void* host_k, const void* host_v, const int16_t* sel,
                         const int16_t* cnt, void* stage_k, void* stage_v, int32_t n_workgroups,
                         hipStream_t stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if ((rc = check_dev(host_k, "host_k", 16)) || (rc = check_dev(host_v, "host_v", 16)) ||
      (rc = check_dev(sel, "sel", 2)) || (rc = check_dev(cnt, "cnt", 2)) || (rc = check_dev(stage_k, "stage_k", 16)) ||
      (rc = check_dev(stage_v, "stage_v", 16)))
    return rc;
  if (n_workgroups < 1) return fail(SPARDA_ERR_INVALID_ARG, "n_workgroups %d < 1", n_workgroups);
  void* dev_ptr[2] = {nullptr, nullptr};
  if ((rc = mapped_pool(host_k, "host_k", pool_bytes(shape), &dev_ptr[0])) ||
      (rc = mapped_pool(host_v, "host_v", pool_bytes(shape), &dev_ptr[1])))
    return rc;
  return hip_status(sparda::launch_gather(static_cast<const uint16_t*>(dev_ptr[0]), static_cast<const uint16_t*>(dev_ptr[1]),
                                          sel, cnt, static_cast<uint16_t*>(stage_k), static_cast<uint16_t*>(stage_v),
                                          (int64_t)shape->batch * shape->n_kv_heads, shape->t_cap, shape->k_total,
                                          n_workgroups, stream),
                    "gather launch");
}

}  // extern "C"

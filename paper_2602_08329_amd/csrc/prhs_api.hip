// C-ABI entry points of libprhs: host-side validation, workspace sizing and
// dispatch to the kernel files.  Validation never touches the device, so every
// error path can be exercised without a GPU.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "prhs.h"
#include "prhs_internal.h"

namespace {

thread_local char g_err[512] = "";

prhs_status fail(prhs_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

prhs_status device_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return PRHS_OK;
  return fail(PRHS_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

prhs_status check_params(const prhs_params* p) {
  if (!p) return fail(PRHS_E_INVALID, "params is NULL");
  if (p->k < 0) return fail(PRHS_E_INVALID, "k must be >= 0 (got %d)", p->k);
  if (p->k_den < 0 || (p->k_den > 0 && p->k_num < 0))
    return fail(PRHS_E_INVALID, "proportional budget needs k_num >= 0, k_den > 0");
  if (p->sink < 0) return fail(PRHS_E_INVALID, "sink must be >= 0");
  if (p->window < 0) return fail(PRHS_E_INVALID, "window must be >= 0");
  if (p->dilate_r < 0) return fail(PRHS_E_INVALID, "dilate_r must be >= 0");
  if (p->refresh_every < 1) return fail(PRHS_E_INVALID, "refresh_every must be >= 1");
  if (p->layer_group < 1) return fail(PRHS_E_INVALID, "layer_group must be >= 1");
  return PRHS_OK;
}

// Shape-only checks of a KV descriptor (pointers checked by callers that read them).
prhs_status check_kv_shape(const prhs_kv* kv) {
  if (!kv) return fail(PRHS_E_INVALID, "kv is NULL");
  if (kv->batch < 0) return fail(PRHS_E_INVALID, "batch must be >= 0");
  if (kv->num_q_heads < 1 || kv->num_kv_heads < 1)
    return fail(PRHS_E_INVALID, "head counts must be >= 1");
  if (kv->num_q_heads % kv->num_kv_heads != 0)
    return fail(PRHS_E_INVALID, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)",
                kv->num_q_heads, kv->num_kv_heads);
  if (kv->num_q_heads / kv->num_kv_heads > 16)
    return fail(PRHS_E_UNSUPPORTED, "query heads per kv head must be <= 16");
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(PRHS_E_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", kv->head_dim);
  if (kv->dtype != PRHS_F32 && kv->dtype != PRHS_BF16)
    return fail(PRHS_E_UNSUPPORTED, "dtype must be PRHS_F32 or PRHS_BF16");
  if (kv->max_seq_len < 0 || kv->max_seq_len >= (1 << prhs::kIdxBits))
    return fail(PRHS_E_UNSUPPORTED, "max_seq_len must be in [0, 2^22)");
  // kernels address rows by 32-bit row ids
  const long long kRowLimit = 1LL << 31;
  if (kv->layout == PRHS_KV_CONTIGUOUS) {
    if (kv->capacity < kv->max_seq_len)
      return fail(PRHS_E_INVALID, "capacity (%d) < max_seq_len (%d)", kv->capacity, kv->max_seq_len);
    if ((long long)kv->batch * kv->num_kv_heads * kv->capacity >= kRowLimit)
      return fail(PRHS_E_UNSUPPORTED, "batch * num_kv_heads * capacity must be < 2^31");
  } else if (kv->layout == PRHS_KV_PAGED) {
    if (kv->page_size < 1) return fail(PRHS_E_INVALID, "page_size must be >= 1");
    if (kv->max_pages < 0 || (long long)kv->max_pages * kv->page_size < kv->max_seq_len)
      return fail(PRHS_E_INVALID, "max_pages * page_size < max_seq_len");
    if (kv->num_pages < 1) return fail(PRHS_E_INVALID, "num_pages must be >= 1");
    if ((long long)kv->num_pages * kv->num_kv_heads * kv->page_size >= kRowLimit)
      return fail(PRHS_E_UNSUPPORTED, "num_pages * num_kv_heads * page_size must be < 2^31");
  } else {
    return fail(PRHS_E_UNSUPPORTED, "unknown layout %d", kv->layout);
  }
  return PRHS_OK;
}

prhs_status check_kv_data(const prhs_kv* kv) {
  if (kv->batch == 0) return PRHS_OK;
  if (!kv->k || !kv->v) return fail(PRHS_E_INVALID, "k or v is NULL");
  if (!kv->seq_lens) return fail(PRHS_E_INVALID, "seq_lens is NULL");
  if (kv->layout == PRHS_KV_PAGED && !kv->block_table)
    return fail(PRHS_E_INVALID, "block_table is NULL for a paged cache");
  return PRHS_OK;
}

prhs::KvView view_of(const prhs_kv* kv) {
  prhs::KvView v;
  v.k = kv->k;
  v.v = kv->v;
  v.table = kv->block_table;
  v.seq_lens = kv->seq_lens;
  v.batch = kv->batch;
  v.hq = kv->num_q_heads;
  v.hkv = kv->num_kv_heads;
  v.d = kv->head_dim;
  v.capacity = kv->capacity;
  v.page_size = kv->page_size;
  v.max_pages = kv->max_pages;
  v.num_pages = kv->num_pages;
  v.max_seq_len = kv->max_seq_len;
  v.paged = kv->layout == PRHS_KV_PAGED ? 1 : 0;
  return v;
}

long long budget_at(const prhs_params* p, long long n0) {
  return p->k_den > 0 ? ((long long)p->k_num * n0) / p->k_den : (long long)p->k;
}

long long middle_at(const prhs_params* p, long long n0) {
  const long long sink_end = p->sink < n0 ? p->sink : n0;
  long long win_start = n0 - p->window;
  if (win_start < sink_end) win_start = sink_end;
  return win_start - sink_end;
}

// Eq. psaw's factor 1 - phi^e of the layer, with e = alpha (l - l_s) /
// (N - l_s) for the 1-based layer l = layer + 1 >= l_s, else 0 (no mask).
// The order of operations is that of the formula, in binary64.
prhs_status psaw_factor(const prhs_psaw* p, double* f) {
  if (!p) return fail(PRHS_E_INVALID, "psaw is NULL");
  if (p->num_layers < 1) return fail(PRHS_E_INVALID, "psaw: num_layers must be >= 1");
  if (p->layer < 0 || p->layer >= p->num_layers)
    return fail(PRHS_E_INVALID, "psaw: layer (%d) must lie in [0, num_layers = %d)", p->layer,
                p->num_layers);
  if (p->l_s < 0 || p->l_s >= p->num_layers)
    return fail(PRHS_E_INVALID, "psaw: l_s (%d) must lie in [0, num_layers = %d)", p->l_s,
                p->num_layers);
  if (p->sink < 0) return fail(PRHS_E_INVALID, "psaw: sink must be >= 0");
  if (!(p->phi > 0.0 && p->phi <= 1.0)) return fail(PRHS_E_INVALID, "psaw: phi must lie in (0, 1]");
  if (!(p->alpha >= 0.0 && p->alpha <= 1e300))
    return fail(PRHS_E_INVALID, "psaw: alpha must be finite and >= 0");
  const int lb = p->layer + 1;
  if (lb < p->l_s) {
    *f = 0.0;
    return PRHS_OK;
  }
  const double e = p->alpha * (double)(lb - p->l_s) / (double)(p->num_layers - p->l_s);
  *f = 1.0 - pow(p->phi, e);
  return PRHS_OK;
}

}  // namespace

extern "C" {

int32_t prhs_abi_version(void) { return PRHS_ABI_VERSION; }

const char* prhs_last_error(void) { return g_err; }

int32_t prhs_max_topk(const prhs_params* p, int32_t max_seq_len) {
  if (check_params(p) != PRHS_OK || max_seq_len < 0) return -1;
  // both the budget and the middle length grow with n0, so their minimum
  // peaks at the longest sequence
  long long kb = budget_at(p, max_seq_len);
  const long long mid = middle_at(p, max_seq_len);
  if (kb > mid) kb = mid;
  if (kb < 0) kb = 0;
  return (int32_t)kb;
}

int32_t prhs_set_capacity(const prhs_params* p, int32_t max_seq_len) {
  if (check_params(p) != PRHS_OK || max_seq_len < 0) return -1;
  const long long kb = budget_at(p, max_seq_len);
  long long m = p->dilate_m < 0 ? kb / 3 : p->dilate_m;
  if (m > kb) m = kb;
  long long cap = (long long)p->sink + kb + 2LL * p->dilate_r * m + p->window + (p->refresh_every - 1);
  if (cap > max_seq_len) cap = max_seq_len;
  return (int32_t)cap;
}

int32_t prhs_schedule(int32_t step, int32_t layer, const prhs_params* p) {
  if (check_params(p) != PRHS_OK || step < 0 || layer < 0) return -1;
  return (step % p->refresh_every == 0 && layer % p->layer_group == 0) ? PRHS_REFRESH : PRHS_REUSE;
}

int32_t prhs_psaw_first_visible(const prhs_psaw* psaw, int32_t n) {
  double f = 0.0;
  if (psaw_factor(psaw, &f) != PRHS_OK) return -1;
  if (n < 0) {
    fail(PRHS_E_INVALID, "n must be >= 0");
    return -1;
  }
  return prhs::psaw_first_visible(f, psaw->sink, n);
}

prhs_status prhs_workspace_size(int32_t op, const prhs_kv* kv, const prhs_params* params,
                                int32_t set_cap, size_t* bytes) {
  if (!bytes) return fail(PRHS_E_INVALID, "bytes is NULL");
  *bytes = 0;
  switch (op) {
    case PRHS_OP_SELECT: {
      prhs_status st = check_kv_shape(kv);
      if (st != PRHS_OK) return st;
      if ((st = check_params(params)) != PRHS_OK) return st;
      *bytes = prhs::select_workspace_bytes(kv->batch * kv->num_kv_heads, kv->max_seq_len,
                                            prhs_max_topk(params, kv->max_seq_len));
      return PRHS_OK;
    }
    case PRHS_OP_DILATE_REUSE:
      return PRHS_OK;
    case PRHS_OP_SPARSE_ATTN: {
      prhs_status st = check_kv_shape(kv);
      if (st != PRHS_OK) return st;
      if (set_cap < 0) return fail(PRHS_E_INVALID, "set_cap must be >= 0");
      *bytes = prhs::attn_workspace_bytes(kv->dtype, false, kv->batch, kv->num_q_heads,
                                          kv->num_kv_heads, kv->head_dim, set_cap);
      return PRHS_OK;
    }
    case PRHS_OP_DENSE_ATTN: {
      prhs_status st = check_kv_shape(kv);
      if (st != PRHS_OK) return st;
      *bytes = prhs::attn_workspace_bytes(kv->dtype, true, kv->batch, kv->num_q_heads,
                                          kv->num_kv_heads, kv->head_dim, kv->max_seq_len);
      return PRHS_OK;
    }
    default:
      return fail(PRHS_E_INVALID, "unknown op %d", op);
  }
}

static prhs_status select_common(const prhs_kv* kv, const void* q, const prhs_params* params,
                                 int32_t* topk_idx, int32_t* topk_len, int32_t k_cap,
                                 int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                                 int32_t* shared_idx, int32_t* shared_len, bool shared,
                                 const int32_t* row_choice, const prhs::GateLaunch* gate,
                                 void* ws, size_t ws_bytes, void* stream, const char* name) {
  prhs_status st = check_kv_shape(kv);
  if (st != PRHS_OK) return st;
  if ((st = check_params(params)) != PRHS_OK) return st;
  if ((st = check_kv_data(kv)) != PRHS_OK) return st;
  if (kv->batch > 0 && (!q || !topk_idx || !topk_len || !set_idx || !set_len))
    return fail(PRHS_E_INVALID, "q, topk_idx, topk_len, set_idx and set_len must be non-NULL");
  if (shared && kv->batch > 0 && (!shared_idx || !shared_len))
    return fail(PRHS_E_INVALID, "shared_idx and shared_len must be non-NULL");
  const int32_t kmax = prhs_max_topk(params, kv->max_seq_len);
  if (kmax > PRHS_MAX_TOPK)
    return fail(PRHS_E_UNSUPPORTED, "top-k of %d exceeds the sort limit %d", kmax, PRHS_MAX_TOPK);
  if (k_cap < kmax || k_cap < 0)
    return fail(PRHS_E_CAPACITY, "k_cap (%d) < largest top-k (%d)", k_cap, kmax);
  long long need = (long long)params->sink + kmax + params->window;
  if (need > kv->max_seq_len) need = kv->max_seq_len;
  if (shared) need = prhs_set_capacity(params, kv->max_seq_len);
  if (set_cap < need || set_cap < 0)
    return fail(PRHS_E_CAPACITY, "set_cap (%d) < %s bound (%lld)", set_cap,
                shared ? "shared set" : "anchor set", need);
  const size_t wsz = prhs::select_workspace_bytes(kv->batch * kv->num_kv_heads, kv->max_seq_len, kmax);
  if (kv->batch > 0 && (!ws || ws_bytes < wsz))
    return fail(PRHS_E_WORKSPACE, "workspace of %zu bytes needed (got %zu)", wsz, ws_bytes);
  if (kv->batch == 0) return PRHS_OK;
  prhs::SelectLaunch a;
  a.kv = view_of(kv);
  a.q = q;
  a.dtype = kv->dtype;
  a.k = params->k;
  a.k_num = params->k_num;
  a.k_den = params->k_den;
  a.sink = params->sink;
  a.window = params->window;
  a.dilate_m = params->dilate_m;
  a.topk_idx = topk_idx;
  a.topk_len = topk_len;
  a.k_cap = k_cap;
  a.set_idx = set_idx;
  a.set_len = set_len;
  a.set_cap = set_cap;
  a.dilate_r = params->dilate_r;
  a.shared_idx = shared ? shared_idx : nullptr;
  a.shared_len = shared ? shared_len : nullptr;
  a.row_choice = row_choice;
  a.gate = gate;
  a.ws = ws;
  a.max_topk = kmax;
  return device_status(prhs::launch_select(a, (hipStream_t)stream), name);
}

prhs_status prhs_select(const prhs_kv* kv, const void* q, const prhs_params* params,
                        int32_t* topk_idx, int32_t* topk_len, int32_t k_cap, int32_t* set_idx,
                        int32_t* set_len, int32_t set_cap, void* ws, size_t ws_bytes,
                        void* stream) {
  return select_common(kv, q, params, topk_idx, topk_len, k_cap, set_idx, set_len, set_cap,
                       nullptr, nullptr, false, nullptr, nullptr, ws, ws_bytes, stream,
                       "prhs_select launch");
}

prhs_status prhs_select_shared(const prhs_kv* kv, const void* q, const prhs_params* params,
                               int32_t* topk_idx, int32_t* topk_len, int32_t k_cap,
                               int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                               int32_t* shared_idx, int32_t* shared_len, void* ws,
                               size_t ws_bytes, void* stream) {
  return select_common(kv, q, params, topk_idx, topk_len, k_cap, set_idx, set_len, set_cap,
                       shared_idx, shared_len, true, nullptr, nullptr, ws, ws_bytes, stream,
                       "prhs_select_shared launch");
}

prhs_status prhs_select_gated(const prhs_kv* kv, const void* q, const prhs_params* params,
                              const int32_t* choice, int32_t* topk_idx, int32_t* topk_len,
                              int32_t k_cap, int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                              int32_t* shared_idx, int32_t* shared_len, void* ws,
                              size_t ws_bytes, void* stream) {
  if (kv && kv->batch > 0 && !choice) return fail(PRHS_E_INVALID, "choice must be non-NULL");
  return select_common(kv, q, params, topk_idx, topk_len, k_cap, set_idx, set_len, set_cap,
                       shared_idx, shared_len, true, choice, nullptr, ws, ws_bytes, stream,
                       "prhs_select_gated launch");
}

prhs_status prhs_dilate_reuse(const prhs_params* params, int32_t batch, int32_t num_kv_heads,
                              const int32_t* topk_idx, const int32_t* topk_len, int32_t k_cap,
                              const int32_t* anchor_lens, const int32_t* seq_lens,
                              int32_t* set_idx, int32_t* set_len, int32_t set_cap, void* stream) {
  prhs_status st = check_params(params);
  if (st != PRHS_OK) return st;
  if (batch < 0 || num_kv_heads < 1) return fail(PRHS_E_INVALID, "batch >= 0 and num_kv_heads >= 1 required");
  if (k_cap < 0 || set_cap < 0) return fail(PRHS_E_INVALID, "k_cap and set_cap must be >= 0");
  if (batch > 0 && (!topk_idx || !topk_len || !anchor_lens || !seq_lens || !set_idx || !set_len))
    return fail(PRHS_E_INVALID, "device arrays must be non-NULL");
  if (batch == 0) return PRHS_OK;
  prhs::DilateLaunch a;
  a.batch = batch;
  a.hkv = num_kv_heads;
  a.topk_idx = topk_idx;
  a.topk_len = topk_len;
  a.k_cap = k_cap;
  a.anchor_lens = anchor_lens;
  a.seq_lens = seq_lens;
  a.set_idx = set_idx;
  a.set_len = set_len;
  a.set_cap = set_cap;
  a.k = params->k;
  a.k_num = params->k_num;
  a.k_den = params->k_den;
  a.sink = params->sink;
  a.window = params->window;
  a.dilate_m = params->dilate_m;
  a.dilate_r = params->dilate_r;
  return device_status(prhs::launch_dilate_reuse(a, (hipStream_t)stream), "prhs_dilate_reuse launch");
}

static prhs_status attention_common(const prhs_kv* kv, const void* q, const int32_t* set_idx,
                                    const int32_t* set_len, int32_t set_cap,
                                    const int32_t* tail_start, const int32_t* unit_row,
                                    const int32_t* unit_tail, int32_t pool_rows,
                                    const int32_t* unit_gate, int32_t units_side,
                                    const prhs_psaw* psaw, float scale,
                                    float* out, float* lse, void* ws, size_t ws_bytes,
                                    void* stream, bool dense, const char* name) {
  prhs_status st = check_kv_shape(kv);
  if (st != PRHS_OK) return st;
  if ((st = check_kv_data(kv)) != PRHS_OK) return st;
  if (kv->batch > 0 && (!q || !out)) return fail(PRHS_E_INVALID, "q and out must be non-NULL");
  if (!dense) {
    if (set_cap < 0) return fail(PRHS_E_INVALID, "set_cap must be >= 0");
    if (kv->batch > 0 && (!set_idx || !set_len))
      return fail(PRHS_E_INVALID, "set_idx and set_len must be non-NULL");
  }
  if (!(scale == scale)) return fail(PRHS_E_INVALID, "scale is NaN");
  double psaw_f = 0.0;
  if (psaw && (st = psaw_factor(psaw, &psaw_f)) != PRHS_OK) return st;
  const int rows_cap = dense ? kv->max_seq_len : set_cap;
  const size_t wsz = prhs::attn_workspace_bytes(kv->dtype, dense, kv->batch, kv->num_q_heads,
                                                kv->num_kv_heads, kv->head_dim, rows_cap);
  if (kv->batch > 0 && (!ws || ws_bytes < wsz))
    return fail(PRHS_E_WORKSPACE, "workspace of %zu bytes needed (got %zu)", wsz, ws_bytes);
  if (kv->batch == 0) return PRHS_OK;
  prhs::AttnLaunch a;
  a.kv = view_of(kv);
  a.q = q;
  a.dtype = kv->dtype;
  a.set_idx = set_idx;
  a.set_len = set_len;
  a.tail_start = tail_start;
  a.unit_row = unit_row;
  a.unit_tail = unit_tail;
  a.pool_rows = pool_rows;
  a.unit_gate = unit_gate;
  a.units_side = units_side;
  a.psaw = psaw != nullptr;
  a.psaw_f = psaw_f;
  a.psaw_sink = psaw ? psaw->sink : 0;
  a.set_cap = set_cap;
  a.scale = scale;
  a.out = out;
  a.lse = lse;
  a.ws = ws;
  return device_status(prhs::launch_attention(a, dense, (hipStream_t)stream), name);
}

prhs_status prhs_sparse_decode_attn(const prhs_kv* kv, const void* q, const int32_t* set_idx,
                                    const int32_t* set_len, int32_t set_cap, float scale,
                                    float* out, float* lse, void* ws, size_t ws_bytes,
                                    void* stream) {
  return attention_common(kv, q, set_idx, set_len, set_cap, nullptr, nullptr, nullptr, 0, nullptr,
                          0, nullptr, scale, out, lse, ws, ws_bytes, stream, false,
                          "prhs_sparse_decode_attn launch");
}

prhs_status prhs_sparse_decode_attn_static(const prhs_kv* kv, const void* q,
                                           const int32_t* set_idx, const int32_t* set_len,
                                           int32_t set_cap, float scale, float* out, float* lse,
                                           void* stream) {
  prhs_status st = check_kv_shape(kv);
  if (st != PRHS_OK) return st;
  if (set_cap < 0) return fail(PRHS_E_INVALID, "set_cap must be >= 0");
  const size_t need = prhs::attn_workspace_bytes(kv->dtype, false, kv->batch, kv->num_q_heads,
                                                 kv->num_kv_heads, kv->head_dim, set_cap);
  if (need > prhs::kStaticScratchBytes)
    return fail(PRHS_E_UNSUPPORTED,
                "split-K partials of %zu bytes exceed the static scratch of %zu bytes", need,
                prhs::kStaticScratchBytes);
  if (kv->batch == 0) return attention_common(kv, q, set_idx, set_len, set_cap, nullptr, nullptr,
                                              nullptr, 0, nullptr, 0, nullptr, scale, out, lse,
                                              nullptr, 0, stream, false,
                                              "prhs_sparse_decode_attn_static");
  void* ws = nullptr;
  if ((st = device_status(prhs::attn_static_scratch(&ws), "static scratch lookup")) != PRHS_OK)
    return st;
  return attention_common(kv, q, set_idx, set_len, set_cap, nullptr, nullptr, nullptr, 0, nullptr,
                          0, nullptr, scale, out, lse, ws, prhs::kStaticScratchBytes, stream, false,
                          "prhs_sparse_decode_attn_static launch");
}

prhs_status prhs_reuse_decode_attn(const prhs_kv* kv, const void* q, const int32_t* set_idx,
                                   const int32_t* set_len, int32_t set_cap,
                                   const int32_t* anchor_lens, float scale, float* out, float* lse,
                                   void* ws, size_t ws_bytes, void* stream) {
  if (kv && kv->batch > 0 && !anchor_lens)
    return fail(PRHS_E_INVALID, "anchor_lens must be non-NULL");
  return attention_common(kv, q, set_idx, set_len, set_cap, anchor_lens, nullptr, nullptr, 0,
                          nullptr, 0, nullptr, scale, out, lse, ws, ws_bytes, stream, false,
                          "prhs_reuse_decode_attn launch");
}

prhs_status prhs_pool_decode_attn(const prhs_kv* kv, const void* q, const int32_t* pool_idx,
                                  const int32_t* pool_len, int32_t pool_rows, int32_t set_cap,
                                  const int32_t* unit_row, const int32_t* unit_tail,
                                  const int32_t* unit_gate, int32_t units_side,
                                  const prhs_psaw* psaw, float scale, float* out, float* lse,
                                  void* ws, size_t ws_bytes, void* stream) {
  if (pool_rows < 0) return fail(PRHS_E_INVALID, "pool_rows must be >= 0");
  if (kv && kv->batch > 0 && (!unit_row || !unit_tail))
    return fail(PRHS_E_INVALID, "unit_row and unit_tail must be non-NULL");
  if (units_side != PRHS_UNITS_ALL && units_side != PRHS_UNITS_RETRIEVING &&
      units_side != PRHS_UNITS_SHARING)
    return fail(PRHS_E_INVALID, "units_side must be PRHS_UNITS_ALL, _RETRIEVING or _SHARING");
  if (units_side != PRHS_UNITS_ALL && kv && kv->batch > 0 && !unit_gate)
    return fail(PRHS_E_INVALID, "unit_gate must be non-NULL with a units_side filter");
  return attention_common(kv, q, pool_idx, pool_len, set_cap, nullptr, unit_row, unit_tail,
                          pool_rows, unit_gate, units_side, psaw, scale, out, lse, ws, ws_bytes,
                          stream, false, "prhs_pool_decode_attn launch");
}

static prhs_status gate_args(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                             int32_t head_dim, int32_t dtype, const void* q,
                             const int32_t* seq_lens, double tau, int32_t num_slots, int32_t slot,
                             void* ref_q, int32_t* ref_valid, int32_t* slot_lens, int32_t* choice,
                             int32_t* row_anchor, int32_t* row_other, int32_t* tail,
                             int32_t record, prhs::GateLaunch* a) {
  if (batch < 0) return fail(PRHS_E_INVALID, "batch must be >= 0");
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0)
    return fail(PRHS_E_INVALID, "num_q_heads must be a positive multiple of num_kv_heads");
  if (head_dim < 1) return fail(PRHS_E_INVALID, "head_dim must be >= 1");
  if (dtype != PRHS_F32 && dtype != PRHS_BF16) return fail(PRHS_E_UNSUPPORTED, "dtype %d", dtype);
  if (!(tau >= 0.0 && tau <= 1.0)) return fail(PRHS_E_INVALID, "tau must lie in [0, 1]");
  if (num_slots < 1 || slot < 0 || slot >= num_slots)
    return fail(PRHS_E_INVALID, "slot (%d) must lie in [0, num_slots = %d)", slot, num_slots);
  if ((long long)2 * num_slots * batch * num_kv_heads >= (1LL << 31))
    return fail(PRHS_E_UNSUPPORTED, "set pool rows exceed 32-bit indices");
  if (batch > 0 && (!q || !seq_lens || !ref_q || !ref_valid || !slot_lens || !choice ||
                    !row_anchor || !row_other || !tail))
    return fail(PRHS_E_INVALID, "device arrays must be non-NULL");
  a->batch = batch;
  a->hq = num_q_heads;
  a->hkv = num_kv_heads;
  a->d = head_dim;
  a->dtype = dtype;
  a->q = q;
  a->seq_lens = seq_lens;
  a->tau = tau;
  a->num_slots = num_slots;
  a->slot = slot;
  a->ref_q = ref_q;
  a->ref_valid = ref_valid;
  a->slot_lens = slot_lens;
  a->choice = choice;
  a->row_anchor = row_anchor;
  a->row_other = row_other;
  a->tail = tail;
  a->record = record ? 1 : 0;
  return PRHS_OK;
}

prhs_status prhs_gate(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                      int32_t dtype, const void* q, const int32_t* seq_lens, double tau,
                      int32_t num_slots, int32_t slot, void* ref_q, int32_t* ref_valid,
                      int32_t* slot_lens, int32_t* choice, int32_t* row_anchor,
                      int32_t* row_other, int32_t* tail, int32_t record, void* stream) {
  prhs::GateLaunch a;
  prhs_status st = gate_args(batch, num_q_heads, num_kv_heads, head_dim, dtype, q, seq_lens, tau,
                             num_slots, slot, ref_q, ref_valid, slot_lens, choice, row_anchor,
                             row_other, tail, record, &a);
  if (st != PRHS_OK || batch == 0) return st;
  return device_status(prhs::launch_gate(a, (hipStream_t)stream), "prhs_gate launch");
}

prhs_status prhs_gate_select(const prhs_kv* kv, const void* q, const prhs_params* params,
                             double tau, int32_t num_slots, int32_t slot, void* ref_q,
                             int32_t* ref_valid, int32_t* slot_lens, int32_t* choice,
                             int32_t* row_anchor, int32_t* row_other, int32_t* tail,
                             int32_t* topk_idx, int32_t* topk_len, int32_t k_cap,
                             int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                             int32_t* shared_idx, int32_t* shared_len, void* ws, size_t ws_bytes,
                             void* stream) {
  prhs_status st = check_kv_shape(kv);
  if (st != PRHS_OK) return st;
  prhs::GateLaunch g;
  st = gate_args(kv->batch, kv->num_q_heads, kv->num_kv_heads, kv->head_dim, kv->dtype, q,
                 kv->seq_lens, tau, num_slots, slot, ref_q, ref_valid, slot_lens, choice,
                 row_anchor, row_other, tail, 1, &g);
  if (st != PRHS_OK) return st;
  return select_common(kv, q, params, topk_idx, topk_len, k_cap, set_idx, set_len, set_cap,
                       shared_idx, shared_len, true, nullptr, &g, ws, ws_bytes, stream,
                       "prhs_gate_select launch");
}

prhs_status prhs_prefill_attn(const prhs_kv* kv, const void* q, int32_t q_len,
                              const prhs_psaw* psaw, float scale, float* out, float* lse,
                              void* stream) {
  prhs_status st = check_kv_shape(kv);
  if (st != PRHS_OK) return st;
  if ((st = check_kv_data(kv)) != PRHS_OK) return st;
  if (kv->dtype != PRHS_BF16)
    return fail(PRHS_E_UNSUPPORTED, "prefill attention is built for bf16 inputs");
  if (q_len < 0) return fail(PRHS_E_INVALID, "q_len must be >= 0 (got %d)", q_len);
  double psaw_f = 0.0;
  if (psaw && (st = psaw_factor(psaw, &psaw_f)) != PRHS_OK) return st;
  if (!(scale > 0.f && scale < INFINITY))
    return fail(PRHS_E_INVALID, "scale must be positive and finite");
  if ((long long)((q_len + 63) / 64) * kv->batch * kv->num_q_heads > 0x7FFFFFFFLL)
    return fail(PRHS_E_UNSUPPORTED, "ceil(q_len / 64) * batch * num_q_heads must be < 2^31");
  if (kv->batch == 0 || q_len == 0) return PRHS_OK;
  if (!q || !out) return fail(PRHS_E_INVALID, "q and out must be non-NULL");
  prhs::PrefillLaunch a;
  a.kv = view_of(kv);
  a.q = q;
  a.T = q_len;
  a.psaw = psaw != nullptr;
  a.psaw_f = psaw_f;
  a.sink = psaw ? psaw->sink : 0;
  a.scale = scale;
  a.out = out;
  a.lse = lse;
  return device_status(prhs::launch_prefill(a, (hipStream_t)stream), "prhs_prefill_attn launch");
}

prhs_status prhs_dense_decode_attn(const prhs_kv* kv, const void* q, float scale, float* out,
                                   float* lse, void* ws, size_t ws_bytes, void* stream) {
  return attention_common(kv, q, nullptr, nullptr, 0, nullptr, nullptr, nullptr, 0, nullptr, 0,
                          nullptr, scale, out, lse, ws, ws_bytes, stream, true,
                          "prhs_dense_decode_attn launch");
}

}  // extern "C"

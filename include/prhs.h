/*
 * prhs.h -- C ABI of libprhs, the MI355X (gfx950) decode hot path of
 * Pre-hoc Sparsity (PrHS): per-KV-head top-k selection, union with sink and
 * recency window, reuse of the selection across decode steps (with neighbour
 * dilation) and across a group of layers, and gather-sparse decode attention.
 *
 * Paper: "Near-Oracle KV Selection via Pre-hoc Sparsity for Long-Context
 * Inference" (arXiv 2602.08329).  Each entry point cites the passage that
 * defines the operation it computes.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers named for tensors (q, k, v, block_table, seq_lens, topk_*, set_*,
 *   out, lse, ws) are DEVICE pointers.  Descriptor structs (prhs_kv,
 *   prhs_params) and size outputs are HOST memory.  No ROCm header is needed:
 *   the stream is passed as void* (a hipStream_t; NULL is the null stream).
 * - The caller owns every buffer.  The library allocates no device memory and
 *   keeps no state between calls; calls on different streams with different
 *   buffers may run concurrently.  Calls sharing a workspace must be ordered.
 * - Workspaces need no initialisation, with one exception: a selection
 *   workspace (PRHS_OP_SELECT) begins with per-row histograms and counters,
 *   2 x align256(R x 8192) + align256(R x 16) bytes for R = batch x
 *   num_kv_heads rows, which must be zero when a call starts and which every
 *   call leaves zero.  Zero-fill a selection workspace before its first use,
 *   and again before a call with more rows than the calls it served so far.
 * - Every call is asynchronous on `stream`; results are valid once the stream
 *   has synchronised.  No call synchronises internally.
 * - Positions are 0-based.  A sequence of current length n attends keys
 *   [0, n): the current token's own key/value is already in the cache (the
 *   sum of Eq. attn_eq runs up to and including the current step).
 * - Argument validation happens on the host before any device work and
 *   returns PRHS_E_INVALID / PRHS_E_UNSUPPORTED / PRHS_E_CAPACITY /
 *   PRHS_E_WORKSPACE; a failed launch returns PRHS_E_DEVICE.  The message of
 *   the last non-OK status of the calling thread is in prhs_last_error().
 * - Device-array preconditions the host cannot see: 0 <= seq_lens[b] <=
 *   max_seq_len, anchor_lens[b] <= seq_lens[b], block-table entries in
 *   [0, num_pages), set indices < seq_lens[b].  Kernels clamp lengths to the
 *   host-declared bounds and skip out-of-range rows instead of reading out of
 *   bounds.  The attention entry points then attend exactly the remaining
 *   valid positions (set entries outside [0, n) and positions on pages
 *   outside the pool are left out); selection results for inputs that break
 *   a precondition are unspecified.
 */
#ifndef PRHS_H_
#define PRHS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PRHS_ABI_VERSION 2

typedef enum prhs_status {
  PRHS_OK = 0,
  PRHS_E_INVALID = -1,      /* null pointer, negative size, inconsistent shape */
  PRHS_E_UNSUPPORTED = -2,  /* head_dim, dtype, group size or k outside what is built */
  PRHS_E_CAPACITY = -3,     /* k_cap or set_cap smaller than the bound the call needs */
  PRHS_E_WORKSPACE = -4,    /* ws null or smaller than prhs_workspace_size() */
  PRHS_E_DEVICE = -5        /* kernel launch failed; see prhs_last_error() */
} prhs_status;

typedef enum prhs_dtype {
  PRHS_F32 = 0,   /* q, K and V in fp32 */
  PRHS_BF16 = 1   /* q, K and V in bf16; all outputs stay fp32 */
} prhs_dtype;

typedef enum prhs_layout {
  PRHS_KV_CONTIGUOUS = 0,  /* K, V: [batch][num_kv_heads][capacity][head_dim] */
  PRHS_KV_PAGED = 1        /* K, V: [num_pages][num_kv_heads][page_size][head_dim];
                              token i of sequence b lives in page
                              block_table[b * max_pages + i / page_size],
                              slot i % page_size */
} prhs_layout;

/* The KV cache of one layer (Sec. 2.1: K^h, V^h in R^{L x d} per head). */
typedef struct prhs_kv {
  int32_t batch;          /* B >= 0 */
  int32_t num_q_heads;    /* Hq >= 1 */
  int32_t num_kv_heads;   /* Hkv >= 1, Hq % Hkv == 0; query head h reads kv head h / (Hq/Hkv) */
  int32_t head_dim;       /* d: 64 or 128 */
  int32_t dtype;          /* prhs_dtype */
  int32_t layout;         /* prhs_layout */
  int32_t capacity;       /* contiguous: token stride per (b, kv head); >= max_seq_len */
  int32_t page_size;      /* paged: tokens per page (>= 1) */
  int32_t max_pages;      /* paged: row length of block_table; max_pages*page_size >= max_seq_len */
  int32_t num_pages;      /* paged: physical pages in K and V */
  const void* k;
  const void* v;
  const int32_t* block_table;  /* paged: [batch][max_pages] int32; ignored when contiguous */
  const int32_t* seq_lens;     /* [batch] current length n_b (includes the current token) */
  int32_t max_seq_len;         /* host-known bound on seq_lens; < 2^22 */
} prhs_kv;

/* Selection budget and reuse schedule (Sec. 4.1; defaults of Sec. 5.1). */
typedef struct prhs_params {
  int32_t k;              /* middle budget when k_den == 0 */
  int32_t k_num, k_den;   /* k_den > 0: per-sequence budget k_b = floor(k_num * n0_b / k_den) */
  int32_t sink;           /* C_sink: positions [0, sink) are always kept */
  int32_t window;         /* C_local: positions [n0 - window, n0) at the anchor */
  int32_t dilate_m;       /* top-m winners that are dilated; < 0 means floor(k_b / 3) */
  int32_t dilate_r;       /* dilation radius r >= 0 */
  int32_t refresh_every;  /* s >= 1: decode steps j with j % s == 0 refresh */
  int32_t layer_group;    /* G >= 1: layers l with l % G == 0 anchor their group */
} prhs_params;

/* Progressive sliding attention window of one layer (Sec. 4.2, Eq. psaw).
 * For the layer with 0-based index `layer` of a model with `num_layers`
 * layers, Eq. psaw's 1-based layer is l = layer + 1 and, at t tokens in view,
 *   P_l(t) = floor((1 - phi^(alpha (l - l_s) / (N - l_s))) t)  for l >= l_s,
 *   P_l(t) = 0                                                  otherwise.
 * The window masks the 1-based positions strictly between C_sink and P, i.e.
 * the 0-based range [sink, P - 1): the visible keys are
 *   [0, min(sink, t)) U [first_visible, t),
 *   first_visible = max(min(sink, t), P_l(t) - 1).
 * The library evaluates the factor 1 - phi^e once per call on the host in
 * binary64 (C pow) and P = floor(factor * t) in binary64 wherever it needs
 * it, host or device, so every position agrees with the same formula
 * evaluated in binary64.  Sec. 5.1's defaults: l_s = floor(3N/4), phi = 0.7,
 * alpha = 1. */
typedef struct prhs_psaw {
  int32_t layer;       /* 0 <= layer < num_layers (0-based) */
  int32_t num_layers;  /* N >= 1 */
  int32_t l_s;         /* pruning depth, 1-based: 0 <= l_s < N */
  int32_t sink;        /* C_sink >= 0 */
  double phi;          /* 0 < phi <= 1 */
  double alpha;        /* alpha >= 0, finite */
} prhs_psaw;

enum {
  PRHS_OP_SELECT = 0,
  PRHS_OP_DILATE_REUSE = 1,
  PRHS_OP_SPARSE_ATTN = 2,
  PRHS_OP_DENSE_ATTN = 3
};

enum { PRHS_REUSE = 0, PRHS_REFRESH = 1 };

/* Which units a pool attention launch attends (prhs_pool_decode_attn). */
enum { PRHS_UNITS_ALL = 0, PRHS_UNITS_RETRIEVING = 1, PRHS_UNITS_SHARING = 2 };

/* Largest top-k budget the selection supports: k_b, after clamping to the
 * middle range length, must not exceed this (PRHS_E_UNSUPPORTED otherwise).
 * For middle ranges beyond one CU's LDS the selection keeps the k_b winners
 * as 8-byte (score, position) pairs in LDS next to its bitmap segment, which
 * bounds k_b. */
#define PRHS_MAX_TOPK 16000

/* ABI version of the loaded library (PRHS_ABI_VERSION). */
int32_t prhs_abi_version(void);

/* Largest middle budget k_b any sequence of length <= max_seq_len gets, after
 * clamping to the middle range; the minimum k_cap for prhs_select.  Returns
 * -1 when params is NULL or inconsistent. */
int32_t prhs_max_topk(const prhs_params* params, int32_t max_seq_len);

/* Smallest set_cap that holds every index set the schedule produces when each
 * call's current length exceeds its anchor length by at most
 * refresh_every - 1: min(max_seq_len, sink + k + 2*r*m + window +
 * refresh_every - 1) (the dilated-set size of the CIS parameterisation
 * appendix plus the tokens decoded since the anchor).  -1 on bad arguments. */
int32_t prhs_set_capacity(const prhs_params* params, int32_t max_seq_len);

/* Device workspace in bytes that entry point `op` (PRHS_OP_*) needs for this
 * cache shape; set_cap is used by PRHS_OP_SPARSE_ATTN only.  0 bytes is a
 * valid answer (ws may then be NULL). */
prhs_status prhs_workspace_size(int32_t op, const prhs_kv* kv, const prhs_params* params,
                                int32_t set_cap, size_t* bytes);

/* Block schedule of CIS (Sec. 4.1): PRHS_REFRESH when decode step `step`
 * opens a block of refresh_every steps and `layer` opens a group of
 * layer_group layers, else PRHS_REUSE.  -1 on bad arguments. */
int32_t prhs_schedule(int32_t step, int32_t layer, const prhs_params* params);

/* Eq. psaw (Sec. 4.2): the first visible non-sink 0-based position of the
 * layer described by `psaw` when n tokens are in view (a decode step at
 * length n, or the prefill query at position n - 1), as defined at
 * prhs_psaw.  Host function.  -1 when psaw is NULL or invalid or n < 0
 * (prhs_last_error() then says why). */
int32_t prhs_psaw_first_visible(const prhs_psaw* psaw, int32_t n);

/* Refresh: score, top-k and anchor set for one layer (Sec. 4.1 Selection
 * Criteria; top-k oracle of Sec. 2.3).
 *
 * For every (b, kv head g) with anchor length n0 = seq_lens[b]:
 *   sigma_i = max over the g-th group's query heads h of q[b][h] . k_i (raw
 *   dot product, computed in fp32) for i in the middle range
 *   [min(sink, n0), max(min(sink, n0), n0 - window));
 *   S* = the min(k_b, middle length) positions of largest sigma, ties going
 *   to the lower position (total order: sigma descending, position
 *   ascending); with m = min(dilate_m or floor(k_b / 3), |S*|),
 *   topk_idx[b][g][0 .. m) = the m highest-ranked members of S* and
 *   topk_idx[b][g][m .. topk_len) = the others, each part in ascending
 *   position order (only the set of the top m matters to the dilation);
 *   set_idx[b][g][0 .. set_len) = sink U top-k U [n0 - window, n0),
 *   ascending and without duplicates (the critical set C_t).
 * q: [batch][num_q_heads][head_dim] in kv->dtype.
 * topk_idx: [batch][num_kv_heads][k_cap] int32, k_cap >= prhs_max_topk().
 * topk_len: [batch][num_kv_heads] int32.
 * set_idx: [batch][num_kv_heads][set_cap] int32, set_cap >= min(max_seq_len,
 *   sink + prhs_max_topk() + window).  set_len: [batch][num_kv_heads] int32.
 * ws: >= prhs_workspace_size(PRHS_OP_SELECT) bytes; its leading histogram
 *   region zero (see the conventions above), the rest clobbered.
 * -0.0 scores rank equal to +0.0; NaN or infinite inputs are a precondition
 * violation. */
prhs_status prhs_select(const prhs_kv* kv, const void* q, const prhs_params* params,
                        int32_t* topk_idx, int32_t* topk_len, int32_t k_cap,
                        int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                        void* ws, size_t ws_bytes, void* stream);

/* Refresh that also caches the dilated shared set (Sec. 4.4: the critical
 * sets of shared heads are known ahead and can be prepared; Eq. neighboring).
 *
 * Same as prhs_select, and in the same launch also writes, for every (b, g),
 *   shared_idx[b][g][0 .. shared_len) = the set prhs_dilate_reuse returns
 *   for these params with anchor_lens = seq_lens = n0,
 * i.e. [0, min(sink, n0)) U S* U {p + j : p in the top m, |j| <= r} U
 * [n0 - window, n0) clipped to [0, n0), ascending and without duplicates.
 * With prhs_reuse_decode_attn it serves every later step of the block and
 * every other layer of the group, so no separate dilation call is needed.
 * shared_idx: [batch][num_kv_heads][set_cap] int32, shared_len:
 * [batch][num_kv_heads] int32.  set_cap (for both sets) must be at least
 * prhs_set_capacity(params, max_seq_len). */
prhs_status prhs_select_shared(const prhs_kv* kv, const void* q, const prhs_params* params,
                               int32_t* topk_idx, int32_t* topk_len, int32_t k_cap,
                               int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                               int32_t* shared_idx, int32_t* shared_len, void* ws,
                               size_t ws_bytes, void* stream);

/* Reuse: build the dilated shared set of a later step or another layer of the
 * group (Def. 3.2 key-value sharing, Sec. 2.2; Eq. neighboring).
 *
 * For every (b, g), with n0 = anchor_lens[b] (the anchor's length at its
 * refresh), n = seq_lens[b] >= n0, S* = topk_idx[b][g][0 .. topk_len) as
 * returned by prhs_select with the same params, whose first
 * m = min(dilate_m or floor(k_b / 3), topk_len) entries are the top m:
 *   set = [0, min(sink, n0)) U S* U {p + j : p in first m of S*, |j| <= r,
 *         0 <= p + j < n} U [max(min(sink, n0), n0 - window), n),
 * ascending and without duplicates.  The set does not depend on any layer's
 * K/V, so one call serves every layer that shares the selection.
 * Writes at most set_cap entries; set_len is clamped to set_cap. */
prhs_status prhs_dilate_reuse(const prhs_params* params, int32_t batch, int32_t num_kv_heads,
                              const int32_t* topk_idx, const int32_t* topk_len, int32_t k_cap,
                              const int32_t* anchor_lens, const int32_t* seq_lens,
                              int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                              void* stream);

/* Token-sparse decode attention (Def. 3.1, Sec. 2.2) over per-kv-head index sets.
 *
 * For every (b, query head h) with g = h / (Hq/Hkv) and
 * S = set_idx[b][g][0 .. min(set_len[b][g], set_cap)):
 *   out[b][h] = sum_{i in S} softmax_S(scale * q[b][h] . k_i) v_i   (fp32)
 *   lse[b][h] = log sum_{i in S} exp(scale * q[b][h] . k_i)        (fp32)
 * i.e. attention renormalised over S (the truncated distribution of the
 * unified-bounds appendix).  An empty S gives out = 0, lse = -inf.  Indices
 * outside [0, seq_lens[b]) are skipped.  lse may be NULL.
 * q: [batch][num_q_heads][head_dim] in kv->dtype.  out: [batch][num_q_heads]
 * [head_dim] fp32.  ws: >= prhs_workspace_size(PRHS_OP_SPARSE_ATTN, set_cap)
 * bytes; its contents need no initialisation and are clobbered. */
prhs_status prhs_sparse_decode_attn(const prhs_kv* kv, const void* q,
                                    const int32_t* set_idx, const int32_t* set_len,
                                    int32_t set_cap, float scale, float* out, float* lse,
                                    void* ws, size_t ws_bytes, void* stream);

/* prhs_sparse_decode_attn without a workspace argument, for callers that
 * cannot allocate device memory (code under stream capture, tight serving
 * loops, hosts that forbid allocation).  Same arguments, semantics and
 * outputs as prhs_sparse_decode_attn, computed by the same kernels; the
 * split-K partials live in a static array of 16 MiB that every device the
 * library runs on holds until the process ends.  No call allocates or frees
 * memory.  Calls whose partials would exceed the array
 * (prhs_workspace_size(PRHS_OP_SPARSE_ATTN) > 16 MiB) return
 * PRHS_E_UNSUPPORTED.  Every call on one device uses that device's single
 * array: calls that overlap on one device (other streams, other host
 * threads) race and must be ordered by the caller. */
prhs_status prhs_sparse_decode_attn_static(const prhs_kv* kv, const void* q,
                                           const int32_t* set_idx, const int32_t* set_len,
                                           int32_t set_cap, float scale, float* out, float* lse,
                                           void* stream);

/* Token-sparse decode attention over a reused set (Def. 3.2 key-value sharing,
 * Sec. 2.2; Eq. neighboring): the shared set of a later decode step without
 * rebuilding it.
 *
 * For n >= n0 the dilated shared set at length n is the one at the anchor
 * length n0 followed by the positions decoded since, [n0, n): neighbours of
 * the middle range never pass n0 - window + 1, and every position in [n0, n)
 * lies in the recency window.  So one prhs_dilate_reuse call at
 * seq_lens = anchor_lens serves every step of the block, and this call
 * attends, for every (b, query head h) with g = h / (Hq/Hkv),
 *   S = {i in set_idx[b][g][0 .. min(set_len[b][g], set_cap)) : i < n0}
 *       U [n0, seq_lens[b]),   n0 = clamp(anchor_lens[b], 0, seq_lens[b]),
 * with the same outputs as prhs_sparse_decode_attn over S.
 * anchor_lens: [batch] int32 device array.  Precondition:
 * set_len[b][g] + seq_lens[b] - n0 <= set_cap (prhs_set_capacity with this
 * refresh period guarantees it); rows beyond set_cap are not attended.
 * ws: >= prhs_workspace_size(PRHS_OP_SPARSE_ATTN, set_cap) bytes. */
prhs_status prhs_reuse_decode_attn(const prhs_kv* kv, const void* q,
                                   const int32_t* set_idx, const int32_t* set_len,
                                   int32_t set_cap, const int32_t* anchor_lens, float scale,
                                   float* out, float* lse, void* ws, size_t ws_bytes,
                                   void* stream);

/* Causal prefill attention of the prompts under the progressive sliding
 * attention window (Sec. 4.2, Eq. psaw: the window narrows during prefill as
 * well as decoding).  For every (b, query head h) with g = h / (Hq/Hkv) and
 * every query position i < min(seq_lens[b], q_len), the query at position i
 * attends the keys of kv head g
 *   S_i = {p <= i : p < sink  or  p >= first_visible(i + 1)}
 * where the query at position i has the t = i + 1 tokens [0, i] in view and
 * first_visible(t) is that of prhs_psaw (the same set a decode step at
 * length i + 1 attends).  With psaw NULL, S_i = [0, i]: plain causal
 * attention (Eq. attn_eq per position).  y_i = sum_{p in S_i} softmax(scale *
 * q_i . k_p) v_p and lse_i as in prhs_sparse_decode_attn.  Query rows at
 * positions >= seq_lens[b] (and < q_len) give y = 0 and lse = -inf.
 * kv:        bf16 cache (contiguous or paged) holding the prompt of
 *            sequence b at positions [0, seq_lens[b]) (fp32 inputs give
 *            PRHS_E_UNSUPPORTED).
 * q:         [batch][num_q_heads][q_len][head_dim] bf16 device array; row i is
 *            the query at position i.
 * psaw:      host descriptor of the layer's window, or NULL (causal).
 * scale:     softmax scale, positive and finite (PRHS_E_INVALID otherwise).
 * out:       [batch][num_q_heads][q_len][head_dim] fp32; lse:
 *            [batch][num_q_heads][q_len] fp32 or NULL.
 * No workspace.  Caller owns every buffer; ceil(q_len / 64) * batch * num_q_heads
 * must be below 2^31 (PRHS_E_UNSUPPORTED otherwise). */
prhs_status prhs_prefill_attn(const prhs_kv* kv, const void* q, int32_t q_len,
                              const prhs_psaw* psaw, float scale, float* out, float* lse,
                              void* stream);

/* Dense decode attention over every cached key [0, seq_lens[b]) (Eq. attn_eq):
 * the baseline the sparse path is measured against, and the k = n special
 * case.  Same outputs and conventions as prhs_sparse_decode_attn.
 * ws: >= prhs_workspace_size(PRHS_OP_DENSE_ATTN) bytes (no initialisation
 * needed). */
prhs_status prhs_dense_decode_attn(const prhs_kv* kv, const void* q, float scale,
                                   float* out, float* lse, void* ws, size_t ws_bytes,
                                   void* stream);

/* ---- Similarity-gated sharing (Sec. 4.1, Similarity Criteria; Eq. cos_sim) ----
 *
 * Instead of a fixed refresh every refresh_every steps, a later step of a
 * block of num_slots steps shares the selection of an earlier step of the
 * block only when their queries are similar.  Per anchor layer of a layer
 * group the caller keeps, for the block's steps 0 .. num_slots-1 ("slots"):
 * the reference queries ref_q [num_slots][B][Hq][d] (dtype of q), the flags
 * ref_valid [num_slots][B*Hkv] (unit retrieved at that slot), the lengths
 * slot_lens [num_slots][B], and a set pool [2][num_slots][B*Hkv][set_cap] of
 * int32 with lengths [2][num_slots][B*Hkv]: kind 0 holds each retrieving
 * step's critical set, kind 1 its dilated shared set.  prhs_gate is called
 * at every step of the block in order, then prhs_select_gated on the
 * retrieving units (writing kind 0 and 1 of the current slot), then one
 * prhs_pool_decode_attn per layer of the group. */

/* Gate for block step `slot` (0 <= slot < num_slots), one decision per
 * (b, kv head g).  Slot 0 always retrieves.  Otherwise the unit shares the
 * most recent earlier slot j with ref_valid[j][u] != 0 for which every query
 * head h of the group satisfies sim(q[b][h], ref_q[j][b][h]) > tau, where
 * sim is the cosine similarity; it is decided exactly as
 *   dot > 0 and dot * dot > ((tau * tau) * |q|^2) * |q_j|^2
 * in binary64 from fp32 sums, which is exact when the inputs are on a grid
 * coarse enough for the fp32 sums to be exact.  0 <= tau <= 1.
 * Writes: choice[u] = j, or -1 when the unit retrieves now;
 *   with record != 0 also the step's record: ref_q[slot] = q;
 *   ref_valid[slot][u] = (choice[u] < 0); slot_lens[slot][b] = seq_lens[b]
 *   (record = 0 takes the same decisions and writes only the four outputs
 *   below, e.g. into separate arrays for a branch that runs beside the
 *   recording one);
 *   row_anchor[u] = pool row the group's anchor layer attends: the current
 *     slot's critical set when retrieving, else slot j's shared set;
 *   row_other[u] = pool row the group's other layers attend: the shared set
 *     of the current slot or of slot j;
 *   tail[u] = first position of the decoded tail to append: seq_lens[b]
 *     (none) when retrieving, else slot_lens[j][b].
 * Pool rows are numbered (kind * num_slots + slot) * (B*Hkv) + u. */
prhs_status prhs_gate(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                      int32_t dtype, const void* q, const int32_t* seq_lens, double tau,
                      int32_t num_slots, int32_t slot, void* ref_q, int32_t* ref_valid,
                      int32_t* slot_lens, int32_t* choice, int32_t* row_anchor,
                      int32_t* row_other, int32_t* tail, int32_t record, void* stream);

/* The gate and the refresh of the retrieving units in one call (Sec. 4.1,
 * Similarity Criteria; Sec. 4.4: only retrieval heads score): exactly
 * prhs_gate with record = 1 followed by prhs_select_gated on its choice, the
 * gate's arrays as in prhs_gate and the selection's as in
 * prhs_select_gated (set_idx / shared_idx: the current slot's pool rows of
 * kind 0 and 1).  q and seq_lens come from kv and the query argument.  When
 * the refresh runs as one fused launch (contiguous bf16 cache, middle range
 * within one CU's LDS, rows filling more than half the CUs) the gate is
 * taken inside that launch, one wave per row before it scores; otherwise
 * the gate kernel runs first.  The decided units' outputs of this step
 * (choice, row_anchor, row_other, tail) are written before any of them is
 * needed by a later launch on the stream. */
prhs_status prhs_gate_select(const prhs_kv* kv, const void* q, const prhs_params* params,
                             double tau, int32_t num_slots, int32_t slot, void* ref_q,
                             int32_t* ref_valid, int32_t* slot_lens, int32_t* choice,
                             int32_t* row_anchor, int32_t* row_other, int32_t* tail,
                             int32_t* topk_idx, int32_t* topk_len, int32_t k_cap,
                             int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                             int32_t* shared_idx, int32_t* shared_len, void* ws, size_t ws_bytes,
                             void* stream);

/* prhs_select_shared for the units the gate sends to retrieval only:
 * (b, g) with choice[b][g] >= 0 are left untouched, the others get their
 * top-k, critical set and dilated shared set exactly as prhs_select_shared
 * computes them.  Pass the current slot's rows of the pool as set_idx
 * (kind 0) and shared_idx (kind 1). */
prhs_status prhs_select_gated(const prhs_kv* kv, const void* q, const prhs_params* params,
                              const int32_t* choice, int32_t* topk_idx, int32_t* topk_len,
                              int32_t k_cap, int32_t* set_idx, int32_t* set_len, int32_t set_cap,
                              int32_t* shared_idx, int32_t* shared_len, void* ws,
                              size_t ws_bytes, void* stream);

/* Token-sparse decode attention where every (b, kv head g) attends its own
 * row of a set pool plus a decoded tail (Def. 3.1 and 3.2, Sec. 2.2),
 * optionally under the progressive sliding attention window (Sec. 4.2,
 * Eq. psaw; CIS + PSAW is the paper's CPE): with r = unit_row[u],
 * n = seq_lens[b] and t0 = clamp(unit_tail[u], 0, n),
 *   S = {i in pool_idx[r][0 .. min(pool_len[r], set_cap)) : i < t0} U [t0, n),
 * minus, when psaw is given, the positions in [psaw->sink, first_visible(n))
 * (the layer's masked range at length n, prhs_psaw), and the outputs of
 * prhs_sparse_decode_attn over S.  A row outside [0, pool_rows) gives an
 * empty set.  pool_idx: [pool_rows][set_cap] int32; unit_row, unit_tail:
 * [B*Hkv] int32 (prhs_gate's row_anchor or row_other, and tail; or the
 * identity rows and per-unit anchor lengths of the fixed schedule's sets);
 * psaw: host descriptor or NULL.  Precondition: pool_len[r] + n - t0 <=
 * set_cap.  ws: >= prhs_workspace_size(PRHS_OP_SPARSE_ATTN, set_cap) bytes.
 * units_side selects the units by the gate's decision: PRHS_UNITS_ALL every
 * unit (unit_gate may be NULL); PRHS_UNITS_RETRIEVING only units with
 * unit_gate[u] < 0; PRHS_UNITS_SHARING only units with unit_gate[u] >= 0
 * (unit_gate: prhs_gate's choice, [B*Hkv]).  The other units' outputs are
 * left untouched, so the retrieving and the sharing units of a layer can be
 * attended by two launches that run concurrently (Sec. 4.4: shared heads do
 * not wait for retrieval) with separate workspaces. */
prhs_status prhs_pool_decode_attn(const prhs_kv* kv, const void* q, const int32_t* pool_idx,
                                  const int32_t* pool_len, int32_t pool_rows, int32_t set_cap,
                                  const int32_t* unit_row, const int32_t* unit_tail,
                                  const int32_t* unit_gate, int32_t units_side,
                                  const prhs_psaw* psaw, float scale, float* out, float* lse,
                                  void* ws, size_t ws_bytes, void* stream);

/* Message for the last non-OK status returned on the calling thread. */
const char* prhs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PRHS_H_ */

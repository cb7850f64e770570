// Internal declarations shared by the libprhs translation units.
// Device-side views of the C-ABI descriptors, KV row addressing, and the
// host-side launch functions each kernel file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace prhs {

// Positions are < 2^22, so a position fits the low half of a 64-bit sort key.
constexpr int kIdxBits = 22;
constexpr uint32_t kIdxMax = (1u << kIdxBits) - 1u;
constexpr int kHistBins = 2048;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Loads of K and V rows, which a launch reads once, with the non-temporal
// (streaming) cache policy: on this chip a streaming read sustains about
// 7 TB/s with it and about 6 TB/s with the default policy.  Only for loads
// that read whole 128-byte lines per instruction: a line shared by several
// load instructions is evicted after its first hit and fetched again.
__device__ __forceinline__ u32x4_t stream_load16(const void* p) {
  return __builtin_nontemporal_load((const u32x4_t*)p);
}
__device__ __forceinline__ u32x2_t stream_load8(const void* p) {
  return __builtin_nontemporal_load((const u32x2_t*)p);
}

// Device view of one layer's KV cache.
struct KvView {
  const void* k;
  const void* v;
  const int32_t* table;
  const int32_t* seq_lens;
  int32_t batch, hq, hkv, d;
  int32_t capacity;   // contiguous token stride
  int32_t page_size, max_pages, num_pages;
  int32_t max_seq_len;
  int32_t paged;
};

// Element offset of the row holding token `pos` of (b, kv head g), or -1 when
// the position or its page lies outside the cache.  Contiguous rows are
// [b][g][pos][d]; paged rows are [page][g][slot][d].
__device__ __forceinline__ int64_t kv_row_offset(const KvView& kv, int b, int g, int pos) {
  if (pos < 0) return -1;
  if (!kv.paged) {
    if (pos >= kv.capacity) return -1;
    return ((int64_t)(b * kv.hkv + g) * kv.capacity + pos) * kv.d;
  }
  int page = pos / kv.page_size;
  if (page >= kv.max_pages) return -1;
  int phys = kv.table[(int64_t)b * kv.max_pages + page];
  if (phys < 0 || phys >= kv.num_pages) return -1;
  return (((int64_t)phys * kv.hkv + g) * kv.page_size + (pos - page * kv.page_size)) * kv.d;
}

// Number of valid cached tokens of sequence b, clamped to what the cache can hold.
__device__ __forceinline__ int kv_seq_len(const KvView& kv, int b) {
  int n = kv.seq_lens[b];
  n = n < 0 ? 0 : n;
  return n > kv.max_seq_len ? kv.max_seq_len : n;
}

// First visible non-sink position when n tokens are in view under the
// progressive sliding attention window (Eq. psaw): P = floor(f n) with the
// layer's factor f = 1 - phi^e (computed once on the host, binary64), and
// the visible keys are [0, min(sink, n)) U [max(min(sink, n), P - 1), n).
// f lies in [0, 1) and n < 2^22, so P fits an int.
__host__ __device__ __forceinline__ int psaw_first_visible(double f, int sink, int n) {
  const int P = (int)floor(f * (double)n);
  const int se = sink < n ? sink : n;
  return se > P - 1 ? se : P - 1;
}

// Length rank of workgroup w of a grid of U workgroups placed on C CUs, when
// the workgroups w = c, c + C, c + 2C, ... run side by side on CU c (the
// order in which this chip fills its CUs when they all fit at once): rounds
// of C ranks, every other round reversed, so that the units of one CU pair
// long with short.  A permutation of [0, U).
__host__ __device__ __forceinline__ int serpentine_rank(int w, int C, int U) {
  const int k = w / C, c = w - k * C;
  const int p = min(C, U - k * C);  // workgroups in this round
  return k * C + ((k & 1) ? p - 1 - c : c);
}

// Unit b * heads + h of length rank t (0 = longest): sequences ordered by
// decreasing cached length, ties by index; the heads of a sequence share its
// length and take consecutive ranks.  s_len holds kv.batch ints of LDS,
// s_out one.  Every thread of the workgroup must call it.
__device__ __forceinline__ int unit_of_length_rank(const KvView& kv, int heads, int t, int* s_len,
                                                   int* s_out) {
  const int B = kv.batch, tb = t / heads;
  for (int b = threadIdx.x; b < B; b += blockDim.x) s_len[b] = kv_seq_len(kv, b);
  __syncthreads();
  for (int b = threadIdx.x; b < B; b += blockDim.x) {
    const int nb = s_len[b];
    int r = 0;
    for (int b2 = 0; b2 < B; ++b2) {
      const int n2 = s_len[b2];
      r += (n2 > nb || (n2 == nb && b2 < b)) ? 1 : 0;
    }
    if (r == tb) *s_out = b * heads + (t - tb * heads);
  }
  __syncthreads();
  return *s_out;
}

// Order-preserving map of an fp32 score to uint32 (larger score -> larger key).
// -0.0 is mapped like +0.0.
__device__ __forceinline__ uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Workgroup barrier that orders LDS accesses only: it waits for this wave's
// LDS operations, not for its outstanding global stores, so a workgroup that
// has written results to global memory (which it never reads back) does not
// stall on their acknowledgement at every later barrier.  Global memory
// exchanged between the workgroup's threads needs __syncthreads() (or
// block_publish) instead.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP lane moves:
// shifts by 1, 2, 4, 8 inside each row of 16 lanes (a lane without a source
// adds 0), then lane 15 of each row into the next row (rows 1, 3) and lane
// 31 into rows 2 and 3.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// 64-bit values here are always packed narrow counters whose sums stay
// inside their fields, so the two 32-bit halves scan independently.
__device__ __forceinline__ uint64_t wave_inclusive_scan(uint64_t x) {
  const uint32_t lo = wave_inclusive_scan((uint32_t)x);
  const uint32_t hi = wave_inclusive_scan((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Exclusive prefix sum over a workgroup of BLOCK threads; `scratch` holds
// BLOCK/64 + 1 elements of LDS (exchanged through LDS only: the barriers do
// not order global memory).  Returns this thread's exclusive prefix and
// the block total in *total.  Must be reached by every thread.  With T =
// uint64_t, several narrow counters packed into one word scan together as
// long as no field overflows (and none straddles bit 32).
template <int BLOCK, typename T = uint32_t, bool REUSE_BARRIER = true>
__device__ __forceinline__ T block_exclusive_scan(T v, T* scratch, T* total) {
  constexpr int W = BLOCK / 64;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const T x = wave_inclusive_scan(v);
  if (lane == 63) scratch[wave] = x;
  lds_barrier();
  // every thread adds up the wave totals itself (broadcast LDS reads)
  T before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    const T s = scratch[w];
    before += w < wave ? s : (T)0;
    tot += s;
  }
  *total = tot;
  // scratch may be written again after return (without REUSE_BARRIER the
  // caller reaches a barrier before it writes scratch again)
  if (REUSE_BARRIER) lds_barrier();
  return before + x - v;
}

// ---------------------------------------------------------------------------
// Host launch functions (defined next to their kernels).

struct GateLaunch;

struct SelectLaunch {
  KvView kv;
  const void* q;
  int dtype;
  int k, k_num, k_den, sink, window, dilate_m;
  int32_t* topk_idx;
  int32_t* topk_len;
  int k_cap;
  int32_t* set_idx;
  int32_t* set_len;
  int set_cap;
  int dilate_r;
  int32_t* shared_idx;  // optional: dilated shared set at the anchor length
  int32_t* shared_len;
  const int32_t* row_choice;  // optional [rows]: only rows with a negative entry are selected
  const GateLaunch* gate;     // optional: take the similarity gate first, select the retrieving rows
  void* ws;
  int max_topk;   // host bound on the clamped budget (sort size)
};
size_t select_workspace_bytes(int rows, int max_seq_len, int max_topk);
hipError_t launch_select(const SelectLaunch& a, hipStream_t stream);

struct DilateLaunch {
  int batch, hkv;
  const int32_t* topk_idx;
  const int32_t* topk_len;
  int k_cap;
  const int32_t* anchor_lens;
  const int32_t* seq_lens;
  int32_t* set_idx;
  int32_t* set_len;
  int set_cap;
  int k, k_num, k_den, sink, window, dilate_m, dilate_r;
};
hipError_t launch_dilate_reuse(const DilateLaunch& a, hipStream_t stream);

struct AttnLaunch {
  KvView kv;
  const void* q;
  int dtype;
  const int32_t* set_idx;  // null for dense
  const int32_t* set_len;
  const int32_t* tail_start;  // [B] or null (reuse attention: set U [tail_start, n))
  const int32_t* unit_row;    // [B*Hkv] or null: pool row each unit attends
  const int32_t* unit_tail;   // [B*Hkv] with unit_row: first position of the unit's tail
  int pool_rows;              // rows of set_idx when unit_row is given
  const int32_t* unit_gate;   // [B*Hkv] or null: the gate's choice per unit, for units_side
  int units_side;             // 0 all units; 1 only units with unit_gate < 0; 2 only >= 0
  int psaw;                   // nonzero: positions in [psaw_sink, first visible) are masked
  double psaw_f;              // the layer's factor 1 - phi^e of Eq. psaw
  int psaw_sink;
  int set_cap;
  float scale;
  float* out;
  float* lse;
  void* ws;
};
// Split geometry shared by workspace sizing and launch.
void attn_split_geometry(int dtype, bool dense, int batch, int hq, int hkv, int rows_cap,
                         int* chunk, int* nsplit);
size_t attn_workspace_bytes(int dtype, bool dense, int batch, int hq, int hkv, int d,
                            int rows_cap);
hipError_t launch_attention(const AttnLaunch& a, bool dense, hipStream_t stream);
// Device address and size of this device's static scratch array for the
// split-K partials of the no-allocation attention entry point (looked up
// once per device with hipGetSymbolAddress; the array is never named on the
// host otherwise).
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
hipError_t attn_static_scratch(void** ptr);

struct GateLaunch {
  int batch, hq, hkv, d, dtype;
  const void* q;
  const int32_t* seq_lens;
  double tau;
  int num_slots, slot;
  void* ref_q;          // [num_slots][B][Hq][d]
  int32_t* ref_valid;   // [num_slots][B*Hkv]
  int32_t* slot_lens;   // [num_slots][B]
  int32_t* choice;      // [B*Hkv]
  int32_t* row_anchor;  // [B*Hkv]
  int32_t* row_other;   // [B*Hkv]
  int32_t* tail;        // [B*Hkv]
  int record;           // nonzero: also record the step (ref_q, ref_valid, slot_lens)
};
hipError_t launch_gate(const GateLaunch& a, hipStream_t stream);

struct PrefillLaunch {
  KvView kv;                  // bf16 cache (contiguous or paged) holding the prompts
  const void* q;              // [B][Hq][T][d]
  int T;
  int psaw;                   // nonzero: the query at position i attends [0, sink) and
  double psaw_f;              // [first visible at i + 1, i] (Eq. psaw factor psaw_f)
  int sink;
  float scale;
  float* out;                 // [B][Hq][T][d]
  float* lse;                 // [B][Hq][T] or null
};
hipError_t launch_prefill(const PrefillLaunch& a, hipStream_t stream);

// Compute units of the current device (cached per device; 0 if unknown).
int device_cus();

}  // namespace prhs

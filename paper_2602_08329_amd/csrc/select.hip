// Refresh-step selection for one layer: ranking scores over the middle range,
// the exact top-k under the order (score desc, position asc), and the
// critical set sink U top-k U window (Sec. 4.1 Selection Criteria; top-k
// oracle of Sec. 2.3); optionally also the dilated shared set at the anchor
// length (Eq. neighboring), and optionally only for the rows a similarity
// gate sends to retrieval.
//
// Three paths, all on the caller's stream (select_path picks one):
//   select_fused   middle range within LDS, contiguous bf16, rows filling
//                  more than half the CUs: one workgroup per row scores into
//                  LDS, takes exact thresholds for k and m over the 32-bit
//                  keys and compacts in position order (which settles ties)
//                  -- one launch;
//   keyed path     middle range within LDS, fewer rows (or a paged or fp32
//                  cache): score_* without histograms spreads each row over
//                  many workgroups and writes its keys, then select_keyed
//                  runs select_fused's selection half, one workgroup per row
//                  -- two launches;
//   radix path     longer middle ranges, one launch each:
//     score_*        sigma_i = max_h q_h . k_i (raw, fp32) -> order-preserving
//                    u32 key; fused histogram of the top 11 key bits
//     select_filter  locate the threshold bin of level 0; keys above it are
//                    selected, keys in it become candidates (with the level-1
//                    histogram fused)
//     select_finish  the remaining radix levels over the candidates as 64-bit
//                    composites (key, kIdxMax - pos), distinct, so ties go to
//                    the lower position; one segmented bitmap pass writes the
//                    ordered outputs.
//                  The per-row histograms and counters the score and filter
//                  kernels accumulate into sit at the front of the workspace;
//                  they are zero when a call starts (the caller zero-fills a
//                  new workspace) and select_finish zeroes each row's again
//                  once it has read them, so no clearing launch is needed.
#include <stdlib.h>

#include "prhs.h"
#include "gate.h"
#include "prhs_internal.h"
#include "setops.h"

namespace prhs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kScoreBlock = 256;
constexpr int kScoreChunk = 1024;   // keys per score workgroup
constexpr int kScoreSub = 2;        // 16-key sub-tiles per wave step of score_bf16
constexpr int kFilterBlock = 256;
constexpr int kFilterPerThread = 16;
constexpr int kFilterChunk = kFilterBlock * kFilterPerThread;
constexpr int kFinishBlock = 1024;
constexpr int kFinishPerThread = 8;  // candidates per thread per pass
constexpr int kFinishTies = 4096;    // level-1 ties the finish kernel keeps in LDS
// positions per bitmap segment of the finish kernel (3 bitmaps of 8 KB): whole
// groups of four words, and below 2^16 so that per-segment counts fit 16-bit
// fields
constexpr int kFinishSegBits = 65408;
// output staging of the finish kernel: a bitmap segment's outputs up to this
// many entries (or what LDS has room for) are gathered in LDS and copied out
// with whole-wave stores
constexpr int kFinishStage = 8192;
// candidates few enough for one wave to rank them directly
constexpr int kSmallRank = 64;
// winners per thread of the finish kernel loaded with its histograms
constexpr int kSelPrefetch = 2;

struct SelArgs {
  KvView kv;
  const void* q;
  int k, k_num, k_den, sink, window, dilate_m;
  int mcap, selcap;
  int sortcap;         // LDS sort buffer entries of select_finish (>= selcap)
  int stagecap;        // LDS output staging entries of select_finish
  int woff;            // select_finish has LDS for per-word output offsets
  int seg_bits;        // select_finish: positions per bitmap segment (a multiple of 32)
  int seg_shift;       // select_finish: one segment, the dilation by shifts of the top-m bitmap
  uint32_t* keys;      // [rows][mcap]
  uint32_t* hist0;     // [rows][2048]
  uint32_t* hist1;     // [rows][2048]
  uint32_t* counters;  // [rows][4]: 0 selected, 1 candidates
  uint2* sel;          // [rows][selcap] (key, position)
  uint2* cand;         // [rows][mcap]
  uint2* cand2;        // [rows][mcap]
  int32_t* topk_idx;
  int32_t* topk_len;
  int k_cap;
  int32_t* set_idx;
  int32_t* set_len;
  int set_cap;
  int dilate_r;
  int32_t* shared_idx;  // optional [rows][set_cap]: the dilated shared set at n0
  int32_t* shared_len;
  int balance_cus;      // fused refresh: > 0 = CU count to balance rows over, 0 = off
  int balance_serpentine;  // with balance_cus: workgroups share CUs side by side
  const int32_t* row_choice;  // optional [rows]: rows with an entry >= 0 are left untouched
  int gate_fused;       // fused refresh: wave 0 takes the similarity gate of its row first
  GateLaunch gate;      // (with gate_fused) and the workgroup selects only a retrieving row
};

// Rows the similarity gate lets share are not selected again.
__device__ __forceinline__ bool row_skipped(const SelArgs& a, int row) {
  return a.row_choice != nullptr && a.row_choice[row] >= 0;
}

struct RowGeom {
  int n0, sink_end, win_start, m, kb;
};

__device__ __forceinline__ RowGeom row_geom(const SelArgs& a, int b) {
  RowGeom r;
  r.n0 = kv_seq_len(a.kv, b);
  r.sink_end = min(a.sink, r.n0);
  r.win_start = max(r.sink_end, r.n0 - a.window);
  r.m = r.win_start - r.sink_end;
  long long kb = a.k_den > 0 ? ((long long)a.k_num * r.n0) / a.k_den : (long long)a.k;
  if (kb < 0) kb = 0;
  if (kb > r.m) kb = r.m;
  r.kb = (int)kb;
  return r;
}

// Radix digits of the 64-bit composite (score key, kIdxMax - position), most
// significant first: 11 + 11 + 10 bits of the score key, then 11 + 11 bits
// of the reversed position (positions are < 2^22).
__device__ __forceinline__ uint32_t level_digit(uint2 e, int level) {
  const uint32_t rp = kIdxMax - e.y;
  switch (level) {
    case 0: return e.x >> 21;
    case 1: return (e.x >> 10) & 0x7FFu;
    case 2: return e.x & 0x3FFu;
    case 3: return (rp >> 11) & 0x7FFu;
    default: return rp & 0x7FFu;
  }
}

// 54-bit composite of a (score key, position) pair: larger score first,
// lower position first among equal scores; every value is distinct.
__device__ __forceinline__ uint64_t composite(uint2 e) {
  return ((uint64_t)e.x << kIdxBits) | (uint64_t)(kIdxMax - e.y);
}

__device__ __forceinline__ int composite_pos(uint64_t c) {
  return (int)(kIdxMax - (uint32_t)(c & kIdxMax));
}

// Finds the bin holding the kk-th largest element of histogram h (LDS,
// kHistBins bins).  Writes bin, remaining rank inside the bin and the bin's
// count to LDS outputs.  Requires 1 <= kk <= sum(h).  All threads must call.
template <int BLOCK>
__device__ void find_threshold(const uint32_t* h, uint32_t kk, uint32_t* scan, int* s_bin,
                               uint32_t* s_krem, uint32_t* s_cnt) {
  constexpr int BPT = kHistBins / BLOCK;
  const int t = threadIdx.x;
  uint32_t local = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) local += h[kHistBins - 1 - (t * BPT + i)];
  uint32_t total;
  uint32_t cum = block_exclusive_scan<BLOCK>(local, scan, &total);
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int bin = kHistBins - 1 - (t * BPT + i);
    const uint32_t c = h[bin];
    if (cum < kk && cum + c >= kk) {
      *s_bin = bin;
      *s_krem = kk - cum;
      *s_cnt = c;
    }
    cum += c;
  }
  lds_barrier();
}

// Adds an LDS histogram (8-byte aligned) into a global one, two bins per
// 64-bit atomic (a bin's count stays below 2^32, so no carry crosses into
// its neighbour), skipping empty pairs.
__device__ __forceinline__ void flush_hist(const uint32_t* h, uint32_t* dst) {
  for (int i = threadIdx.x; i < kHistBins / 2; i += blockDim.x) {
    const uint2 c = ((const uint2*)h)[i];
    if (c.x | c.y)
      atomicAdd((unsigned long long*)dst + i, (unsigned long long)c.x | ((unsigned long long)c.y << 32));
  }
}

// A DPP lane move of a float inside each row of 16 lanes (every lane has a
// source for the moves used here).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xF,
                                                    0xF, false));
}

// bf16 scoring on MFMA: per 16 keys, S[key][head] = K_tile(16 x d) . Q^T(d x 16)
// with the group's g <= 16 query heads in the columns (unused columns zero).
// Keys are loaded whole, d/8 lanes of 16 bytes per key (the operand order,
// 4 lanes per key, would read 64-byte pieces of 16 keys per load, which this
// chip serves at well under half the rate), with the streaming cache policy,
// and reach operand order through a per-wave LDS tile of 16 keys: lane l
// takes dims 32kk + 8(l/16) .. +7 of key l%16 for product kk, the same
// permutation of d as the query operand.  Products of bf16 values are exact
// in fp32 and the accumulation is fp32.  Each wave handles 16 SUB keys per
// step and prefetches its next step's loads while multiplying the current
// one.
template <int D, int SUB = 4>
struct ScoreStep {
  static constexpr int kSub = SUB;  // 16-key sub-tiles per step
  u32x4_t kraw[SUB][D / 32];        // sub-tile s, load j: key 16s + j (64 / (d/8)) + l / (d/8)
};

// Slot of 16-byte chunk c of key r (< 16) in a wave's LDS tile, XOR-swizzled
// so that the whole-key writes and the operand-order reads hit distinct banks.
template <int D>
__device__ __forceinline__ int score_slot(int r, int c) {
  constexpr int CH = D / 8;
  return r * CH + (c ^ (r & (CH - 1)));
}

template <int D, bool PAGED>
__device__ __forceinline__ int32_t score_row(const SelArgs& a, const RowGeom& rg, int b, int g,
                                             int i, int end, int p0, const int32_t* s_page) {
  if (i >= end) return -1;
  const int pos = rg.sink_end + i;
  if (!PAGED) return (b * a.kv.hkv + g) * a.kv.capacity + pos;
  const int phys = s_page[pos / a.kv.page_size - p0];
  if (phys < 0) return -1;
  return (phys * a.kv.hkv + g) * a.kv.page_size + pos % a.kv.page_size;
}

template <int D, bool PAGED, int SUB>
__device__ __forceinline__ void score_load(ScoreStep<D, SUB>& S, const SelArgs& a, const RowGeom& rg,
                                           int b, int g, int t, int end, int p0,
                                           const int32_t* s_page, int lane) {
  constexpr int CH = D / 8, RPI = 64 / CH;  // chunks per key, keys per load
  const __bf16* kbase = (const __bf16*)a.kv.k;
  const int kc = lane % CH, kr = lane / CH;
#pragma unroll
  for (int s = 0; s < SUB; ++s)
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
      const int32_t row =
          score_row<D, PAGED>(a, rg, b, g, t + s * 16 + j * RPI + kr, end, p0, s_page);
      S.kraw[s][j] = stream_load16(kbase + (int64_t)(row < 0 ? 0 : row) * D + kc * 8);
    }
}

// kst: the wave's LDS tile of 16 x d bf16.  LDS operations of one wave
// complete in order; the wave barriers keep the compiler from moving them
// across each other.
template <int D, int SUB, bool HIST = true>
__device__ __forceinline__ void score_consume(const ScoreStep<D, SUB>& S, const bf16x8_t* qf, int G,
                                              int gp, int t, int end, int lane, uint32_t* keys,
                                              uint32_t* hist, u32x4_t* kst) {
  constexpr int CH = D / 8, RPI = 64 / CH;
  const int col = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int s = 0; s < SUB; ++s) {
#pragma unroll
    for (int j = 0; j < D / 32; ++j) kst[score_slot<D>(j * RPI + lane / CH, lane % CH)] = S.kraw[s][j];
    __builtin_amdgcn_wave_barrier();
    bf16x8_t kf[D / 32];
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk)
      kf[kk] = __builtin_bit_cast(bf16x8_t, kst[score_slot<D>(col, 4 * kk + grp)]);
    __builtin_amdgcn_wave_barrier();
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kk], qf[kk], acc, 0, 0, 0);
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = col < G ? acc[e] : -INFINITY;
    // maximum over the group's gp columns (aligned lane groups inside a row
    // of 16) by DPP lane moves: swaps of neighbours and of pairs in each
    // quad, then the mirrors of each half row and of the row
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (gp > 1) v[e] = fmaxf(v[e], dpp_f32<0xB1>(v[e]));   // quad_perm [1,0,3,2]
      if (gp > 2) v[e] = fmaxf(v[e], dpp_f32<0x4E>(v[e]));   // quad_perm [2,3,0,1]
      if (gp > 4) v[e] = fmaxf(v[e], dpp_f32<0x141>(v[e]));  // row_half_mirror
      if (gp > 8) v[e] = fmaxf(v[e], dpp_f32<0x140>(v[e]));  // row_mirror
    }
    if (col == 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = t + s * 16 + grp * 4 + e;
        if (i < end) {
          const uint32_t key = score_key(v[e]);
          keys[i] = key;
          if (HIST) atomicAdd(&hist[key >> 21], 1u);
        }
      }
    }
  }
}

// HIST: also accumulate the rows' level-0 histograms into hist0 (the radix
// path); without, the keys alone (the keyed path builds its histogram in LDS).
template <int D, bool PAGED, bool HIST>
__global__ __launch_bounds__(kScoreBlock) __attribute__((amdgpu_waves_per_eu(4))) void score_bf16(SelArgs a) {
  constexpr int KS = D / 32;
  __shared__ __attribute__((aligned(8))) uint32_t hist[kHistBins];
  __shared__ int32_t s_page[kScoreChunk + 1];
  __shared__ u32x4_t s_kst[kScoreBlock / 64][16 * (D / 8)];
  const int row = blockIdx.y;
  if (row_skipped(a, row)) return;
  const int b = row / a.kv.hkv, g = row % a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  const int base = blockIdx.x * kScoreChunk;
  if (base >= rg.m || rg.kb <= 0) return;
  const int end = min(rg.m, base + kScoreChunk);
  for (int i = threadIdx.x; i < kHistBins; i += kScoreBlock) hist[i] = 0u;
  int p0 = 0;
  if (PAGED) {
    // the chunk's pages, resolved once
    const int ps = a.kv.page_size;
    p0 = (rg.sink_end + base) / ps;
    const int np = (rg.sink_end + end - 1) / ps - p0 + 1;
    for (int i = threadIdx.x; i < np; i += kScoreBlock) {
      const int page = p0 + i;
      int phys = -1;
      if (page < a.kv.max_pages) phys = a.kv.table[(int64_t)b * a.kv.max_pages + page];
      s_page[i] = (phys >= 0 && phys < a.kv.num_pages) ? phys : -1;
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int G = a.kv.hq / a.kv.hkv;
  const __bf16* q = (const __bf16*)a.q;
  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const int qh = col < G ? col : 0;
    const uint4* qp = (const uint4*)(q + ((size_t)b * a.kv.hq + g * G + qh) * D + grp * 8);
    const uint4 v = qp[4 * kk];
    qf[kk] = __builtin_bit_cast(bf16x8_t, col < G ? v : make_uint4(0, 0, 0, 0));
  }
  int gp = 1;
  while (gp < G) gp <<= 1;
  uint32_t* keys = a.keys + (size_t)row * a.mcap;

  // each wave takes 16 kScoreSub keys per step, the workgroup kStep
  constexpr int kStep = 16 * kScoreSub * (kScoreBlock / 64);
  const int t0 = base + wave * 16 * kScoreSub;
  const int iters = t0 < end ? (end - t0 + kStep - 1) / kStep : 0;
  if (iters > 0) {
    ScoreStep<D, kScoreSub> A, B;
    int t = t0;
    score_load<D, PAGED>(A, a, rg, b, g, t, end, p0, s_page, lane);
    int i = 0;
    for (; i + 2 < iters; i += 2) {
      score_load<D, PAGED>(B, a, rg, b, g, t + kStep, end, p0, s_page, lane);
      score_consume<D, kScoreSub, HIST>(A, qf, G, gp, t, end, lane, keys, hist, s_kst[wave]);
      score_load<D, PAGED>(A, a, rg, b, g, t + 2 * kStep, end, p0, s_page, lane);
      score_consume<D, kScoreSub, HIST>(B, qf, G, gp, t + kStep, end, lane, keys, hist, s_kst[wave]);
      t += 2 * kStep;
    }
    if (i + 1 < iters) {
      score_load<D, PAGED>(B, a, rg, b, g, t + kStep, end, p0, s_page, lane);
      score_consume<D, kScoreSub, HIST>(A, qf, G, gp, t, end, lane, keys, hist, s_kst[wave]);
      score_consume<D, kScoreSub, HIST>(B, qf, G, gp, t + kStep, end, lane, keys, hist, s_kst[wave]);
    } else {
      score_consume<D, kScoreSub, HIST>(A, qf, G, gp, t, end, lane, keys, hist, s_kst[wave]);
    }
  }
  if (HIST) {
    __syncthreads();
    flush_hist(hist, a.hist0 + (size_t)row * kHistBins);
  }
}

// fp32 scoring on the vector ALU: one key per thread, the group's query heads
// staged in LDS, sequential fp32 fused multiply-adds over d.
template <int D, bool HIST>
__global__ __launch_bounds__(kScoreBlock) void score_f32(SelArgs a) {
  __shared__ __attribute__((aligned(8))) uint32_t hist[kHistBins];
  __shared__ float qs[16 * D];
  const int row = blockIdx.y;
  if (row_skipped(a, row)) return;
  const int b = row / a.kv.hkv, g = row % a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  const int base = blockIdx.x * kScoreChunk;
  if (base >= rg.m || rg.kb <= 0) return;
  const int end = min(rg.m, base + kScoreChunk);
  const int G = a.kv.hq / a.kv.hkv;
  const float* q = (const float*)a.q;
  for (int i = threadIdx.x; i < kHistBins; i += kScoreBlock) hist[i] = 0u;
  for (int i = threadIdx.x; i < G * D; i += kScoreBlock)
    qs[i] = q[((size_t)b * a.kv.hq + g * G) * D + i];
  __syncthreads();
  const float* kb = (const float*)a.kv.k;
  uint32_t* keys = a.keys + (size_t)row * a.mcap;
  for (int i = base + threadIdx.x; i < end; i += kScoreBlock) {
    const int64_t off = kv_row_offset(a.kv, b, g, rg.sink_end + i);
    float best = -INFINITY;
    for (int h = 0; h < G; ++h) {
      float acc = 0.f;
      if (off >= 0) {
        const float4* kp = (const float4*)(kb + off);
        for (int j = 0; j < D / 4; ++j) {
          const float4 x = kp[j];
          const float* qh = qs + h * D + 4 * j;
          acc = fmaf(qh[0], x.x, acc);
          acc = fmaf(qh[1], x.y, acc);
          acc = fmaf(qh[2], x.z, acc);
          acc = fmaf(qh[3], x.w, acc);
        }
      }
      best = fmaxf(best, acc);
    }
    const uint32_t key = score_key(best);
    keys[i] = key;
    if (HIST) atomicAdd(&hist[key >> 21], 1u);
  }
  __syncthreads();
  if (HIST) flush_hist(hist, a.hist0 + (size_t)row * kHistBins);
}

// Level-0 split of a chunk of keys: keys above the threshold bin are
// selected, keys inside it become candidates (with the level-1 histogram).
// Each thread holds 16 keys; one workgroup prefix sum and one atomic per
// output list place them.
__global__ __launch_bounds__(kFilterBlock) void select_filter(SelArgs a) {
  __shared__ __attribute__((aligned(8))) uint32_t h[kHistBins];
  __shared__ uint32_t scan[kFilterBlock / 64 + 1];
  __shared__ int s_bin;
  __shared__ uint32_t s_krem, s_cnt;
  __shared__ uint32_t s_base[2];
  const int row = blockIdx.y;
  const int base = blockIdx.x * kFilterChunk;
  const int tid = threadIdx.x;
  // The key chunk and the level-0 histogram load before the row's length
  // (and the gate's choice) are known, so that all of them share one memory
  // latency: every key index below mcap lies inside the row's key array.
  const uint32_t* keys = a.keys + (size_t)row * a.mcap;
  uint32_t key[kFilterPerThread];
#pragma unroll
  for (int k = 0; k < kFilterPerThread; ++k) {
    const int i = base + tid + k * kFilterBlock;
    key[k] = i < a.mcap ? keys[i] : 0u;
  }
  constexpr int HPT = kHistBins / kFilterBlock;
  uint32_t hv[HPT];
#pragma unroll
  for (int j = 0; j < HPT; ++j) hv[j] = a.hist0[(size_t)row * kHistBins + tid + j * kFilterBlock];
  if (row_skipped(a, row)) return;
  const int b = row / a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  if (base >= rg.m || rg.kb <= 0) return;
  const int end = min(rg.m, base + kFilterChunk);
  const bool all = rg.kb >= rg.m;
  int bin = 0;
  bool resolved = true;
  if (!all) {
#pragma unroll
    for (int j = 0; j < HPT; ++j) h[tid + j * kFilterBlock] = hv[j];
    __syncthreads();
    find_threshold<kFilterBlock>(h, (uint32_t)rg.kb, scan, &s_bin, &s_krem, &s_cnt);
    bin = s_bin;
    resolved = (s_cnt == s_krem);
    __syncthreads();
    for (int i = tid; i < kHistBins; i += kFilterBlock) h[i] = 0u;
  }
  uint32_t tmask = 0, kmask = 0;
#pragma unroll
  for (int k = 0; k < kFilterPerThread; ++k) {
    const int i = base + tid + k * kFilterBlock;
    const int d0 = (int)(key[k] >> 21);
    const bool valid = i < end;
    const bool take = valid && (all || d0 > bin || (resolved && d0 == bin));
    const bool keep = valid && !all && !resolved && d0 == bin;
    tmask |= (take ? 1u : 0u) << k;
    kmask |= (keep ? 1u : 0u) << k;
  }
  const uint32_t packed = ((uint32_t)__popc(tmask) << 16) | (uint32_t)__popc(kmask);
  uint32_t total;
  const uint32_t pre = block_exclusive_scan<kFilterBlock>(packed, scan, &total);
  uint32_t* cnt = a.counters + row * 4;
  if (tid == 0 && total != 0u) {
    // both list offsets in one 64-bit atomic: cnt[0] (selected) is the low
    // word, cnt[1] (candidates) the high one; neither count reaches 2^32
    const unsigned long long add =
        (unsigned long long)(total >> 16) | ((unsigned long long)(total & 0xFFFFu) << 32);
    const unsigned long long old = atomicAdd((unsigned long long*)cnt, add);
    s_base[0] = (uint32_t)old;
    s_base[1] = (uint32_t)(old >> 32);
  }
  __syncthreads();
  uint32_t ot = s_base[0] + (pre >> 16), ok = s_base[1] + (pre & 0xFFFFu);
  uint2* sel = a.sel + (size_t)row * a.selcap;
  uint2* cand = a.cand + (size_t)row * a.mcap;
#pragma unroll
  for (int k = 0; k < kFilterPerThread; ++k) {
    const uint2 e = make_uint2(key[k], (uint32_t)(rg.sink_end + base + tid + k * kFilterBlock));
    if ((tmask >> k) & 1u) {
      if (ot < (uint32_t)a.selcap) sel[ot] = e;
      ++ot;
    }
    if ((kmask >> k) & 1u) {
      if (ok < (uint32_t)a.mcap) cand[ok] = e;
      atomicAdd(&h[(e.x >> 10) & 0x7FFu], 1u);
      ++ok;
    }
  }
  if (!all && !resolved) {
    __syncthreads();
    flush_hist(h, a.hist1 + (size_t)row * kHistBins);
  }
}

// Whether bitmap bm has a set bit at any position in [lo, hi).
__device__ __forceinline__ bool any_bits(const uint32_t* bm, int lo, int hi) {
  if (lo >= hi) return false;
  const int w0 = lo >> 5, w1 = (hi - 1) >> 5;
  for (int w = w0; w <= w1; ++w) {
    uint32_t m = bm[w];
    if (w == w0) m &= ~0u << (lo & 31);
    if (w == w1) m &= 0xFFFFFFFFu >> (31 - ((hi - 1) & 31));
    if (m) return true;
  }
  return false;
}

__device__ __forceinline__ uint32_t coherent_load(uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Makes this workgroup's global-memory writes visible to all of its threads.
// Workgroup scope suffices: only the writing workgroup reads them back.
__device__ __forceinline__ void block_publish() {
  __threadfence_block();
  __syncthreads();
  __threadfence_block();
}

// Splits `count` candidates of src by radix digit `level` against bin bl:
// digit above bl (or equal, when the bin is taken whole) goes to the output
// list sel; digit equal to bl is kept, either as a 64-bit composite in the LDS
// buffer `keep_lds` or in the global list `keep_glb`.  Returns the number
// kept.  Every thread of the workgroup must call it.  The first pass of
// candidates may come loaded already (`first`; values past count unused).
struct CandPass {  // one pass of candidates: src[tid + k * kFinishBlock]
  uint2 x[kFinishPerThread];
};
__device__ __forceinline__ uint32_t split_candidates(const SelArgs& a, uint32_t* nsel, uint2* sel,
                                                     const uint2* src, uint32_t count, int level,
                                                     uint32_t bl, bool resolved, uint64_t* keep_lds,
                                                     uint2* keep_glb, uint32_t* scan,
                                                     uint32_t* s_base,
                                                     const CandPass* first = nullptr) {
  const int tid = threadIdx.x;
  uint32_t kept = 0;
  for (uint32_t e0 = 0; e0 < count; e0 += kFinishBlock * kFinishPerThread) {
    uint2 x[kFinishPerThread];
    uint32_t tmask = 0, kmask = 0;
#pragma unroll
    for (int k = 0; k < kFinishPerThread; ++k) {
      const uint32_t e = e0 + tid + k * kFinishBlock;
      x[k] = first && e0 == 0 ? first->x[k] : (e < count ? src[e] : make_uint2(0u, 0u));
    }
#pragma unroll
    for (int k = 0; k < kFinishPerThread; ++k) {
      const bool valid = e0 + tid + k * kFinishBlock < count;
      const uint32_t dg = level_digit(x[k], level);
      tmask |= (valid && (dg > bl || (resolved && dg == bl)) ? 1u : 0u) << k;
      kmask |= (valid && !resolved && dg == bl ? 1u : 0u) << k;
    }
    const uint32_t packed = ((uint32_t)__popc(tmask) << 16) | (uint32_t)__popc(kmask);
    uint32_t total;
    const uint32_t pre = block_exclusive_scan<kFinishBlock>(packed, scan, &total);
    if (tid == 0) {
      *s_base = *nsel;
      *nsel += total >> 16;
    }
    __syncthreads();
    uint32_t ot = *s_base + (pre >> 16), ok = kept + (pre & 0xFFFFu);
#pragma unroll
    for (int k = 0; k < kFinishPerThread; ++k) {
      if ((tmask >> k) & 1u) {
        if (ot < (uint32_t)a.selcap) sel[ot] = x[k];
        ++ot;
      }
      if ((kmask >> k) & 1u) {
        if (keep_lds) keep_lds[ok] = composite(x[k]);
        else if (ok < (uint32_t)a.mcap) keep_glb[ok] = x[k];
        ++ok;
      }
    }
    kept += total & 0xFFFFu;
    __syncthreads();
  }
  return kept;
}

// Radix select to the end inside the global candidate lists (levels from
// `level` to 4), for the rare rows whose ties do not fit LDS.
__device__ void radix_global(const SelArgs& a, uint32_t* nsel, uint2* sel, uint2* src, uint2* dst,
                             uint32_t count, uint32_t krem, int level, uint32_t* h, uint32_t* scan,
                             int* s_bin, uint32_t* s_krem, uint32_t* s_cnt, uint32_t* s_base) {
  const int tid = threadIdx.x;
  for (; level <= 4; ++level) {
    __syncthreads();
    for (int i = tid; i < kHistBins; i += kFinishBlock) h[i] = 0u;
    __syncthreads();
    for (uint32_t e0 = 0; e0 < count; e0 += kFinishBlock * kFinishPerThread) {
      uint2 x[kFinishPerThread];
#pragma unroll
      for (int k = 0; k < kFinishPerThread; ++k) {
        const uint32_t e = e0 + tid + k * kFinishBlock;
        x[k] = e < count ? src[e] : make_uint2(0u, 0u);
      }
#pragma unroll
      for (int k = 0; k < kFinishPerThread; ++k)
        if (e0 + tid + k * kFinishBlock < count) atomicAdd(&h[level_digit(x[k], level)], 1u);
    }
    __syncthreads();
    find_threshold<kFinishBlock>(h, krem, scan, s_bin, s_krem, s_cnt);
    const uint32_t bl = (uint32_t)*s_bin;
    const bool resolved = *s_cnt == *s_krem;
    const uint32_t krem_next = *s_krem;
    const uint32_t kept = split_candidates(a, nsel, sel, src, count, level, bl, resolved, nullptr,
                                           dst, scan, s_base);
    block_publish();
    if (resolved) break;
    count = kept < (uint32_t)a.mcap ? kept : (uint32_t)a.mcap;
    krem = krem_next;
    uint2* tmp = src;
    src = dst;
    dst = tmp;
  }
}

// The k-th largest (1 <= k <= c) of the c <= kSmallRank composites among
// get(0..n-1) whose bits under pmask equal prefix: one pass gathers them into
// `small` (LDS), then each lane of wave 0 counts the gathered values above
// its own.  The values are distinct, so exactly one lane has k - 1 above it.
// Every thread must call it.
template <typename Get>
__device__ uint64_t lds_kth_small(Get get, uint32_t n, uint32_t k, uint64_t prefix, uint64_t pmask,
                                  uint64_t* small, uint32_t* s_n, uint64_t* s_out) {
  const int tid = threadIdx.x;
  if (tid == 0) *s_n = 0u;
  __syncthreads();
  for (uint32_t i = tid; i < n; i += kFinishBlock) {
    const uint64_t x = get(i);
    if ((x & pmask) == prefix) {
      const uint32_t slot = atomicAdd(s_n, 1u);
      if (slot < (uint32_t)kSmallRank) small[slot] = x;
    }
  }
  __syncthreads();
  const uint32_t c = min(*s_n, (uint32_t)kSmallRank);
  if (tid < kSmallRank) {
    const uint64_t x = (uint32_t)tid < c ? small[tid] : 0ull;
    uint32_t above = 0;
    for (uint32_t j = 0; j < c; ++j) above += small[j] > x ? 1u : 0u;
    if ((uint32_t)tid < c && above == k - 1u) *s_out = x;
  }
  __syncthreads();
  return *s_out;
}

// LDS scratch of the threshold searches.
struct KthScratch {
  uint32_t* h;
  uint32_t* scan;
  int* s_bin;
  uint32_t *s_krem, *s_cnt, *s_n;
  uint64_t *small, *s_out;
};

// Threshold T with exactly k of the n distinct composites get(0..n-1) at or
// above it (1 <= k <= n): radix select over 11-bit digits of the 54-bit
// values, stopping as soon as a whole bin is taken, and ranking the
// candidates directly once at most kSmallRank remain.  With lv0 > 0 the
// digits of levels below lv0 are already known: `prefix` (under `pmask`)
// holds them, and k counts within the `count` composites that share them
// (count may exceed the true number when unknown).  The values must be
// readable from LDS.  Every thread must call it.
template <typename Get>
__device__ uint64_t lds_kth_largest(Get get, uint32_t n, uint32_t k, const KthScratch& ks,
                                    int lv0 = 0, uint64_t prefix = 0, uint64_t pmask = 0,
                                    uint32_t count = 0xFFFFFFFFu) {
  const int tid = threadIdx.x;
  uint32_t krem = k;
  if (lv0 == 0 && count > n) count = n;
  for (int lv = lv0; lv < 5; ++lv) {
    if (count <= (uint32_t)kSmallRank)
      return lds_kth_small(get, n, krem, prefix, pmask, ks.small, ks.s_n, ks.s_out);
    const int sh = lv < 4 ? 43 - 11 * lv : 0;
    const uint64_t dmask = lv < 4 ? 0x7FFull : 0x3FFull;
    for (int i = tid; i < kHistBins; i += kFinishBlock) ks.h[i] = 0u;
    __syncthreads();
    for (uint32_t i = tid; i < n; i += kFinishBlock) {
      const uint64_t x = get(i);
      if ((x & pmask) == prefix) atomicAdd(&ks.h[(uint32_t)((x >> sh) & dmask)], 1u);
    }
    __syncthreads();
    find_threshold<kFinishBlock>(ks.h, krem, ks.scan, ks.s_bin, ks.s_krem, ks.s_cnt);
    const uint32_t bin = (uint32_t)*ks.s_bin, krem2 = *ks.s_krem, cnt = *ks.s_cnt;
    prefix |= (uint64_t)bin << sh;
    pmask |= dmask << sh;
    if (cnt == krem2) break;
    krem = krem2;
    count = cnt;
  }
  return prefix;
}

// Finishes the selection of one row (one workgroup per row): the level-0 and
// level-1 thresholds come from the histograms of the score and filter
// kernels; one pass over the level-0 candidates moves the level-1 winners to
// the output list and stages the level-1 ties in LDS.  Winners and staged
// ties, as distinct 54-bit composites in LDS, then give the exact k_b-th and
// m-th largest by LDS radix select; one segmented bitmap pass writes the top
// m, the other winners, the anchor set and the shared set, each ascending by
// position.
__global__ __launch_bounds__(kFinishBlock) void select_finish(SelArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint64_t dyn[];  // sort buffer: a.sortcap entries
  __shared__ uint32_t h[kHistBins];
  __shared__ uint32_t scan[kFinishBlock / 64 + 1];
  __shared__ uint64_t scan64[kFinishBlock / 64 + 1];
  __shared__ int s_bin;
  __shared__ uint32_t s_krem, s_cnt, s_base;
  __shared__ uint32_t s_nsel;  // entries in the row's output list sel (only this workgroup appends)
  __shared__ uint64_t s_small[kSmallRank];
  __shared__ uint64_t s_out;
  __shared__ uint32_t s_n;
  const KthScratch ks{h, scan, &s_bin, &s_krem, &s_cnt, &s_n, s_small, &s_out};
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  uint32_t* cnt = a.counters + row * 4;
  uint2* sel = a.sel + (size_t)row * a.selcap;
  const uint2* cand = a.cand + (size_t)row * a.mcap;
  // The counters, both histograms, the first pass of level-0 candidates and
  // the first kSelPrefetch winners per thread load before the row's length
  // (and the gate's choice) are known, so that they share one memory
  // latency.  Every index stays inside the row's lists (mcap candidates,
  // selcap winners); values past the counts are loaded and never used.
  const uint32_t nsel0 = coherent_load(&cnt[0]);  // the filter's winners
  const uint32_t count0_all = coherent_load(&cnt[1]);
  constexpr int HPT = kHistBins / kFinishBlock;
  uint32_t h0[HPT], h1[HPT];
#pragma unroll
  for (int j = 0; j < HPT; ++j) {
    h0[j] = a.hist0[(size_t)row * kHistBins + tid + j * kFinishBlock];
    h1[j] = a.hist1[(size_t)row * kHistBins + tid + j * kFinishBlock];
  }
  CandPass cp0;
#pragma unroll
  for (int k = 0; k < kFinishPerThread; ++k) {
    const int e = tid + k * kFinishBlock;
    cp0.x[k] = e < a.mcap ? cand[e] : make_uint2(0u, 0u);
  }
  uint2 sp0[kSelPrefetch];
#pragma unroll
  for (int k = 0; k < kSelPrefetch; ++k) {
    const int j = tid + k * kFinishBlock;
    sp0[k] = j < a.selcap ? sel[j] : make_uint2(0u, 0u);
  }
  if (row_skipped(a, row)) return;
  const int b = row / a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  uint32_t n_lds = 0;  // staged ties in dyn[0, n_lds)
  // m from the budget before clamping to the middle range (floor(k / 3) by
  // default), clamped to the winners
  const long long kraw = a.k_den > 0 ? ((long long)a.k_num * rg.n0) / a.k_den : (long long)a.k;
  const long long mm = a.dilate_m < 0 ? (kraw < 0 ? 0 : kraw) / 3 : a.dilate_m;
  const uint32_t kb_u = rg.kb > 0 ? (uint32_t)rg.kb : 0u;
  const uint32_t m0 = (uint32_t)(mm > (long long)kb_u ? kb_u : mm);
  // digits already known from the global histograms: the k-th largest lies
  // in level-0 bin b0 and level-1 bin b1, krem1 deep among the staged ties;
  // the m-th largest lies in level-0 bin bm0, kremm0 deep
  int b0 = -1, b1 = -1, bm0 = -1;
  uint32_t krem1 = 0, kremm0 = 0;
  bool m_resolved0 = false;

  if (rg.kb > 0 && rg.kb < rg.m) {
    if (tid == 0) s_nsel = nsel0;
#pragma unroll
    for (int j = 0; j < HPT; ++j) h[tid + j * kFinishBlock] = h0[j];
    __syncthreads();
    if (m0 > 0) {
      find_threshold<kFinishBlock>(h, m0, scan, &s_bin, &s_krem, &s_cnt);
      bm0 = s_bin;
      kremm0 = s_krem;
      m_resolved0 = s_cnt == s_krem;
      __syncthreads();
    }
    find_threshold<kFinishBlock>(h, (uint32_t)rg.kb, scan, &s_bin, &s_krem, &s_cnt);
    b0 = s_bin;
    if (s_cnt != s_krem) {
      const uint32_t krem0 = s_krem;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < HPT; ++j) h[tid + j * kFinishBlock] = h1[j];
      __syncthreads();
      find_threshold<kFinishBlock>(h, krem0, scan, &s_bin, &s_krem, &s_cnt);
      b1 = s_bin;
      krem1 = s_krem;
      const uint32_t c1 = s_cnt;
      const bool resolved1 = c1 == krem1;
      const bool in_lds = !resolved1 && c1 + (uint32_t)rg.kb <= (uint32_t)a.sortcap;
      const uint32_t count0 = min(count0_all, (uint32_t)a.mcap);
      uint2* cand2 = a.cand2 + (size_t)row * a.mcap;
      const uint32_t kept = split_candidates(a, &s_nsel, sel, cand, count0, 1, b1, resolved1,
                                             in_lds ? dyn : nullptr, cand2, scan, &s_base, &cp0);
      block_publish();
      if (in_lds) {
        n_lds = kept;
      } else if (!resolved1) {
        b1 = -1;
        radix_global(a, &s_nsel, sel, cand2, a.cand + (size_t)row * a.mcap,
                     min(kept, (uint32_t)a.mcap), krem1, 2, h, scan, &s_bin, &s_krem, &s_cnt,
                     &s_base);
      }
    }
  } else if (tid == 0) {
    s_nsel = nsel0;
  }
  block_publish();

  const uint32_t n_sel = rg.kb > 0 ? min(s_nsel, (uint32_t)a.selcap) : 0u;
  const uint32_t total = n_sel + n_lds;
  // winner j is sel[j]: the filter's ones (j < nsel0) prefetched for the
  // first kSelPrefetch passes, the ones appended here read back
#pragma unroll
  for (int k = 0; k < kSelPrefetch; ++k) {
    const uint32_t j = tid + k * kFinishBlock;
    if (j < n_sel) dyn[n_lds + j] = composite(j < nsel0 ? sp0[k] : sel[j]);
  }
  for (uint32_t j = tid + kSelPrefetch * kFinishBlock; j < n_sel; j += kFinishBlock)
    dyn[n_lds + j] = composite(sel[j]);
  __syncthreads();
  // winners: the kout largest composites; top: the m largest of them
  const uint32_t kout = min(total, kb_u);
  const uint32_t m = (uint32_t)(mm > (long long)kout ? kout : mm);
  auto get = [&](uint32_t i) { return dyn[i]; };
  constexpr uint64_t kD0 = 0x7FFull << 43, kD1 = 0x7FFull << 32;
  uint64_t c_k = 0ull;
  if (kout < total) {
    if (b1 >= 0 && n_lds > 0 && n_sel + krem1 == kout)  // among the ties, from level 2
      c_k = lds_kth_largest(get, n_lds, krem1, ks, 2,
                            ((uint64_t)b0 << 43) | ((uint64_t)b1 << 32), kD0 | kD1, n_lds);
    else
      c_k = lds_kth_largest(get, total, kout, ks);
  }
  uint64_t c_m = ~0ull;
  if (m > 0) {
    if (bm0 >= 0 && m == m0)  // level-0 digit from the global histogram
      c_m = m_resolved0 ? (uint64_t)bm0 << 43
                        : lds_kth_largest(get, total, kremm0, ks, 1, (uint64_t)bm0 << 43, kD0);
    else
      c_m = lds_kth_largest(get, total, m, ks);
  }
  // One ordered pass over the middle range writes all outputs: per bitmap
  // segment the winners W (x >= c_k), the top m T (x >= c_m) and the +-r
  // neighbours D of T are marked together, and one scan of four packed counts
  // gives each thread its offsets into the top m, the other winners, the
  // anchor set (W) and the shared set (W | D).  Neighbours outside the middle
  // range fall in the sink, the window or outside [0, n0).
  const bool shared = a.shared_idx != nullptr;
  const int r = a.dilate_r;
  const int seg_bits = a.seg_bits;
  const int segw = seg_bits >> 5;
  // With seg_shift the middle range is one segment and the neighbours of the
  // top m come from shifts of its bitmap (r < 32), so there is no third
  // bitmap.
  const bool shiftd = a.seg_shift != 0;
  // The bitmaps start 16-byte aligned after the sort buffer, segw is a
  // multiple of 4 (whole groups of four words), and 16 bytes of slack follow
  // the last bitmap, so that every word read below (a group of four, a word
  // before or after one) stays inside the buffer.
  uint32_t* bw = (uint32_t*)(dyn + ((a.sortcap + 1) & ~1));
  uint32_t* bt = bw + segw;
  uint32_t* bd = shiftd ? nullptr : bt + segw;
  uint32_t* bend = bt + (shiftd ? 1 : 2) * segw + 4;
  // optional per-word output offsets [segw], then the output staging
  uint64_t* woff = a.woff ? (uint64_t*)bend : nullptr;
  int32_t* stage = a.woff ? (int32_t*)(woff + segw) : (int32_t*)bend;  // a.stagecap entries
  int32_t* topk = a.topk_idx + (size_t)row * a.k_cap;
  int32_t* out = a.set_idx + (size_t)row * a.set_cap;
  int32_t* sh = shared ? a.shared_idx + (size_t)row * a.set_cap : nullptr;
  for (int i = tid; i < rg.sink_end; i += kFinishBlock) {
    if (i < a.set_cap) {
      out[i] = i;
      if (shared) sh[i] = i;
    }
  }
  int pos_t = 0, pos_r = (int)m, pos_w = rg.sink_end, pos_s = rg.sink_end;
  for (int seg_lo = rg.sink_end; seg_lo < rg.win_start; seg_lo += seg_bits) {
    const int seg_hi = min(rg.win_start, seg_lo + seg_bits);
    const int nwords = (seg_hi - seg_lo + 31) >> 5;
    const int ngrp = (nwords + 3) >> 2;  // groups of four words (the last one padded with zeros)
    const uint32_t lastw = ((seg_hi - seg_lo) & 31) ? (1u << ((seg_hi - seg_lo) & 31)) - 1u : ~0u;
    for (int w = tid; w < 4 * ngrp; w += kFinishBlock) {
      bw[w] = 0u;
      bt[w] = 0u;
      if (!shiftd) bd[w] = 0u;
    }
    lds_barrier();
    // the dilation-only neighbours of word w given the top-m words c0 (its
    // own), cp and cn (before and after it, zero outside the segment)
    auto spread = [&](int w, uint32_t c0, uint32_t cp, uint32_t cn) -> uint32_t {
      uint32_t acc = 0u;
      for (int d = 1; d <= r; ++d) acc |= (c0 << d) | (cp >> (32 - d)) | (c0 >> d) | (cn << (32 - d));
      return w == nwords - 1 ? acc & lastw : acc;
    };
    // the same for any word w < nwords: marked, or shifted from the top-m
    // words around it (all three read unconditionally: bt[-1] and bt[nwords]
    // lie inside the buffer)
    auto dil = [&](int w) -> uint32_t {
      if (!shiftd) return bd[w];
      const uint32_t c0 = bt[w], cp = bt[w - 1], cn = bt[w + 1];
      return spread(w, c0, w > 0 ? cp : 0u, w + 1 < nwords ? cn : 0u);
    };
    for (uint32_t i = tid; i < total; i += kFinishBlock) {
      const uint64_t x = dyn[i];
      if (x < c_k) continue;
      const int p = composite_pos(x);
      const bool top = x >= c_m;
      if (p >= seg_lo && p < seg_hi) {
        mark_bit(bw, seg_lo, p);
        if (top) mark_bit(bt, seg_lo, p);
      }
      if (shared && top && !shiftd) {
        const int lo = max(p - r, seg_lo), hi = min(p + r, seg_hi - 1);
        for (int q = lo; q <= hi; ++q) mark_bit(bd, seg_lo, q);
      }
    }
    __syncthreads();
    // Packed counts of a word's top m, other winners, all winners and shared
    // set; each 16-bit field of a segment's totals fits (fewer than 2^16
    // positions, or the host's bound on the outputs of one segment).
    auto word_counts = [&](int w) -> uint64_t {
      const uint32_t W = bw[w], T = bt[w], S = W | (shared ? dil(w) : 0u);
      return (uint64_t)__popc(T) | ((uint64_t)__popc(W & ~T) << 16) |
             ((uint64_t)__popc(W) << 32) | ((uint64_t)__popc(S) << 48);
    };
    const int wpt = (nwords + kFinishBlock - 1) / kFinishBlock;
    const int lane = tid & 63, wv = tid >> 6;
    // without woff: thread t owns words [t*wpt, (t+1)*wpt)
    const int w_begin = min(nwords, tid * wpt), w_end = min(nwords, w_begin + wpt);
    uint64_t tot = 0, off = 0;
    if (woff) {
      // Every word's output offsets, in word order.  Each lane takes groups
      // of four consecutive words (16-byte reads of each bitmap and the two
      // words around the group, all issued together), its group's total
      // goes through a wave scan per row of 64 groups, then one scan of the
      // waves' totals.
      const int gpt = (ngrp + kFinishBlock - 1) / kFinishBlock;
      const int gbase = wv * 64 * gpt;  // wave wv's groups, lane l at gbase + 64 j + l
      uint64_t carry = 0;
      for (int j = 0; j < gpt; ++j) {
        const int gi = gbase + 64 * j + lane;
        const int w0 = 4 * gi;
        uint64_t c[4] = {0u, 0u, 0u, 0u};
        if (gi < ngrp) {
          const uint4 W4 = *(const uint4*)(bw + w0), T4 = *(const uint4*)(bt + w0);
          const uint4 D4 = shiftd ? make_uint4(0u, 0u, 0u, 0u) : *(const uint4*)(bd + w0);
          const uint32_t tp = bt[w0 - 1], tn = bt[w0 + 4];
          const uint32_t Wv[4] = {W4.x, W4.y, W4.z, W4.w}, Tv[4] = {T4.x, T4.y, T4.z, T4.w};
          const uint32_t Dv[4] = {D4.x, D4.y, D4.z, D4.w};
          // neighbours of the group's words (pad words past nwords are zero)
          const uint32_t Pv[4] = {w0 > 0 ? tp : 0u, Tv[0], Tv[1], Tv[2]};
          const uint32_t Nv[4] = {Tv[1], Tv[2], Tv[3], w0 + 4 < nwords ? tn : 0u};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t W = Wv[i], T = Tv[i];
            const uint32_t S = W | (shared ? (shiftd ? spread(w0 + i, T, Pv[i], Nv[i]) : Dv[i]) : 0u);
            c[i] = w0 + i < nwords ? (uint64_t)__popc(T) | ((uint64_t)__popc(W & ~T) << 16) |
                                         ((uint64_t)__popc(W) << 32) | ((uint64_t)__popc(S) << 48)
                                   : 0u;
          }
        }
        const uint64_t gsum = c[0] + c[1] + c[2] + c[3];
        const uint64_t inc = wave_inclusive_scan(gsum);
        if (gi < ngrp) {
          const uint64_t o0 = carry + inc - gsum, o1 = o0 + c[0], o2 = o1 + c[1], o3 = o2 + c[2];
          ulonglong2* wo = (ulonglong2*)(woff + w0);
          wo[0] = make_ulonglong2(o0, o1);
          wo[1] = make_ulonglong2(o2, o3);
        }
        carry += (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)inc, 63) |
                 ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(inc >> 32), 63) << 32);
      }
      if (lane == 0) scan64[wv] = carry;
      lds_barrier();
      uint64_t before = 0;
      for (int v = 0; v < kFinishBlock / 64; ++v) {
        const uint64_t x = scan64[v];
        before += v < wv ? x : 0u;
        tot += x;
      }
      if (before != 0u) {
        for (int j = 0; j < gpt; ++j) {
          const int gi = gbase + 64 * j + lane;
          if (gi >= ngrp) continue;
          ulonglong2* wo = (ulonglong2*)(woff + 4 * gi);
          ulonglong2 x0 = wo[0], x1 = wo[1];
          x0.x += before; x0.y += before; x1.x += before; x1.y += before;
          wo[0] = x0;
          wo[1] = x1;
        }
      }
    } else {
      uint64_t cnt = 0;
      for (int w = w_begin; w < w_end; ++w) cnt += word_counts(w);
      off = block_exclusive_scan<kFinishBlock, uint64_t>(cnt, scan64, &tot);
    }
    // the segment's outputs: top m, other winners, anchor set, shared set
    const int n_t = (int)(tot & 0xFFFFu), n_r = (int)((tot >> 16) & 0xFFFFu);
    const int n_w = (int)((tot >> 32) & 0xFFFFu), n_s = shared ? (int)(tot >> 48) : 0;
    // Staged in LDS when they fit, then copied out with whole-wave stores
    // (scattered stores from the bit loop below leave most lanes idle and
    // cost the CU one store instruction per few entries); else written
    // directly.
    const bool staged = n_t + n_r + n_w + n_s <= a.stagecap;
    int32_t* dt = staged ? stage : topk + pos_t;
    int32_t* dr = staged ? stage + n_t : topk + pos_r;
    int32_t* dw = staged ? stage + n_t + n_r : out + pos_w;
    int32_t* ds = staged ? stage + n_t + n_r + n_w : (shared ? sh + pos_s : nullptr);
    const int lim_t = staged ? n_t : a.k_cap - pos_t, lim_r = staged ? n_r : a.k_cap - pos_r;
    const int lim_w = staged ? n_w : a.set_cap - pos_w, lim_s = staged ? n_s : a.set_cap - pos_s;
    if (woff) {
      // Per-entry writes: with each word's output offsets in LDS, every
      // winner places itself (word offset + set bits below it), so clustered
      // winners do not serialise on the thread owning their words; the
      // dilation-only positions of the shared set are placed by the top-m
      // winners that reach them (shifted dilation) or walked per word.
      lds_barrier();
      for (uint32_t i = tid; i < total; i += kFinishBlock) {
        const uint64_t x = dyn[i];
        if (x < c_k) continue;
        const int p = composite_pos(x);
        if (p < seg_lo || p >= seg_hi) continue;
        const int rel = p - seg_lo, w = rel >> 5;
        const uint32_t below = (1u << (rel & 31)) - 1u;
        const uint64_t o = woff[w];
        const uint32_t W = bw[w], T = bt[w];
        if (x >= c_m) {
          const int j = (int)(o & 0xFFFFu) + __popc(T & below);
          if (j < lim_t) dt[j] = p;
        } else {
          const int j = (int)((o >> 16) & 0xFFFFu) + __popc(W & ~T & below);
          if (j < lim_r) dr[j] = p;
        }
        const int jw = (int)((o >> 32) & 0xFFFFu) + __popc(W & below);
        if (jw < lim_w) dw[jw] = p;
        if (shared) {
          const int js = (int)(o >> 48) + __popc((W | dil(w)) & below);
          if (js < lim_s) ds[js] = p;
        }
        if (shared && shiftd && x >= c_m) {
          // the dilation-only neighbours of this top-m winner that no lower
          // top-m winner reaches (each is written by the lowest one in reach)
          for (int d = -r; d <= r; ++d) {
            const int q = rel + d;
            if (d == 0 || q < 0 || q >= seg_hi - seg_lo) continue;
            const int wq = q >> 5;
            const uint32_t bq = 1u << (q & 31);
            const uint32_t Wq = bw[wq];
            if ((Wq & bq) || any_bits(bt, max(0, q - r), rel)) continue;
            const int js = (int)(woff[wq] >> 48) + __popc((Wq | dil(wq)) & (bq - 1u));
            if (js < lim_s) ds[js] = seg_lo + q;
          }
        }
      }
      if (shared && !shiftd) {
        for (int w = tid; w < nwords; w += kFinishBlock) {
          const uint32_t W = bw[w], S = W | dil(w);
          uint32_t bits = S & ~W;
          const int js0 = (int)(woff[w] >> 48);
          while (bits) {
            const int bit = __ffs(bits) - 1;
            bits &= bits - 1u;
            const int js = js0 + __popc(S & ((1u << bit) - 1u));
            if (js < lim_s) ds[js] = seg_lo + (w << 5) + bit;
          }
        }
      }
    } else {
      int ot = (int)(off & 0xFFFFu), orr = (int)((off >> 16) & 0xFFFFu);
      int ow = (int)((off >> 32) & 0xFFFFu), os = (int)(off >> 48);
      for (int w = w_begin; w < w_end; ++w) {
        const uint32_t W = bw[w], T = bt[w];
        uint32_t bits = shared ? (W | dil(w)) : W;
        const int base = seg_lo + (w << 5);
        while (bits) {
          const int bit = __ffs(bits) - 1;
          const uint32_t one = 1u << bit;
          bits &= bits - 1u;
          const int p = base + bit;
          if (W & one) {
            if (T & one) {
              if (ot < lim_t) dt[ot] = p;
              ++ot;
            } else {
              if (orr < lim_r) dr[orr] = p;
              ++orr;
            }
            if (ow < lim_w) dw[ow] = p;
            ++ow;
          }
          if (shared) {
            if (os < lim_s) ds[os] = p;
            ++os;
          }
        }
      }
    }
    if (staged) {
      lds_barrier();
      for (int i = tid; i < n_t; i += kFinishBlock)
        if (pos_t + i < a.k_cap) topk[pos_t + i] = stage[i];
      for (int i = tid; i < n_r; i += kFinishBlock)
        if (pos_r + i < a.k_cap) topk[pos_r + i] = stage[n_t + i];
      for (int i = tid; i < n_w; i += kFinishBlock)
        if (pos_w + i < a.set_cap) out[pos_w + i] = stage[n_t + n_r + i];
      for (int i = tid; i < n_s; i += kFinishBlock)
        if (pos_s + i < a.set_cap) sh[pos_s + i] = stage[n_t + n_r + n_w + i];
    }
    pos_t += n_t;
    pos_r += n_r;
    pos_w += n_w;
    pos_s += (int)(tot >> 48);
    lds_barrier();
  }
  if (tid == 0) a.topk_len[row] = (int32_t)kout;
  // then the window, after the winners (and after the dilated middle)
  const int nw = rg.n0 - rg.win_start;
  for (int i = tid; i < nw; i += kFinishBlock) {
    if (pos_w + i < a.set_cap) out[pos_w + i] = rg.win_start + i;
    if (shared && pos_s + i < a.set_cap) sh[pos_s + i] = rg.win_start + i;
  }
  if (nw > 0) {
    pos_w += nw;
    pos_s += nw;
  }
  if (tid == 0) {
    a.set_len[row] = pos_w < a.set_cap ? pos_w : a.set_cap;
    if (shared) a.shared_len[row] = pos_s < a.set_cap ? pos_s : a.set_cap;
  }
  // leave the row's histograms and counters zero for the next call (every
  // thread read its own histogram entries and the counters long before)
  for (int i = tid; i < kHistBins; i += kFinishBlock) {
    a.hist0[(size_t)row * kHistBins + i] = 0u;
    a.hist1[(size_t)row * kHistBins + i] = 0u;
  }
  if (tid < 4) cnt[tid] = 0u;
}

// Exact threshold of one selection target over the LDS key array: a key
// with (key >> sh) > p is selected, and so are the first `take` keys (in
// position order) with (key >> sh) == p.  take = 0xFFFFFFFF selects them
// all.  Because ties go to the lower position, this is the same set as the
// k largest (key, -position) composites.
struct KeyThreshold {
  int sh;
  uint32_t p, take;
};

// Radix levels over the 32-bit key: bits [31:21], [20:10], [9:0].
__device__ __forceinline__ int key_level_shift(int lv) { return lv == 0 ? 21 : (lv == 1 ? 10 : 0); }

// The crossing bins of two targets in one pass over two histograms: for
// target j (ka for ha, kb for hb; 0 = no search), the bin where the count
// taken from the top reaches the target, the remainder taken inside it and
// its count, into res[3j .. 3j + 2].  One packed scan serves both.  Every
// thread must call it.
template <int BLOCK>
__device__ void find_threshold_pair(const uint32_t* ha, const uint32_t* hb, uint32_t ka,
                                    uint32_t kb, uint64_t* scan64, uint32_t* res) {
  constexpr int BPT = kHistBins / BLOCK;
  const int t = threadIdx.x;
  uint32_t la = 0, lb = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int bin = kHistBins - 1 - (t * BPT + i);
    la += ha[bin];
    lb += hb[bin];
  }
  uint64_t total;
  // the barrier below comes before scan64 is written again
  const uint64_t cum = block_exclusive_scan<BLOCK, uint64_t, false>(
      (uint64_t)la | ((uint64_t)lb << 32), scan64, &total);
  uint32_t ca = (uint32_t)cum, cb = (uint32_t)(cum >> 32);
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int bin = kHistBins - 1 - (t * BPT + i);
    const uint32_t c = ha[bin], d = hb[bin];
    if (ca < ka && ca + c >= ka) {
      res[0] = (uint32_t)bin;
      res[1] = ka - ca;
      res[2] = c;
    }
    if (cb < kb && cb + d >= kb) {
      res[3] = (uint32_t)bin;
      res[4] = kb - cb;
      res[5] = d;
    }
    ca += c;
    cb += d;
  }
  lds_barrier();
}

// Thresholds for the ka and the kb largest of the n LDS keys at once (a
// target of 0 selects nothing, one of n or more everything): radix levels
// in lockstep, one pass over the keys per level building both targets'
// next-digit histograms (h for ka, h2 for kb), one scan finding both bins.
// h holds the level-0 histogram (key >> 21) of all n keys on entry; h and h2
// are overwritten.  res: 6 words of LDS.  Reached by every thread.
template <int BLOCK>
__device__ void key_threshold_pair(const uint32_t* keys, uint32_t n, uint32_t ka, uint32_t kb,
                                   uint32_t* h, uint32_t* h2, uint64_t* scan64, uint32_t* res,
                                   KeyThreshold* out) {
  const int tid = threadIdx.x;
  KeyThreshold t[2];
  uint32_t kk[2] = {ka, kb};
  bool live[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    live[j] = kk[j] > 0 && kk[j] < n;
    if (kk[j] == 0) t[j] = {0, 0xFFFFFFFFu, 0u};       // nothing: key > max never holds
    else if (kk[j] >= n) t[j] = {0, 0u, 0xFFFFFFFFu};  // everything
    else t[j] = {21, 0u, 0u};
  }
  for (int lv = 0; lv < 3 && (live[0] || live[1]); ++lv) {
    const int sh = key_level_shift(lv);
    if (lv > 0) {
      // next-digit histograms over the keys that share each live prefix (a
      // finished target's prefix is replaced by a value no key shift reaches)
      const int psh = key_level_shift(lv - 1);
      const uint32_t dmask = lv == 1 ? 0x7FFu : 0x3FFu;
      const uint32_t pa = live[0] ? t[0].p : 0xFFFFFFFFu, pb = live[1] ? t[1].p : 0xFFFFFFFFu;
      for (int i = tid; i < kHistBins; i += BLOCK) {
        if (live[0]) h[i] = 0u;
        if (live[1]) h2[i] = 0u;
      }
      lds_barrier();
      // four consecutive keys per thread and read (16-byte LDS reads of
      // consecutive lanes; the array is 16-byte aligned), the last partial
      // group element by element
      for (uint32_t i0 = 4 * tid; i0 < n; i0 += 4 * BLOCK) {
        uint32_t kv[4];
        if (i0 + 4 <= n) {
          const uint4 v = *(const uint4*)(keys + i0);
          kv[0] = v.x;
          kv[1] = v.y;
          kv[2] = v.z;
          kv[3] = v.w;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) kv[u] = keys[min(i0 + u, n - 1)];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const bool in = i0 + u < n;
          const uint32_t x = kv[u] >> psh, d = (kv[u] >> sh) & dmask;
          if (in && x == pa) atomicAdd(&h[d], 1u);
          if (in && x == pb) atomicAdd(&h2[d], 1u);
        }
      }
      lds_barrier();
    }
    find_threshold_pair<BLOCK>(h, lv == 0 ? h : h2, live[0] ? kk[0] : 0u, live[1] ? kk[1] : 0u,
                               scan64, res);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (!live[j]) continue;
      const uint32_t bin = res[3 * j], krem = res[3 * j + 1], cnt = res[3 * j + 2];
      t[j].p = lv == 0 ? bin : ((t[j].p << (key_level_shift(lv - 1) - sh)) | bin);
      t[j].sh = sh;
      if (cnt == krem) {  // the whole bin is taken
        t[j].take = 0xFFFFFFFFu;
        live[j] = false;
      } else {
        kk[j] = krem;
      }
    }
  }
  // the first kk keys equal to the full 32-bit threshold
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (live[j]) t[j].take = kk[j];
    out[j] = t[j];
  }
}

// The t lowest set bits of x (all of them when x has t or fewer).
__device__ __forceinline__ uint64_t lowest_bits(uint64_t x, uint32_t t) {
  if (t >= (uint32_t)__popcll(x)) return x;
  uint64_t r = 0;
  for (uint32_t j = 0; j < t; ++j) {
    const uint64_t b = x & (~x + 1u);
    r |= b;
    x ^= b;
  }
  return r;
}

constexpr int kFusedMaxKeys = 24576;         // middle range held in LDS (96 KB)
constexpr int kBmWords = kFusedMaxKeys / 32;  // words of a bitmap over the middle range
static_assert(2 * kBmWords <= kHistBins, "two selection bitmaps in the histogram");
static_assert(kFusedMaxKeys % 64 == 0, "whole 64-key chunks");
// LDS scratch of the selection half beside the histogram: the second
// threshold histogram, then the shared-set bitmap and two tie bitmaps
constexpr int kTailScratchWords = 3 * kBmWords > kHistBins ? 3 * kBmWords : kHistBins;

// x with the value of lane L replaced by the wave-uniform v (v_writelane
// writes that lane whatever the execution mask).
template <int L>
__device__ __forceinline__ uint32_t put_lane(uint32_t x, uint32_t v) {
  asm("v_writelane_b32 %0, %1, %2" : "+v"(x) : "s"(v), "i"(L));
  return x;
}

// A value every lane of the wave holds, moved to a scalar register.
__device__ __forceinline__ uint32_t wave_uniform(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)x);
}
__device__ __forceinline__ uint64_t wave_uniform(uint64_t x) {
  return (uint64_t)wave_uniform((uint32_t)x) | ((uint64_t)wave_uniform((uint32_t)(x >> 32)) << 32);
}

// Lanes of chunk c (middle indices 64c + lane) that lie below M.
__device__ __forceinline__ uint64_t chunk_lanes(int c, int M) {
  const int rem = M - (c << 6);
  return rem >= 64 ? ~0ull : (rem <= 0 ? 0ull : (1ull << rem) - 1ull);
}

// Thresholds of the two selections as compare bounds: keys above G are
// taken and keys in [E, G] are ties, of which `take` are taken in position
// order (all when unbounded).  A selection's candidates are the keys at or
// above C: C = E, except without ties taken (take = 0), where C = G + 1 (no
// key at all when G is the largest key: cnone).  Where a bounded, nonzero
// number of ties is taken, the keys above G are kept apart as well.
struct SelBounds {
  uint32_t Gm, Cm, Gk, Ck;
  bool cnone_m, cnone_k;
};

// Lane masks of chunk c's 64 keys (key of this lane in kv), kept in lane J
// of the wave's registers: w[0..1] the top-m candidates, w[2..3] those of
// k_b, and with SPLIT w[4..7] the keys above G of each.
template <int J, bool SPLIT>
__device__ __forceinline__ void chunk_masks(uint32_t kv, int c, int M, const SelBounds& sb,
                                            uint32_t (&w)[8]) {
  const uint64_t vm = chunk_lanes(c, M);
  const uint64_t cm = __builtin_amdgcn_ballot_w64(kv >= sb.Cm) & (sb.cnone_m ? 0ull : vm);
  const uint64_t ck = __builtin_amdgcn_ballot_w64(kv >= sb.Ck) & (sb.cnone_k ? 0ull : vm);
  w[0] = put_lane<J>(w[0], (uint32_t)cm);
  w[1] = put_lane<J>(w[1], (uint32_t)(cm >> 32));
  w[2] = put_lane<J>(w[2], (uint32_t)ck);
  w[3] = put_lane<J>(w[3], (uint32_t)(ck >> 32));
  if (SPLIT) {
    const uint64_t gtm = __builtin_amdgcn_ballot_w64(kv > sb.Gm) & vm;
    const uint64_t gtk = __builtin_amdgcn_ballot_w64(kv > sb.Gk) & vm;
    w[4] = put_lane<J>(w[4], (uint32_t)gtm);
    w[5] = put_lane<J>(w[5], (uint32_t)(gtm >> 32));
    w[6] = put_lane<J>(w[6], (uint32_t)gtk);
    w[7] = put_lane<J>(w[7], (uint32_t)(gtk >> 32));
  }
}

// Four chunks from J0 of block blk (chunks 16 blk + j), their loads first.
template <int J0, bool SPLIT>
__device__ __forceinline__ void chunk_masks4(const uint32_t* s_keys, int blk, int M, int lane,
                                             const SelBounds& sb, uint32_t (&w)[8]) {
  const int c = (blk << 4) + J0;
  uint32_t kv[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) kv[u] = s_keys[min(((c + u) << 6) + lane, M - 1)];
  chunk_masks<J0 + 0, SPLIT>(kv[0], c + 0, M, sb, w);
  chunk_masks<J0 + 1, SPLIT>(kv[1], c + 1, M, sb, w);
  chunk_masks<J0 + 2, SPLIT>(kv[2], c + 2, M, sb, w);
  chunk_masks<J0 + 3, SPLIT>(kv[3], c + 3, M, sb, w);
}

// Candidate masks cm (top m) and ck (top k_b) of one chunk into lane J of w.
template <int J>
__device__ __forceinline__ void put_masks(uint32_t (&w)[4], uint64_t cm, uint64_t ck) {
  w[0] = put_lane<J>(w[0], (uint32_t)cm);
  w[1] = put_lane<J>(w[1], (uint32_t)(cm >> 32));
  w[2] = put_lane<J>(w[2], (uint32_t)ck);
  w[3] = put_lane<J>(w[3], (uint32_t)(ck >> 32));
}

// Four whole chunks from J0 of a block of 16 inside the middle range (keys
// of this lane at kp[64 j]): candidates are the keys above Tm and Tk.
template <int J0>
__device__ __forceinline__ void chunk_masks4_inner(const uint32_t* kp, uint32_t Tm, uint32_t Tk,
                                                   uint32_t (&w)[4]) {
  uint32_t kv[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) kv[u] = kp[(J0 + u) << 6];
  put_masks<J0 + 0>(w, __builtin_amdgcn_ballot_w64(kv[0] > Tm), __builtin_amdgcn_ballot_w64(kv[0] > Tk));
  put_masks<J0 + 1>(w, __builtin_amdgcn_ballot_w64(kv[1] > Tm), __builtin_amdgcn_ballot_w64(kv[1] > Tk));
  put_masks<J0 + 2>(w, __builtin_amdgcn_ballot_w64(kv[2] > Tm), __builtin_amdgcn_ballot_w64(kv[2] > Tk));
  put_masks<J0 + 3>(w, __builtin_amdgcn_ballot_w64(kv[3] > Tm), __builtin_amdgcn_ballot_w64(kv[3] > Tk));
}

// The candidate and strict bitmaps of the middle range (words 2c, 2c + 1
// for chunk c): wave w takes blocks of 16 chunks from block w in steps of
// W; lane j collects chunk j's words, then lanes 0..15 store them.  With
// `inner` (every tie or none taken, and no candidate bound at 0, so that
// "above T" expresses each selection), blocks wholly inside the middle
// range take the short path.
template <int W, bool SPLIT>
__device__ __forceinline__ void build_bitmaps(const uint32_t* s_keys, int M, int wave, int lane,
                                              const SelBounds& sb, bool inner, uint32_t Tm,
                                              uint32_t Tk, uint32_t* wm, uint32_t* wk,
                                              uint32_t* wgm, uint32_t* wgk) {
  const int nch = (M + 63) >> 6;
  const int nblk = (nch + 15) >> 4;
  for (int blk = wave; blk < nblk; blk += W) {
    if (!SPLIT && inner && ((blk + 1) << 10) <= M) {
      uint32_t w4[4] = {0u, 0u, 0u, 0u};
      const uint32_t* kp = s_keys + (blk << 10) + lane;
      chunk_masks4_inner<0>(kp, Tm, Tk, w4);
      chunk_masks4_inner<4>(kp, Tm, Tk, w4);
      chunk_masks4_inner<8>(kp, Tm, Tk, w4);
      chunk_masks4_inner<12>(kp, Tm, Tk, w4);
      if (lane < 16) {
        ((uint2*)wm)[(blk << 4) + lane] = make_uint2(w4[0], w4[1]);
        ((uint2*)wk)[(blk << 4) + lane] = make_uint2(w4[2], w4[3]);
      }
      continue;
    }
    uint32_t w8[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    chunk_masks4<0, SPLIT>(s_keys, blk, M, lane, sb, w8);
    chunk_masks4<4, SPLIT>(s_keys, blk, M, lane, sb, w8);
    chunk_masks4<8, SPLIT>(s_keys, blk, M, lane, sb, w8);
    chunk_masks4<12, SPLIT>(s_keys, blk, M, lane, sb, w8);
    const int c = (blk << 4) + lane;
    if (lane < 16 && c < nch) {
      ((uint2*)wm)[c] = make_uint2(w8[0], w8[1]);
      ((uint2*)wk)[c] = make_uint2(w8[2], w8[3]);
      if (SPLIT) {
        ((uint2*)wgm)[c] = make_uint2(w8[4], w8[5]);
        ((uint2*)wgk)[c] = make_uint2(w8[6], w8[7]);
      }
    }
  }
}

// Whole refresh of one row in one workgroup, for many short rows: MFMA
// scores of the middle range into LDS as order-preserving keys with their
// level-0 histogram, then the selection half below (exact thresholds for
// the k_b and m largest, the selections as position-ordered bitmaps, which
// also settle ties): top m, other winners, anchor set, shared set.
// Contiguous bf16 caches whose middle range fits LDS.
// Row of fused-refresh workgroup w when there are more rows than CUs: rows
// by decreasing length.  One workgroup per CU: the workgroups that start
// last, as earlier ones finish, carry the shortest rows (longest-first
// scheduling); several side by side on a CU: serpentine ranks pair long
// rows with short ones.  Sequences rank by length, ties by index; all kv
// heads of a sequence have its length.  A mapping only: every row is taken
// exactly once.
constexpr int kBalanceMaxBatch = 256;

__device__ int fused_row(const SelArgs& a, int w, int* s_len, int* s_row) {
  const int ncu = a.balance_cus;
  const int B = a.kv.batch, H = a.kv.hkv, rows = B * H;
  if (ncu <= 0 || rows <= ncu || B > kBalanceMaxBatch) return w;
  // one workgroup per CU: later workgroups start as earlier ones finish, so
  // rank order is longest first; several per CU side by side: serpentine
  const int t = a.balance_serpentine ? serpentine_rank(w, ncu, rows) : w;
  return unit_of_length_rank(a.kv, H, t, s_len, s_row);
}

// Selection half of the fused refresh, after the row's middle-range keys
// (order-preserving u32, position order) are in s_keys and their level-0
// histogram (key >> 21) in h: exact thresholds for the k_b and m largest,
// the selections as bitmaps over the middle positions (whose order settles
// ties), and from them the top m, the other winners, the anchor set and,
// with a shared-set output, the dilated shared set.  h2: kTailScratchWords
// words of LDS scratch; res: 6 words.  Reached by every thread of the
// workgroup.
template <int BLOCK>
__device__ void fused_select_tail(const SelArgs& a, int row, const RowGeom& rg, uint32_t* s_keys,
                                  uint32_t* h, uint32_t* h2, uint64_t* scan64, uint32_t* res) {
  constexpr int W = BLOCK / 64;
  static_assert(kHistBins % BLOCK == 0, "whole histogram bins per thread");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int M = rg.m;
  const int se = rg.sink_end;
  const uint32_t kout = (uint32_t)rg.kb;
  const long long kraw = a.k_den > 0 ? ((long long)a.k_num * rg.n0) / a.k_den : (long long)a.k;
  long long mm = a.dilate_m < 0 ? (kraw < 0 ? 0 : kraw) / 3 : a.dilate_m;
  const uint32_t m = (uint32_t)(mm > (long long)kout ? kout : mm);
  KeyThreshold th[2];
  key_threshold_pair<BLOCK>(s_keys, (uint32_t)M, m, kout, h, h2, scan64, res, th);
  const KeyThreshold tm = th[0], tk = th[1];
  // The selections as bitmaps over the middle indices (bit i % 32 of word
  // i / 32 for middle index i), built a chunk of 64 keys per wave step from
  // lane masks of the compares: a threshold (sh, p) splits the keys into
  // those above G = (p << sh) | (2^sh - 1), the ties in [p << sh, G], and
  // the rest.  Every tie is taken when take is unbounded, none when it is 0;
  // otherwise the first `take` ties in position order (pass below).
  const bool shared = a.shared_idx != nullptr;
  const int nwords = (M + 31) >> 5;
  uint32_t* wm = h;                   // top m
  uint32_t* wk = h + kBmWords;        // top k_b
  uint32_t* wsh = h2;                 // dilated shared set
  uint32_t* wgm = h2 + kBmWords;      // keys above the m threshold (split ties only)
  uint32_t* wgk = h2 + 2 * kBmWords;  // keys above the k_b threshold (split ties only)
  const uint32_t take_m = wave_uniform(tm.take), take_k = wave_uniform(tk.take);
  const bool split_m = take_m != 0xFFFFFFFFu && take_m != 0u;
  const bool split_k = take_k != 0xFFFFFFFFu && take_k != 0u;
  SelBounds sb;
  sb.Gm = wave_uniform((tm.p << tm.sh) | ((1u << tm.sh) - 1u));
  sb.Gk = wave_uniform((tk.p << tk.sh) | ((1u << tk.sh) - 1u));
  sb.Cm = take_m == 0u ? sb.Gm + 1u : wave_uniform(tm.p << tm.sh);
  sb.Ck = take_k == 0u ? sb.Gk + 1u : wave_uniform(tk.p << tk.sh);
  sb.cnone_m = take_m == 0u && sb.Gm == 0xFFFFFFFFu;
  sb.cnone_k = take_k == 0u && sb.Gk == 0xFFFFFFFFu;
  // "above T" forms: T = C - 1, or G where no tie is taken
  const uint32_t Tm = take_m == 0u ? sb.Gm : sb.Cm - 1u, Tk = take_k == 0u ? sb.Gk : sb.Ck - 1u;
  const bool inner = !split_m && !split_k && (take_m == 0u || sb.Cm > 0u) && (take_k == 0u || sb.Ck > 0u);
  if (split_m || split_k)
    build_bitmaps<W, true>(s_keys, M, wave, lane, sb, inner, Tm, Tk, wm, wk, wgm, wgk);
  else
    build_bitmaps<W, false>(s_keys, M, wave, lane, sb, inner, Tm, Tk, wm, wk, wgm, wgk);
  lds_barrier();
  // thread t owns words [t * wpt, (t + 1) * wpt)
  const int wpt = (nwords + BLOCK - 1) / BLOCK;
  const int w_begin = min(nwords, tid * wpt), w_end = min(nwords, w_begin + wpt);
  if (split_m || split_k) {
    // split ties: keep the first `take` of them in position order
    uint32_t em = 0, ek = 0;
    for (int w = w_begin; w < w_end; ++w) {
      if (split_m) em += (uint32_t)__popc(wm[w] & ~wgm[w]);
      if (split_k) ek += (uint32_t)__popc(wk[w] & ~wgk[w]);
    }
    uint64_t tt;
    const uint64_t pe = block_exclusive_scan<BLOCK, uint64_t>((uint64_t)em | ((uint64_t)ek << 32), scan64, &tt);
    uint32_t rm = (uint32_t)pe, rk = (uint32_t)(pe >> 32);
    for (int w = w_begin; w < w_end; ++w) {
      if (split_m) {
        const uint32_t eq = wm[w] & ~wgm[w];
        wm[w] = wgm[w] | (uint32_t)lowest_bits(eq, take_m > rm ? take_m - rm : 0u);
        rm += (uint32_t)__popc(eq);
      }
      if (split_k) {
        const uint32_t eq = wk[w] & ~wgk[w];
        wk[w] = wgk[w] | (uint32_t)lowest_bits(eq, take_k > rk ? take_k - rk : 0u);
        rk += (uint32_t)__popc(eq);
      }
    }
    lds_barrier();
  }
  const int r = a.dilate_r;
  if (shared) {
    // the winners and the +-r neighbours of the top m that stay in the
    // middle range; radii below one word by shifts of neighbouring words
    const uint32_t last = (M & 31) ? (1u << (M & 31)) - 1u : 0xFFFFFFFFu;
    for (int w = w_begin; w < w_end; ++w) {
      uint32_t acc = wk[w];
      if (r < 32) {
        const uint32_t c0 = wm[w], cp = w > 0 ? wm[w - 1] : 0u, cn = w + 1 < nwords ? wm[w + 1] : 0u;
        for (int d = 1; d <= r; ++d) acc |= (c0 << d) | (cp >> (32 - d)) | (c0 >> d) | (cn << (32 - d));
      }
      wsh[w] = w == nwords - 1 ? acc & last : acc;
    }
    if (r >= 32) {
      lds_barrier();
      for (int w = w_begin; w < w_end; ++w) {
        uint32_t bits = wm[w];
        while (bits) {
          const int i = (w << 5) + __ffs(bits) - 1;
          bits &= bits - 1u;
          const int lo = max(0, i - r), hi = min(M - 1, i + r);
          for (int x = lo >> 5; x <= hi >> 5; ++x) {
            const int b0 = max(lo - (x << 5), 0), b1 = min(hi - (x << 5), 31);
            const uint32_t span = (b1 - b0 == 31) ? 0xFFFFFFFFu : (((1u << (b1 - b0 + 1)) - 1u) << b0);
            atomicOr(&wsh[x], span);
          }
        }
      }
    }
    lds_barrier();
  }
  // output offsets: one scan of four 16-bit counts per thread (top m, the
  // other winners, all winners, the shared set), over 16-bit units of the
  // bitmaps so that every wave takes part: thread t owns units
  // [t * upt, (t + 1) * upt)
  const int nunits = (M + 15) >> 4;
  const int upt = (nunits + BLOCK - 1) / BLOCK;
  const int u_begin = min(nunits, tid * upt), u_end = min(nunits, u_begin + upt);
  uint32_t cm = 0, co = 0, ck = 0, cs = 0;
  for (int u = u_begin; u < u_end; ++u) {
    const int sh16 = (u & 1) << 4;
    const uint32_t x = (wm[u >> 1] >> sh16) & 0xFFFFu, y = (wk[u >> 1] >> sh16) & 0xFFFFu;
    cm += (uint32_t)__popc(x);
    co += (uint32_t)__popc(y & ~x);
    ck += (uint32_t)__popc(y);
    if (shared) cs += (uint32_t)__popc((wsh[u >> 1] >> sh16) & 0xFFFFu);
  }
  uint64_t tot;
  const uint64_t pre = block_exclusive_scan<BLOCK, uint64_t>(
      (uint64_t)cm | ((uint64_t)co << 16) | ((uint64_t)ck << 32) | ((uint64_t)cs << 48), scan64, &tot);
  int32_t* topk = a.topk_idx + (size_t)row * a.k_cap;
  int32_t* out = a.set_idx + (size_t)row * a.set_cap;
  int32_t* shv = shared ? a.shared_idx + (size_t)row * a.set_cap : nullptr;
  uint32_t oa = (uint32_t)pre & 0xFFFFu, ob = m + ((uint32_t)(pre >> 16) & 0xFFFFu);
  uint32_t os = se + ((uint32_t)(pre >> 32) & 0xFFFFu), ss = se + (uint32_t)(pre >> 48);
  const uint32_t kcap = (uint32_t)a.k_cap, scap = (uint32_t)a.set_cap;
  for (int u = u_begin; u < u_end; ++u) {
    const int base = se + (u << 4), sh16 = (u & 1) << 4;
    const uint32_t x = (wm[u >> 1] >> sh16) & 0xFFFFu, y = (wk[u >> 1] >> sh16) & 0xFFFFu;
    for (uint32_t bits = x; bits; bits &= bits - 1u, ++oa)
      if (oa < kcap) topk[oa] = base + __ffs(bits) - 1;
    for (uint32_t bits = y & ~x; bits; bits &= bits - 1u, ++ob)
      if (ob < kcap) topk[ob] = base + __ffs(bits) - 1;
    for (uint32_t bits = y; bits; bits &= bits - 1u, ++os)
      if (os < scap) out[os] = base + __ffs(bits) - 1;
    if (shared)
      for (uint32_t bits = (wsh[u >> 1] >> sh16) & 0xFFFFu; bits; bits &= bits - 1u, ++ss)
        if (ss < scap) shv[ss] = base + __ffs(bits) - 1;
  }
  const uint32_t total_k = (uint32_t)(tot >> 32) & 0xFFFFu;
  const uint32_t total_s = (uint32_t)(tot >> 48);
  const int nw = rg.n0 - rg.win_start;
  int pos = se + (int)total_k, pos2 = se + (int)total_s;
  for (int i = tid; i < se; i += BLOCK) {
    if (i < a.set_cap) out[i] = i;
    if (shared && i < a.set_cap) shv[i] = i;
  }
  for (int i = tid; i < nw; i += BLOCK) {
    if (pos + i < a.set_cap) out[pos + i] = rg.win_start + i;
    if (shared && pos2 + i < a.set_cap) shv[pos2 + i] = rg.win_start + i;
  }
  if (nw > 0) {
    pos += nw;
    pos2 += nw;
  }
  if (tid == 0) {
    a.topk_len[row] = (int32_t)kout;
    a.set_len[row] = pos < a.set_cap ? pos : a.set_cap;
    if (shared) a.shared_len[row] = pos2 < a.set_cap ? pos2 : a.set_cap;
  }
}

template <int D, int BLOCK>
__global__ __launch_bounds__(BLOCK) void select_fused(SelArgs a) {
  constexpr int KS = D / 32;
  extern __shared__ __attribute__((aligned(16))) uint32_t s_keys[];  // [middle length]
  __shared__ uint32_t h[kHistBins];
  __shared__ uint64_t scan64[BLOCK / 64 + 1];
  __shared__ uint32_t s_res[6];
  __shared__ int s_len[kBalanceMaxBatch];
  __shared__ int s_row;
  __shared__ u32x4_t s_kst[BLOCK / 64][16 * (D / 8)];
  static_assert(sizeof(s_kst) >= kTailScratchWords * sizeof(uint32_t),
                "the selection's scratch in the staging tiles");
  __shared__ int s_choice;
  const int row = fused_row(a, blockIdx.x, s_len, &s_row);
  if (a.gate_fused) {
    // the gate of this row's unit (recording the step); a sharing row is done
    if (threadIdx.x < 64) {
      const int c = gate_unit<__bf16>(a.gate, row, threadIdx.x);
      if (threadIdx.x == 0) s_choice = c;
    }
    lds_barrier();
    if (s_choice >= 0) return;
  } else if (row_skipped(a, row)) {
    return;
  }
  const int b = row / a.kv.hkv, g = row % a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  const int tid = threadIdx.x;
  const int M = rg.m;
  for (int i = tid; i < kHistBins; i += BLOCK) h[i] = 0u;
  __syncthreads();
  if (rg.kb > 0) {
    const int lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const int G = a.kv.hq / a.kv.hkv;
    const __bf16* q = (const __bf16*)a.q;
    bf16x8_t qf[KS];
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int qh = col < G ? col : 0;
      const uint4* qp = (const uint4*)(q + ((size_t)b * a.kv.hq + g * G + qh) * D + grp * 8);
      const uint4 v = qp[4 * kk];
      qf[kk] = __builtin_bit_cast(bf16x8_t, col < G ? v : make_uint4(0, 0, 0, 0));
    }
    int gp = 1;
    while (gp < G) gp <<= 1;
    constexpr int kStride = 32 * (BLOCK / 64);
    const int t0 = wave * 32;
    const int iters = t0 < M ? (M - t0 + kStride - 1) / kStride : 0;
    if (iters > 0) {
      ScoreStep<D, 2> A, B;
      int t = t0;
      score_load<D, false>(A, a, rg, b, g, t, M, 0, nullptr, lane);
      int i = 0;
      for (; i + 2 < iters; i += 2) {
        score_load<D, false>(B, a, rg, b, g, t + kStride, M, 0, nullptr, lane);
        score_consume<D>(A, qf, G, gp, t, M, lane, s_keys, h, s_kst[wave]);
        score_load<D, false>(A, a, rg, b, g, t + 2 * kStride, M, 0, nullptr, lane);
        score_consume<D>(B, qf, G, gp, t + kStride, M, lane, s_keys, h, s_kst[wave]);
        t += 2 * kStride;
      }
      if (i + 1 < iters) {
        score_load<D, false>(B, a, rg, b, g, t + kStride, M, 0, nullptr, lane);
        score_consume<D>(A, qf, G, gp, t, M, lane, s_keys, h, s_kst[wave]);
        score_consume<D>(B, qf, G, gp, t + kStride, M, lane, s_keys, h, s_kst[wave]);
      } else {
        score_consume<D>(A, qf, G, gp, t, M, lane, s_keys, h, s_kst[wave]);
      }
    }
  }
  __syncthreads();
  // the staging tiles are free now: they hold the selection's scratch
  fused_select_tail<BLOCK>(a, row, rg, s_keys, h, (uint32_t*)&s_kst[0][0], scan64, s_res);
}

// Selection of one row whose middle-range keys a scoring kernel (without
// histograms) wrote to the workspace: the keys go to LDS with their level-0
// histogram, then the fused refresh's selection half.  Used when the rows
// fill at most half the CUs, so that scoring first spreads each row over
// many workgroups.  All of a thread's key loads are issued before any is
// stored.
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void select_keyed(SelArgs a) {
  constexpr int kPer = 16;  // keys per thread per batch
  extern __shared__ __attribute__((aligned(16))) uint32_t s_keys[];  // [middle length]
  __shared__ uint32_t h[kHistBins];
  __shared__ uint32_t h2[kTailScratchWords];
  __shared__ uint64_t scan64[BLOCK / 64 + 1];
  __shared__ uint32_t s_res[6];
  const int row = blockIdx.x;
  if (row_skipped(a, row)) return;
  const RowGeom rg = row_geom(a, row / a.kv.hkv);
  const int tid = threadIdx.x;
  for (int i = tid; i < kHistBins; i += BLOCK) h[i] = 0u;
  __syncthreads();
  if (rg.kb > 0) {
    const uint32_t* keys = a.keys + (size_t)row * a.mcap;
    for (int base = 0; base < rg.m; base += BLOCK * kPer) {
      uint32_t v[kPer];
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int i = base + tid + k * BLOCK;
        v[k] = i < rg.m ? keys[i] : 0u;
      }
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int i = base + tid + k * BLOCK;
        if (i < rg.m) {
          s_keys[i] = v[k];
          atomicAdd(&h[v[k] >> 21], 1u);
        }
      }
    }
  }
  __syncthreads();
  fused_select_tail<BLOCK>(a, row, rg, s_keys, h, h2, scan64, s_res);
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr int kLdsBytes = 160 * 1024;  // LDS of one CU

}  // namespace

// CUs of the current device (0 when unknown); also used by the prefill launch.
int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cus[dev] = n > 0 ? n : -1;
  }
  return cus[dev] > 0 ? cus[dev] : 0;
}

namespace {

enum class SelPath { kFused, kKeyed, kRadix };

// The refresh's launch sequence.  Middle ranges that fit LDS: one fused
// launch when the rows (one workgroup each) fill more than half the CUs and
// the cache is contiguous bf16, else scoring spread over many workgroups per
// row followed by one selection workgroup per row (keyed).  Longer middle
// ranges: the radix path (clear, score, filter, finish).
// PRHS_SELECT_PATH=fused|keyed|split forces a path where it applies.
SelPath select_path(int dtype, bool paged, int rows, int mcap) {
  static const int force = [] {
    const char* e = getenv("PRHS_SELECT_PATH");
    if (!e) return 0;
    if (e[0] == 'f') return 1;
    if (e[0] == 'k') return 2;
    if (e[0] == 's') return 3;
    return 0;
  }();
  const bool fits = mcap <= kFusedMaxKeys;
  const bool fused_ok = fits && dtype == 1 && !paged;
  if (force == 1 && fused_ok) return SelPath::kFused;
  if (force == 2 && fits) return SelPath::kKeyed;
  if (force == 3) return SelPath::kRadix;
  if (!fits) return SelPath::kRadix;
  const int cus = device_cus();
  if (fused_ok && (cus <= 0 || 2 * rows > cus)) return SelPath::kFused;
  return SelPath::kKeyed;
}

// CUs of the current device, for the fused refresh's row balancing (0 when
// unknown or when PRHS_SELECT_BALANCE=0).
int balance_cus() {
  static const int enabled = [] {
    const char* e = getenv("PRHS_SELECT_BALANCE");
    return e ? atoi(e) : 1;
  }();
  return enabled ? device_cus() : 0;
}

struct SelLayout {
  size_t keys, hist0, hist1, counters, sel, cand, cand2, total;
};

// The zero-between-calls region (histograms, counters) comes first, so a
// workspace keeps it in place for calls with fewer rows too.
SelLayout select_layout(int rows, int mcap, int selcap) {
  SelLayout L;
  size_t off = 0;
  L.hist0 = off;    off += align256((size_t)rows * kHistBins * 4);
  L.hist1 = off;    off += align256((size_t)rows * kHistBins * 4);
  L.counters = off; off += align256((size_t)rows * 16);
  L.keys = off;     off += align256((size_t)rows * mcap * 4);
  L.sel = off;      off += align256((size_t)rows * selcap * 8);
  L.cand = off;     off += align256((size_t)rows * mcap * 8);
  L.cand2 = off;    off += align256((size_t)rows * mcap * 8);
  L.total = off;
  return L;
}

}  // namespace

size_t select_workspace_bytes(int rows, int max_seq_len, int max_topk) {
  const int mcap = max_seq_len > 0 ? max_seq_len : 1;
  const int selcap = max_topk > 0 ? max_topk : 1;
  return select_layout(rows, mcap, selcap).total;
}

hipError_t launch_select(const SelectLaunch& s, hipStream_t stream) {
  const int rows = s.kv.batch * s.kv.hkv;
  if (rows == 0) return hipSuccess;
  SelArgs a;
  a.kv = s.kv;
  a.q = s.q;
  a.k = s.k;
  a.k_num = s.k_num;
  a.k_den = s.k_den;
  a.sink = s.sink;
  a.window = s.window;
  a.dilate_m = s.dilate_m;
  a.mcap = s.kv.max_seq_len > 0 ? s.kv.max_seq_len : 1;
  a.selcap = s.max_topk > 0 ? s.max_topk : 1;
  const SelLayout L = select_layout(rows, a.mcap, a.selcap);
  char* ws = (char*)s.ws;
  a.keys = (uint32_t*)(ws + L.keys);
  a.hist0 = (uint32_t*)(ws + L.hist0);
  a.hist1 = (uint32_t*)(ws + L.hist1);
  a.counters = (uint32_t*)(ws + L.counters);
  a.sel = (uint2*)(ws + L.sel);
  a.cand = (uint2*)(ws + L.cand);
  a.cand2 = (uint2*)(ws + L.cand2);
  a.topk_idx = s.topk_idx;
  a.topk_len = s.topk_len;
  a.k_cap = s.k_cap;
  a.set_idx = s.set_idx;
  a.set_len = s.set_len;
  a.set_cap = s.set_cap;
  a.dilate_r = s.dilate_r;
  a.shared_idx = s.shared_idx;
  a.shared_len = s.shared_len;
  a.balance_cus = 0;
  a.balance_serpentine = 0;
  a.seg_bits = kFinishSegBits;
  a.seg_shift = 0;
  a.row_choice = s.row_choice;
  a.gate_fused = 0;

  const SelPath path = select_path(s.dtype, s.kv.paged != 0, rows, a.mcap);
  if (s.gate) {
    if (path == SelPath::kFused) {
      a.gate_fused = 1;   // the gate runs inside the refresh launch
      a.gate = *s.gate;
    } else {
      // a launch of its own, then the path's kernels on the retrieving rows
      const hipError_t e = launch_gate(*s.gate, stream);
      if (e != hipSuccess) return e;
      a.row_choice = s.gate->choice;
    }
  }
  // many short contiguous bf16 rows: the whole refresh in one launch
  if (path == SelPath::kFused) {
    const size_t dyn = (size_t)a.mcap * 4;
    a.balance_cus = balance_cus();
    // 1024-thread workgroups (one per CU) when the rows fit the CUs, or when
    // two 512-thread ones would not fit one CU's LDS either (long middle
    // ranges: more waves stream each row); otherwise 512-thread workgroups,
    // two to a CU, so that one's selection overlaps the other's scoring.
    // Either way only while the workgroup's LDS (static part plus the key
    // array) fits the CU's 160 KB.
    bool wide = a.balance_cus <= 0 || rows <= a.balance_cus;
    if (!wide) {
      hipFuncAttributes fb;
      const hipError_t eb =
          s.kv.d == 128 ? hipFuncGetAttributes(&fb, (const void*)select_fused<128, 512>)
                        : hipFuncGetAttributes(&fb, (const void*)select_fused<64, 512>);
      if (eb != hipSuccess) return eb;
      wide = 2 * (fb.sharedSizeBytes + dyn) > (size_t)kLdsBytes;
    }
    if (wide) {
      hipFuncAttributes fa;
      const hipError_t ea =
          s.kv.d == 128 ? hipFuncGetAttributes(&fa, (const void*)select_fused<128, 1024>)
                        : hipFuncGetAttributes(&fa, (const void*)select_fused<64, 1024>);
      if (ea != hipSuccess) return ea;
      wide = fa.sharedSizeBytes + dyn <= (size_t)kLdsBytes;
    }
    a.balance_serpentine = wide ? 0 : 1;
    hipError_t e = hipSuccess;
#define PRHS_FUSED_LAUNCH(DV, BL)                                                           \
  {                                                                                         \
    if (dyn > 65536)                                                                        \
      e = hipFuncSetAttribute((const void*)select_fused<DV, BL>,                             \
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);        \
    if (e == hipSuccess)                                                                    \
      hipLaunchKernelGGL((select_fused<DV, BL>), dim3(rows), dim3(BL), dyn, stream, a);     \
  }
    if (s.kv.d == 128) {
      if (wide) PRHS_FUSED_LAUNCH(128, 1024) else PRHS_FUSED_LAUNCH(128, 512)
    } else {
      if (wide) PRHS_FUSED_LAUNCH(64, 1024) else PRHS_FUSED_LAUNCH(64, 512)
    }
#undef PRHS_FUSED_LAUNCH
    return e != hipSuccess ? e : hipGetLastError();
  }
  // the middle range is shorter than max_seq_len; size grids by max_seq_len
  const int mid_max = a.mcap;
  const bool radix = path == SelPath::kRadix;
  const dim3 sgrid((mid_max + kScoreChunk - 1) / kScoreChunk, rows);
#define PRHS_SCORE_LAUNCH(HIST)                                                               \
  if (s.dtype == 1) {                                                                         \
    const bool paged = s.kv.paged != 0;                                                       \
    if (s.kv.d == 128) {                                                                      \
      if (paged) hipLaunchKernelGGL((score_bf16<128, true, HIST>), sgrid, dim3(kScoreBlock), 0, stream, a);  \
      else hipLaunchKernelGGL((score_bf16<128, false, HIST>), sgrid, dim3(kScoreBlock), 0, stream, a);       \
    } else {                                                                                  \
      if (paged) hipLaunchKernelGGL((score_bf16<64, true, HIST>), sgrid, dim3(kScoreBlock), 0, stream, a);   \
      else hipLaunchKernelGGL((score_bf16<64, false, HIST>), sgrid, dim3(kScoreBlock), 0, stream, a);        \
    }                                                                                         \
  } else {                                                                                    \
    if (s.kv.d == 128) hipLaunchKernelGGL((score_f32<128, HIST>), sgrid, dim3(kScoreBlock), 0, stream, a);   \
    else hipLaunchKernelGGL((score_f32<64, HIST>), sgrid, dim3(kScoreBlock), 0, stream, a);                  \
  }
  if (radix) {
    PRHS_SCORE_LAUNCH(true)
  } else {
    PRHS_SCORE_LAUNCH(false)
  }
#undef PRHS_SCORE_LAUNCH
  if (!radix) {
    // keyed: one 1024-thread selection workgroup per row over the keys in LDS
    const size_t dyn = (size_t)a.mcap * 4;
    if (dyn > 65536) {
      const hipError_t e = hipFuncSetAttribute((const void*)select_keyed<1024>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(select_keyed<1024>, dim3(rows), dim3(1024), dyn, stream, a);
    return hipGetLastError();
  }
  const dim3 fgrid((mid_max + kFilterChunk - 1) / kFilterChunk, rows);
  hipLaunchKernelGGL(select_filter, fgrid, dim3(kFilterBlock), 0, stream, a);
  // LDS buffer: the k winners plus up to kFinishTies level-1 ties, as far as
  // the CU's LDS holds them beside the kernel's static LDS and the bitmap
  // segment (the host bound PRHS_MAX_TOPK keeps the winners alone inside
  // it); the output staging takes what remains, up to kFinishStage entries
  static const long long finish_static = [] {
    hipFuncAttributes fa;
    return hipFuncGetAttributes(&fa, (const void*)select_finish) == hipSuccess
               ? (long long)fa.sharedSizeBytes : -1LL;
  }();
  if (finish_static < 0) return hipErrorInvalidDeviceFunction;
  // LDS plan for segments of seg_bits positions with nbm bitmaps each
  struct FinishPlan {
    int sortcap, woff, stagecap;
    size_t dyn;
  };
  // (seg_bits a multiple of 128: bitmaps of whole 16-byte groups of words)
  auto plan = [&](long long seg_bits, long long nbm, FinishPlan* fp) {
    // the bitmaps start 16-byte aligned after the sort buffer (one entry of
    // padding when sortcap is odd) and end with 16 bytes of slack; 16 bytes
    // more cover the dynamic buffer's alignment after the static LDS
    const long long bm_bytes = nbm * seg_bits / 8 + 16;
    const long long avail = (long long)kLdsBytes - finish_static - 16 - bm_bytes - 8;
    long long cap = (long long)a.selcap + kFinishTies;
    if (cap > avail / 8) cap = avail / 8;
    if (cap < a.selcap) return false;
    long long rest = avail - cap * 8;
    const long long woff_bytes = seg_bits / 32 * 8;
    fp->sortcap = (int)cap;
    fp->woff = rest >= woff_bytes ? 1 : 0;
    if (fp->woff) rest -= woff_bytes;
    fp->stagecap = (int)(rest / 4 < kFinishStage ? rest / 4 : kFinishStage);
    fp->dyn = (size_t)(((cap + 1) & ~1LL) * 8 + bm_bytes + (fp->woff ? woff_bytes : 0) +
                       (long long)fp->stagecap * 4);
    return true;
  };
  // the whole middle range as one segment when its outputs keep the packed
  // counts below 2^16 (at most max_topk winners, each with at most 2r
  // neighbours), the radius is below a word (the neighbours then come from
  // shifts of the top-m bitmap, two bitmaps instead of three) and the full
  // tie buffer and the per-word offsets still fit LDS
  FinishPlan fp{};
  const long long one_bits = ((long long)a.mcap + 127) / 128 * 128;
  bool one = s.dilate_r < 32 && (long long)a.selcap * (2LL * s.dilate_r + 1) < 65536 &&
             plan(one_bits, 2, &fp) && fp.sortcap == a.selcap + kFinishTies && fp.woff;
  if (one) {
    a.seg_bits = (int)one_bits;
    a.seg_shift = 1;
  } else {
    if (!plan(kFinishSegBits, 3, &fp)) return hipErrorInvalidValue;  // unreachable for k_b <= PRHS_MAX_TOPK
    a.seg_bits = kFinishSegBits;
    a.seg_shift = 0;
  }
  a.sortcap = fp.sortcap;
  a.woff = fp.woff;
  a.stagecap = fp.stagecap;
  const size_t dyn = fp.dyn;
  if (dyn > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)select_finish,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_finish, dim3(rows), dim3(kFinishBlock), dyn, stream, a);
  return hipGetLastError();
}

}  // namespace prhs

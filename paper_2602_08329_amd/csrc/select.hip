// Refresh-step selection for one layer: ranking scores over the middle range,
// exact top-k by multi-level radix select, ordering by (score desc, position
// asc), and the critical set sink U top-k U window (Sec. 4.1 Selection
// Criteria; top-k oracle of Sec. 3.3).
//
// Pipeline (one launch each, all on the caller's stream):
//   select_clear   zero the per-row histograms and counters
//   score_*        sigma_i = max_h q_h . k_i (raw, fp32) -> order-preserving
//                  u32 key; fused histogram of the top 11 key bits
//   select_filter  locate the threshold bin of level 0; keys above it are
//                  selected, keys in it become candidates (with the level-1
//                  histogram fused)
//   select_finish  remaining radix levels over the candidates, the 64-bit
//                  composite (key, kIdxMax - pos) making every key distinct so
//                  ties go to the lower position; bitonic sort of the k
//                  winners in LDS; ordered compaction of the anchor set.
#include "prhs_internal.h"
#include "setops.cuh"

namespace prhs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kScoreBlock = 256;
constexpr int kScoreChunk = 1024;   // keys per score workgroup
constexpr int kFilterBlock = 256;
constexpr int kFilterChunk = 4096;  // keys per filter workgroup
constexpr int kFinishBlock = 1024;

struct SelArgs {
  KvView kv;
  const void* q;
  int k, k_num, k_den, sink, window;
  int mcap, selcap;
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
};

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
  __syncthreads();
}

__global__ __launch_bounds__(256) void select_clear(SelArgs a) {
  const int row = blockIdx.x;
  for (int i = threadIdx.x; i < kHistBins; i += 256) {
    a.hist0[(size_t)row * kHistBins + i] = 0u;
    a.hist1[(size_t)row * kHistBins + i] = 0u;
  }
  if (threadIdx.x < 4) a.counters[row * 4 + threadIdx.x] = 0u;
}

__device__ __forceinline__ void flush_hist(const uint32_t* h, uint32_t* dst) {
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
    const uint32_t c = h[i];
    if (c) atomicAdd(&dst[i], c);
  }
}

// bf16 scoring on MFMA: per 16 keys, S[key][head] = K_tile(16 x d) . Q^T(d x 16)
// with the group's g <= 16 query heads in the columns (unused columns zero).
// Lane l loads d/2 contiguous bytes of key l%16; the contraction runs over a
// permutation of d shared by both operands.  Products of bf16 values are exact
// in fp32 and the accumulation is fp32.
template <int D>
__global__ __launch_bounds__(kScoreBlock) void score_bf16(SelArgs a) {
  constexpr int KS = D / 32;  // MFMA k-steps
  constexpr int SUB = 4;      // 16-key sub-tiles per wave iteration
  __shared__ uint32_t hist[kHistBins];
  const int row = blockIdx.y;
  const int b = row / a.kv.hkv, g = row % a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  const int base = blockIdx.x * kScoreChunk;
  if (base >= rg.m || rg.kb <= 0) return;
  const int end = min(rg.m, base + kScoreChunk);
  for (int i = threadIdx.x; i < kHistBins; i += kScoreBlock) hist[i] = 0u;
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int G = a.kv.hq / a.kv.hkv;
  const __bf16* q = (const __bf16*)a.q;
  const __bf16* kbase = (const __bf16*)a.kv.k;
  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    if (col < G) {
      const uint4* qp = (const uint4*)(q + ((size_t)b * a.kv.hq + g * G + col) * D + grp * (D / 4));
      qf[kk] = __builtin_bit_cast(bf16x8_t, qp[kk]);
    } else {
      qf[kk] = __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
    }
  }
  int gp = 1;
  while (gp < G) gp <<= 1;

  uint32_t* keys = a.keys + (size_t)row * a.mcap;
  for (int t = base + wave * 16 * SUB; t < end; t += 4 * 16 * SUB) {
    bf16x8_t kf[SUB][KS];
#pragma unroll
    for (int s = 0; s < SUB; ++s) {
      const int i = t + s * 16 + col;
      int64_t off = -1;
      if (i < end) off = kv_row_offset(a.kv, b, g, rg.sink_end + i);
      const uint4* kp = (const uint4*)(kbase + (off < 0 ? 0 : off) + grp * (D / 4));
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        kf[s][kk] = __builtin_bit_cast(bf16x8_t, off < 0 ? make_uint4(0, 0, 0, 0) : kp[kk]);
    }
#pragma unroll
    for (int s = 0; s < SUB; ++s) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s][kk], qf[kk], acc, 0, 0, 0);
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = col < G ? acc[e] : -INFINITY;
      for (int off = 1; off < gp; off <<= 1) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = fmaxf(v[e], __shfl_xor(v[e], off, 16));
      }
      if (col == 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = t + s * 16 + grp * 4 + e;
          if (i < end) {
            const uint32_t key = score_key(v[e]);
            keys[i] = key;
            atomicAdd(&hist[key >> 21], 1u);
          }
        }
      }
    }
  }
  __syncthreads();
  flush_hist(hist, a.hist0 + (size_t)row * kHistBins);
}

// fp32 scoring on the vector ALU: one key per thread, the group's query heads
// staged in LDS, sequential fp32 fused multiply-adds over d.
template <int D>
__global__ __launch_bounds__(kScoreBlock) void score_f32(SelArgs a) {
  __shared__ uint32_t hist[kHistBins];
  __shared__ float qs[16 * D];
  const int row = blockIdx.y;
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
    atomicAdd(&hist[key >> 21], 1u);
  }
  __syncthreads();
  flush_hist(hist, a.hist0 + (size_t)row * kHistBins);
}

__global__ __launch_bounds__(kFilterBlock) void select_filter(SelArgs a) {
  __shared__ uint32_t h[kHistBins];
  __shared__ uint32_t scan[kFilterBlock / 64 + 1];
  __shared__ int s_bin;
  __shared__ uint32_t s_krem, s_cnt;
  const int row = blockIdx.y;
  const int b = row / a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  const int base = blockIdx.x * kFilterChunk;
  if (base >= rg.m || rg.kb <= 0) return;
  const int end = min(rg.m, base + kFilterChunk);
  const bool all = rg.kb >= rg.m;
  int bin = 0;
  bool resolved = true;
  if (!all) {
    for (int i = threadIdx.x; i < kHistBins; i += kFilterBlock) h[i] = a.hist0[(size_t)row * kHistBins + i];
    __syncthreads();
    find_threshold<kFilterBlock>(h, (uint32_t)rg.kb, scan, &s_bin, &s_krem, &s_cnt);
    bin = s_bin;
    resolved = (s_cnt == s_krem);
    __syncthreads();
    for (int i = threadIdx.x; i < kHistBins; i += kFilterBlock) h[i] = 0u;
    __syncthreads();
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t* keys = a.keys + (size_t)row * a.mcap;
  uint32_t* cnt = a.counters + row * 4;
  uint2* sel = a.sel + (size_t)row * a.selcap;
  uint2* cand = a.cand + (size_t)row * a.mcap;
  for (int i0 = base + wave * 64; i0 < end; i0 += kFilterBlock) {
    const int i = i0 + lane;
    const bool valid = i < end;
    uint2 e = make_uint2(0u, 0u);
    bool take = false, keep = false;
    if (valid) {
      e = make_uint2(keys[i], (uint32_t)(rg.sink_end + i));
      if (all) {
        take = true;
      } else {
        const int d0 = (int)(e.x >> 21);
        take = d0 > bin || (resolved && d0 == bin);
        keep = !resolved && d0 == bin;
      }
    }
    const int slot = wave_append(take, &cnt[0]);
    if (slot >= 0 && slot < a.selcap) sel[slot] = e;
    const int slot2 = wave_append(keep, &cnt[1]);
    if (slot2 >= 0 && slot2 < a.mcap) {
      cand[slot2] = e;
      atomicAdd(&h[(e.x >> 10) & 0x7FFu], 1u);
    }
  }
  if (!all && !resolved) {
    __syncthreads();
    flush_hist(h, a.hist1 + (size_t)row * kHistBins);
  }
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

__global__ __launch_bounds__(kFinishBlock) void select_finish(SelArgs a) {
  extern __shared__ uint64_t dyn[];
  __shared__ uint32_t h[kHistBins];
  __shared__ uint32_t scan[kFinishBlock / 64 + 1];
  __shared__ int s_bin;
  __shared__ uint32_t s_krem, s_cnt, s_dst;
  const int row = blockIdx.x;
  const int b = row / a.kv.hkv;
  const RowGeom rg = row_geom(a, b);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t* cnt = a.counters + row * 4;
  uint2* sel = a.sel + (size_t)row * a.selcap;

  if (rg.kb > 0 && rg.kb < rg.m) {
    for (int i = tid; i < kHistBins; i += kFinishBlock) h[i] = a.hist0[(size_t)row * kHistBins + i];
    __syncthreads();
    find_threshold<kFinishBlock>(h, (uint32_t)rg.kb, scan, &s_bin, &s_krem, &s_cnt);
    if (s_cnt != s_krem) {
      uint2* src = a.cand + (size_t)row * a.mcap;
      uint2* dst = a.cand2 + (size_t)row * a.mcap;
      uint32_t count = min(coherent_load(&cnt[1]), (uint32_t)a.mcap);
      uint32_t krem = s_krem;
      for (int level = 1; level <= 4; ++level) {
        __syncthreads();
        if (level == 1) {
          for (int i = tid; i < kHistBins; i += kFinishBlock) h[i] = a.hist1[(size_t)row * kHistBins + i];
        } else {
          for (int i = tid; i < kHistBins; i += kFinishBlock) h[i] = 0u;
          __syncthreads();
          for (uint32_t e = tid; e < count; e += kFinishBlock) atomicAdd(&h[level_digit(src[e], level)], 1u);
        }
        if (tid == 0) s_dst = 0u;
        __syncthreads();
        find_threshold<kFinishBlock>(h, krem, scan, &s_bin, &s_krem, &s_cnt);
        const uint32_t bl = (uint32_t)s_bin;
        const bool resolved = s_cnt == s_krem;
        for (uint32_t e0 = wave * 64; e0 < count; e0 += kFinishBlock) {
          const uint32_t e = e0 + lane;
          const bool valid = e < count;
          const uint2 x = valid ? src[e] : make_uint2(0u, 0u);
          const uint32_t dg = level_digit(x, level);
          const bool take = valid && (dg > bl || (resolved && dg == bl));
          const bool keep = valid && !resolved && dg == bl;
          const int slot = wave_append(take, &cnt[0]);
          if (slot >= 0 && slot < a.selcap) sel[slot] = x;
          const int slot2 = wave_append(keep, &s_dst);
          if (slot2 >= 0 && slot2 < a.mcap) dst[slot2] = x;
        }
        block_publish();
        if (resolved) break;
        count = s_dst;
        krem = s_krem;
        uint2* tmp = src;
        src = dst;
        dst = tmp;
      }
    }
  }
  block_publish();

  uint32_t total = 0;
  if (rg.kb > 0) total = min(coherent_load(&cnt[0]), (uint32_t)min(rg.kb, a.selcap));
  uint32_t P = 1;
  while (P < total) P <<= 1;
  for (uint32_t i = tid; i < P; i += kFinishBlock) {
    uint64_t c = 0;
    if (i < total) {
      const uint2 e = sel[i];
      c = ((uint64_t)e.x << 32) | (uint64_t)(kIdxMax - e.y);
    }
    dyn[i] = c;
  }
  __syncthreads();
  // bitonic sort, descending by the composite key
  for (uint32_t kk = 2; kk <= P; kk <<= 1) {
    for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
      for (uint32_t i = tid; i < P; i += kFinishBlock) {
        const uint32_t ixj = i ^ j;
        if (ixj > i) {
          const uint64_t x = dyn[i], y = dyn[ixj];
          const bool desc = (i & kk) == 0;
          if (desc ? (x < y) : (x > y)) {
            dyn[i] = y;
            dyn[ixj] = x;
          }
        }
      }
      __syncthreads();
    }
  }
  int32_t* topk = a.topk_idx + (size_t)row * a.k_cap;
  for (uint32_t i = tid; i < total; i += kFinishBlock)
    topk[i] = (int32_t)(kIdxMax - (uint32_t)(dyn[i] & 0xFFFFFFFFull));
  if (tid == 0) a.topk_len[row] = (int32_t)total;
  block_publish();
  build_index_set<kFinishBlock>(topk, (int)total, 0, 0, rg.sink_end, rg.win_start, rg.n0,
                                a.set_idx + (size_t)row * a.set_cap, a.set_cap, a.set_len + row,
                                (uint32_t*)dyn, scan);
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct SelLayout {
  size_t keys, hist0, hist1, counters, sel, cand, cand2, total;
};

SelLayout select_layout(int rows, int mcap, int selcap) {
  SelLayout L;
  size_t off = 0;
  L.keys = off;     off += align256((size_t)rows * mcap * 4);
  L.hist0 = off;    off += align256((size_t)rows * kHistBins * 4);
  L.hist1 = off;    off += align256((size_t)rows * kHistBins * 4);
  L.counters = off; off += align256((size_t)rows * 16);
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

  // the middle range is shorter than max_seq_len; size grids by max_seq_len
  const int mid_max = a.mcap;
  hipLaunchKernelGGL(select_clear, dim3(rows), dim3(256), 0, stream, a);
  const dim3 sgrid((mid_max + kScoreChunk - 1) / kScoreChunk, rows);
  if (s.dtype == 1) {
    if (s.kv.d == 128) hipLaunchKernelGGL(score_bf16<128>, sgrid, dim3(kScoreBlock), 0, stream, a);
    else hipLaunchKernelGGL(score_bf16<64>, sgrid, dim3(kScoreBlock), 0, stream, a);
  } else {
    if (s.kv.d == 128) hipLaunchKernelGGL(score_f32<128>, sgrid, dim3(kScoreBlock), 0, stream, a);
    else hipLaunchKernelGGL(score_f32<64>, sgrid, dim3(kScoreBlock), 0, stream, a);
  }
  const dim3 fgrid((mid_max + kFilterChunk - 1) / kFilterChunk, rows);
  hipLaunchKernelGGL(select_filter, fgrid, dim3(kFilterBlock), 0, stream, a);
  uint32_t P = 1;
  while ((int)P < a.selcap) P <<= 1;
  size_t dyn = (size_t)P * 8;
  if (dyn < (size_t)kSegWords * 4) dyn = (size_t)kSegWords * 4;
  if (dyn > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)select_finish,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(select_finish, dim3(rows), dim3(kFinishBlock), dyn, stream, a);
  return hipGetLastError();
}

}  // namespace prhs

// Decode attention over a per-kv-head index set (token-sparse attention,
// Def. 3.1) or over every cached key (Eq. attn_eq), split-K:
//
// attn_split_*: one workgroup per (unit, split) handles a contiguous chunk of
// the unit's index list: it gathers K/V rows, computes scaled logits and keeps
// an online softmax (running max m, running sum l, unnormalised output o).  A
// unit that fits one split writes its output directly; otherwise each split
// stores (m, l, o) and
// attn_merge: one workgroup per query head of a split unit combines them in
// split order,
//   y = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s,
//   lse = ln 2 * (M + log2 sum_s 2^(m_s - M) l_s).
// The merge is a launch of its own: merging inside the split kernel would need
// device-scope fences, which on this chip write back and invalidate a whole
// L2 slice per workgroup.
//
// Latency: the workgroup first resolves every list entry of its chunk to a
// physical row id (the set entries load together with the unit's lengths,
// then block-table loads for paged caches) and stages the ids in LDS.  Waves
// then walk 32-row tiles with two register buffers: the K/V loads of the next
// tile are in flight while the current tile is multiplied.  Loads are issued
// unconditionally (a missing row reads row 0) and invalid rows are masked
// afterwards, so no load waits on a branch.
//
// bf16 inputs use MFMA for both products of a wave's 32-row tile:
//   S^T (32 keys x 16 heads) = K_tile . Q^T  (v_mfma_f32_16x16x32_bf16, two 16-row halves)
//   O^T (d x 16 heads)      += V_tile^T . P^T, P split into bf16 hi + lo parts so
//                              the probabilities keep ~16 significant bits.
// Every K and V load reads whole rows (d/8 lanes of 16 bytes per row), the
// pattern that sustains full bandwidth per CU; the MFMA operand order of K
// (4 lanes per key) would read 64-byte pieces of 16 rows per load, which
// this chip serves at well under half that rate.  K therefore goes through
// a per-wave LDS tile (XOR-swizzled, conflict-free both ways) into operand
// order; the dimension order inside a row is permuted identically on K and
// Q.  V needs no transpose: a lane's 8 rows x 8 dims block feeds the second
// product directly.  K and V bytes are read once, with the streaming policy.
// fp32 inputs take a vector-ALU path (16 lanes per row, one query head per
// workgroup).
#include <stdlib.h>

#include <mutex>

#include "prhs_internal.h"

namespace prhs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kRowsPerThread = 8;   // staged list entries per thread
constexpr int kMaxSplits = 4096;
// Sparse sets of at most this many rows per unit are not split: a launch of
// one workgroup per unit beats a split launch plus its merge launch.
constexpr int kNoSplitRows = 512;

struct AttnArgs {
  KvView kv;
  const void* q;
  const int32_t* set_idx;
  const int32_t* set_len;
  const int32_t* tail_start;  // [B] or null: rows also cover [tail_start[b], n_b)
  const int32_t* unit_row;    // [units] or null: pool row of set_idx each unit attends
  const int32_t* unit_tail;   // [units] with unit_row: first position of the unit's tail
  int pool_rows;
  const int32_t* unit_gate;   // [units] or null: the gate's choice per unit
  int units_side;             // 1: only units with unit_gate < 0; 2: only >= 0; else all
  int psaw;                   // nonzero: positions in [psaw_sink, first visible) are skipped
  double psaw_f;              // Eq. psaw factor of the layer (first visible at length n:
  int psaw_sink;              // psaw_first_visible(psaw_f, psaw_sink, n))
  int set_cap;
  float scale_log2;
  int chunk, nsplit;
  float* part_o;    // [B*Hq][nsplit][D]
  float* part_ml;   // [B*Hq][nsplit][2]
  float* out;
  float* lse;
};

// The rows a unit attends, in order: the first `base` come from its index
// set (entries at or beyond t0 are skipped), then the tail positions
// [t0, t0 + L - base).  Dense: rows are the positions [0, n_b).  Without a
// tail t0 = n_b.  L never exceeds set_cap, the bound the split geometry uses.
// The set is row u of set_idx, or with a pool the row unit_row[u] (a row
// outside the pool gives an empty set) and the tail from unit_tail[u].
struct UnitSpan {
  int L, base, t0;
  int mask_lo, mask_hi;  // rows at positions in [mask_lo, mask_hi) are skipped (PSAW)
};

template <bool DENSE>
__device__ __forceinline__ UnitSpan unit_span(const AttnArgs& a, int u, int b, int nb) {
  UnitSpan sp;
  sp.t0 = nb;
  sp.mask_lo = sp.mask_hi = 0;
  if (DENSE) {
    sp.L = sp.base = nb;
    return sp;
  }
  if (a.psaw) {
    sp.mask_lo = a.psaw_sink;
    sp.mask_hi = psaw_first_visible(a.psaw_f, a.psaw_sink, nb);
  }
  int row = u, t0 = nb;
  bool tail = false;
  if (a.unit_row) {
    row = a.unit_row[u];
    t0 = a.unit_tail[u];
    tail = true;
    if (row < 0 || row >= a.pool_rows) {
      sp.L = sp.base = 0;
      return sp;
    }
  } else if (a.tail_start) {
    t0 = a.tail_start[b];
    tail = true;
  }
  int L = a.set_len[row];
  L = L < 0 ? 0 : (L > a.set_cap ? a.set_cap : L);
  sp.base = L;
  if (tail) {
    t0 = t0 < 0 ? 0 : (t0 > nb ? nb : t0);
    sp.t0 = t0;
    L += nb - t0;
    L = L > a.set_cap ? a.set_cap : L;
  }
  sp.L = L;
  return sp;
}

// Units a launch leaves alone (their outputs untouched): with a side filter,
// the ones on the other side of the gate's decision.
__device__ __forceinline__ bool unit_excluded(const AttnArgs& a, int u) {
  if (!a.unit_gate || (a.units_side != 1 && a.units_side != 2)) return false;
  const bool retrieving = a.unit_gate[u] < 0;
  return a.units_side == 1 ? !retrieving : retrieving;
}

// Row id (element offset / d) of position pos of (b, kv head g), or -1 when
// the position lies outside [0, nb) or outside the cache.
template <bool PAGED>
__device__ __forceinline__ int32_t phys_row(const KvView& kv, int b, int g, int pos, int nb) {
  if (pos < 0 || pos >= nb) return -1;
  if (!PAGED) {
    if (pos >= kv.capacity) return -1;
    return (b * kv.hkv + g) * kv.capacity + pos;
  }
  const int page = pos / kv.page_size;
  if (page >= kv.max_pages) return -1;
  const int phys = kv.table[(int64_t)b * kv.max_pages + page];
  if (phys < 0 || phys >= kv.num_pages) return -1;
  return (phys * kv.hkv + g) * kv.page_size + (pos - page * kv.page_size);
}

// Loads the set entries [start, start + chunk) of unit u before the unit's
// length is known, so that these loads share one memory latency with the
// length loads.  Entries at or past the length are loaded and never used; a
// set row holds set_cap entries, so every load stays inside it.
template <bool DENSE>
__device__ __forceinline__ void prefetch_entries(const AttnArgs& a, int u, int start,
                                                 int32_t (&raw)[kRowsPerThread]) {
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) raw[k] = -1;
  if (DENSE) return;
  int row = u;
  bool ok = true;
  if (a.unit_row) {
    row = a.unit_row[u];
    ok = row >= 0 && row < a.pool_rows;
  }
  const int32_t* idx = a.set_idx + (size_t)(ok ? row : 0) * a.set_cap;
  const int lim = min(start + a.chunk, a.set_cap);
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int t = start + (int)threadIdx.x + k * (int)blockDim.x;
    if (ok && t < lim) raw[k] = idx[t];
  }
}

// Resolves list entries [start, start + n) of the unit to row ids in s_row,
// from the entries prefetch_entries loaded; for a paged cache all block-table
// loads of a thread are issued before any is used.  n <= blockDim * 8.
template <bool DENSE, bool PAGED>
__device__ __forceinline__ void stage_rows(const AttnArgs& a, const int32_t (&raw)[kRowsPerThread],
                                           int start, int n, const UnitSpan& sp, int nb, int b,
                                           int g, int32_t* s_row) {
  int pos[kRowsPerThread];
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int r = threadIdx.x + k * blockDim.x;
    const int t = start + r;
    pos[k] = -1;
    if (r < n) {
      if (DENSE) {
        pos[k] = t;
      } else {
        int p;
        if (t < sp.base) {
          p = raw[k];
          p = p < sp.t0 ? p : -1;
        } else {
          p = sp.t0 + (t - sp.base);
        }
        pos[k] = (p >= sp.mask_lo && p < sp.mask_hi) ? -1 : p;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int r = threadIdx.x + k * blockDim.x;
    if (r < n) s_row[r] = phys_row<PAGED>(a.kv, b, g, pos[k], nb);
  }
  __syncthreads();
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Maximum over the lanes col, col + 16, col + 32 and col + 48 (the four
// lane groups of one MFMA column), by the cross-half and cross-row lane
// swaps: each swap of a value with itself leaves a lane holding its own
// value and its partner's, one in each result.
__device__ __forceinline__ float max_over_groups(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Maximum over all 64 lanes, in every lane: rotations by 8, 4, 2 and 1
// inside each row of 16 lanes (DPP row_ror), then across the four rows.
__device__ __forceinline__ float wave_max(float v) {
#define PRHS_ROR_MAX(CTRL)                                                                    \
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), \
                                                          CTRL, 0xF, 0xF, false)))
  PRHS_ROR_MAX(0x128);  // row_ror:8
  PRHS_ROR_MAX(0x124);  // row_ror:4
  PRHS_ROR_MAX(0x122);  // row_ror:2
  PRHS_ROR_MAX(0x121);  // row_ror:1
#undef PRHS_ROR_MAX
  return max_over_groups(v);
}

// Sum over the same four lanes.
__device__ __forceinline__ float sum_over_groups(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <int DB>
struct VRow;
template <>
struct VRow<8> {  // d = 128: 8 bf16 per lane per row
  uint32_t w[4];
};
template <>
struct VRow<4> {  // d = 64: 4 bf16 per lane per row
  uint32_t w[2];
};

template <int DB>
__device__ __forceinline__ VRow<DB> load_vrow(const __bf16* p) {
  VRow<DB> v;
  if constexpr (DB == 8) {
    const u32x4_t x = stream_load16(p);
    v.w[0] = x[0]; v.w[1] = x[1]; v.w[2] = x[2]; v.w[3] = x[3];
  } else {
    const u32x2_t x = stream_load8(p);
    v.w[0] = x[0]; v.w[1] = x[1];
  }
  return v;
}


// Registers of one wave's 32-row tile: K rows as loaded (whole rows, D/8
// lanes of 16 bytes per row, so every load reads whole 128-byte lines), V
// rows (16s + 4 grp + j) and the validity of the V rows, which are also the
// rows of the lane's logits.
template <int D>
struct Tile {
  static constexpr int KS = D / 32;  // products per 16-row half = K loads per half
  static constexpr int DB = D / 16;
  u32x4_t kraw[2][KS];
  VRow<DB> vf[2][4];
  uint32_t ok;
};

// K staging in LDS: a wave's 32 x D tile, row-major in 16-byte chunks, chunk
// c of tile row r at slot c ^ (r mod D/8), so that both the row-wise writes
// and the MFMA-order reads (16 rows, one chunk each) hit distinct banks.
template <int D>
__device__ __forceinline__ int kst_slot(int r, int c) {
  constexpr int CH = D / 8;
  return r * CH + (c ^ (r & (CH - 1)));
}

// LDS bytes per wave: its K staging tile, reused at the end for its G output
// rows of D + 1 floats.
__host__ __device__ constexpr int attn_wave_bytes(int D, int G) {
  return ((32 * D * 2 > G * (D + 1) * 4 ? 32 * D * 2 : G * (D + 1) * 4) + 15) & ~15;
}

template <int D>
__device__ __forceinline__ void load_tile(Tile<D>& T, const int32_t* s_row, int r0, int n,
                                          const __bf16* kb, const __bf16* vb, int lane) {
  constexpr int KS = D / 32;
  constexpr int DB = D / 16;
  constexpr int CH = D / 8, RPI = 64 / CH;  // chunks per row, rows per K load
  const int col = lane & 15, grp = lane >> 4;
  const int kc = lane % CH, kr = lane / CH;
  // all row ids of the tile first (unconditional LDS reads: s_row spans whole
  // tiles), then every load, so that no load waits on a single LDS read
  int rk[2][KS], rv[2][4];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      const int r = r0 + 16 * s + j * RPI + kr;
      const int x = s_row[r];
      rk[s][j] = r < n ? x : -1;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = r0 + 16 * s + grp * 4 + j;
      const int x = s_row[r];
      rv[s][j] = r < n ? x : -1;
    }
  }
  T.ok = 0u;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int j = 0; j < KS; ++j)
      T.kraw[s][j] = stream_load16(kb + (int64_t)(rk[s][j] < 0 ? 0 : rk[s][j]) * D + kc * 8);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      T.vf[s][j] = load_vrow<DB>(vb + (int64_t)(rv[s][j] < 0 ? 0 : rv[s][j]) * D + col * DB);
      if (rv[s][j] >= 0) T.ok |= 1u << (s * 4 + j);
    }
  }
}

// Online-softmax state of one wave: lane (col, grp) owns query head col and
// output dims grp * d/4 .. (grp + 1) * d/4 - 1 via the o[] accumulators.
template <int D>
struct WaveState {
  float m, l;
  f32x4_t o[D / 16];
};

template <int D>
__device__ __forceinline__ void consume_tile(Tile<D>& T, WaveState<D>& st, const bf16x8_t* qf,
                                             float scale_log2, u32x4_t* kst, int lane) {
  constexpr int KS = D / 32;
  constexpr int DB = D / 16;
  constexpr int CH = D / 8, RPI = 64 / CH;
  const int col = lane & 15, grp = lane >> 4;
  // K rows to MFMA operand order through the wave's LDS tile: lane (col,
  // grp) takes dims 32kk + 8grp .. +7 of tile row 16s + col for product kk.
  // LDS operations of one wave complete in order; the wave barriers keep
  // the compiler from moving them across each other.
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int j = 0; j < KS; ++j) kst[kst_slot<D>(16 * s + j * RPI + lane / CH, lane % CH)] = T.kraw[s][j];
  __builtin_amdgcn_wave_barrier();
  bf16x8_t kf[2][KS];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      kf[s][kk] = __builtin_bit_cast(bf16x8_t, kst[kst_slot<D>(16 * s + col, 4 * kk + grp)]);
  __builtin_amdgcn_wave_barrier();
  float x[2][4];
  float mt = -INFINITY;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s][kk], qf[kk], acc, 0, 0, 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool ok = (T.ok >> (s * 4 + e)) & 1u;
      x[s][e] = ok ? acc[e] * scale_log2 : -INFINITY;
      mt = fmaxf(mt, x[s][e]);
    }
  }
  // rows past the set read a stand-in row: zero their V values (a zero
  // probability times a non-finite value would still be NaN), only in the
  // waves that have such rows
  if (__builtin_amdgcn_ballot_w64(T.ok != 0xFFu)) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (!((T.ok >> (s * 4 + e)) & 1u)) {
#pragma unroll
          for (int w = 0; w < DB / 2; ++w) T.vf[s][e].w[w] = 0u;
        }
  }
  mt = max_over_groups(mt);
  // lazy rescaling: the reference st.m (and with it o and l) moves only when
  // some head of the wave sees its maximum rise by more than 2^8, so the
  // probabilities stay below 2^8; o / l does not depend on the reference
  const float m_new = fmaxf(st.m, mt);
  if (__builtin_amdgcn_ballot_w64(m_new > st.m + 8.f)) {
    const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(st.m - m_new);
    st.m = m_new;
    st.l *= alpha;
#pragma unroll
    for (int blk = 0; blk < DB; ++blk) st.o[blk] *= alpha;
  }
  // while st.m is -inf every score is -inf too: a finite reference makes
  // every probability 0 without a branch
  const float mref = st.m == -INFINITY ? 0.f : st.m;
  float psum = 0.f;
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int j0 = 2 * w, j1 = 2 * w + 1;
    const float p0 = __builtin_amdgcn_exp2f(x[j0 >> 2][j0 & 3] - mref);
    const float p1 = __builtin_amdgcn_exp2f(x[j1 >> 2][j1 & 3] - mref);
    psum += p0 + p1;
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{p0, p1}, bf16x2_t));
    hi[w] = h;
    lo[w] = __builtin_bit_cast(uint32_t, __builtin_convertvector(
        f32x2_t{p0 - __uint_as_float(h << 16), p1 - __uint_as_float(h & 0xFFFF0000u)}, bf16x2_t));
  }
  st.l += psum;
  const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
  const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
#pragma unroll
  for (int blk = 0; blk < DB; ++blk) {
    uint32_t aw[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int j0 = 2 * w, j1 = 2 * w + 1;
      // element blk of rows j0 (low half) and j1 (high half), one byte
      // permute: selector bytes 0-3 index the second source, 4-7 the first
      aw[w] = __builtin_amdgcn_perm(T.vf[j1 >> 2][j1 & 3].w[blk >> 1], T.vf[j0 >> 2][j0 & 3].w[blk >> 1],
                                    (blk & 1) ? 0x07060302u : 0x05040100u);
    }
    const bf16x8_t av = __builtin_bit_cast(bf16x8_t, make_uint4(aw[0], aw[1], aw[2], aw[3]));
    st.o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, phi, st.o[blk], 0, 0, 0);
    st.o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, plo, st.o[blk], 0, 0, 0);
  }
}

// Writes out/lse of query head bh from (M, sum, unnormalised numerator).
__device__ __forceinline__ void write_final(const AttnArgs& a, size_t bh, int D, int dim, float M,
                                            float num, float den) {
  a.out[bh * D + dim] = den > 0.f ? num / den : 0.f;
  if (a.lse && dim == 0) a.lse[bh] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
}

template <int D, bool DENSE, bool PAGED>
__global__ __launch_bounds__(512) void attn_split_bf16(AttnArgs a) {
  constexpr int KS = D / 32;
  constexpr int DB = D / 16;
  // dynamic LDS: [nwaves][attn_wave_bytes] wave regions (K staging, then the
  // wave's outputs), then the staged row ids [blockDim * kRowsPerThread]
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  __shared__ float sm_m[8][16];
  __shared__ float sm_l[8][16];
  const int split = blockIdx.x, u = blockIdx.y;
  const int hkv = a.kv.hkv, hq = a.kv.hq, G = hq / hkv;
  const int wbytes = attn_wave_bytes(D, G);
  int32_t* s_row = (int32_t*)(dyn + (size_t)(blockDim.x >> 6) * wbytes);
  const int b = u / hkv, g = u % hkv;
  const int start = split * a.chunk;
  const int nwaves = blockDim.x >> 6;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;
  // set entries, query and lengths load together
  int32_t raw[kRowsPerThread];
  prefetch_entries<DENSE>(a, u, start, raw);
  const __bf16* qb = (const __bf16*)a.q;
  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const int qh = col < G ? col : 0;
    const uint4* qp = (const uint4*)(qb + ((size_t)b * hq + g * G + qh) * D + grp * 8);
    const uint4 v = qp[4 * kk];
    qf[kk] = __builtin_bit_cast(bf16x8_t, col < G ? v : make_uint4(0, 0, 0, 0));
  }
  const int nb = kv_seq_len(a.kv, b);
  if (!DENSE && unit_excluded(a, u)) return;
  const UnitSpan sp = unit_span<DENSE>(a, u, b, nb);
  const int L = sp.L;
  if (L == 0 && split == 0) {  // empty set: y = 0, lse = -inf
    for (int e = threadIdx.x; e < G * D; e += blockDim.x)
      write_final(a, (size_t)b * hq + g * G + e / D, D, e % D, -INFINITY, 0.f, 0.f);
    return;
  }
  if (start >= L) return;
  const int n = min(L, start + a.chunk) - start;
  stage_rows<DENSE, PAGED>(a, raw, start, n, sp, nb, b, g, s_row);

  const __bf16* kb = (const __bf16*)a.kv.k;
  const __bf16* vb = (const __bf16*)a.kv.v;
  WaveState<D> st;
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int i = 0; i < DB; ++i) st.o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // this wave's tiles: wave, wave + nwaves, ...; the steady-state body always
  // has a next tile, so its prefetch is unconditional and the compiler can
  // wait for the current buffer only
  const int ntiles = (n + 31) >> 5;
  const int iters = wave < ntiles ? (ntiles - wave + nwaves - 1) / nwaves : 0;
  if (iters > 0) {
    Tile<D> A, B;
    u32x4_t* kst = (u32x4_t*)(dyn + (size_t)wave * wbytes);
    const int step = 32 * nwaves;
    int r0 = wave * 32;
    load_tile<D>(A, s_row, r0, n, kb, vb, lane);
    int i = 0;
    for (; i + 2 < iters; i += 2) {
      load_tile<D>(B, s_row, r0 + step, n, kb, vb, lane);
      consume_tile<D>(A, st, qf, a.scale_log2, kst, lane);
      load_tile<D>(A, s_row, r0 + 2 * step, n, kb, vb, lane);
      consume_tile<D>(B, st, qf, a.scale_log2, kst, lane);
      r0 += 2 * step;
    }
    if (i + 1 < iters) {
      load_tile<D>(B, s_row, r0 + step, n, kb, vb, lane);
      consume_tile<D>(A, st, qf, a.scale_log2, kst, lane);
      consume_tile<D>(B, st, qf, a.scale_log2, kst, lane);
    } else {
      consume_tile<D>(A, st, qf, a.scale_log2, kst, lane);
    }
  }

  st.l = sum_over_groups(st.l);
  if (grp == 0) {
    sm_m[wave][col] = st.m;
    sm_l[wave][col] = st.l;
  }
  if (col < G) {
    float* wo = (float*)(dyn + (size_t)wave * wbytes) + col * (D + 1);
#pragma unroll
    for (int blk = 0; blk < DB; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) wo[(grp * 4 + i) * DB + blk] = st.o[blk][i];
  }
  __syncthreads();
  const int nsp = (L + a.chunk - 1) / a.chunk;
  for (int e = threadIdx.x; e < G * D; e += blockDim.x) {
    const int h = e / D, dim = e - h * D;
    float M = -INFINITY;
    for (int w = 0; w < nwaves; ++w) M = fmaxf(M, sm_m[w][h]);
    float num = 0.f, den = 0.f;
    if (M != -INFINITY) {
      for (int w = 0; w < nwaves; ++w) {
        const float f = __builtin_amdgcn_exp2f(sm_m[w][h] - M);
        num += f * ((const float*)(dyn + (size_t)w * wbytes))[h * (D + 1) + dim];
        den += f * sm_l[w][h];
      }
    }
    const size_t bh = (size_t)b * hq + g * G + h;
    if (nsp == 1) {
      write_final(a, bh, D, dim, M, num, den);
    } else {
      const size_t pidx = bh * a.nsplit + split;
      a.part_o[pidx * D + dim] = num;
      if (dim == 0) {
        a.part_ml[pidx * 2] = M;
        a.part_ml[pidx * 2 + 1] = den;
      }
    }
  }
}

template <int D, bool DENSE, bool PAGED>
__global__ __launch_bounds__(256) void attn_split_f32(AttnArgs a) {
  constexpr int DPL = D / 16;
  __shared__ float sm_m[4], sm_l[4];
  __shared__ float sm_o[4][D];
  __shared__ int32_t s_row[256 * kRowsPerThread];
  const int split = blockIdx.x, bh = blockIdx.y;
  const int hkv = a.kv.hkv, hq = a.kv.hq, G = hq / hkv;
  const int b = bh / hq, h = bh % hq, g = h / G, u = b * hkv + g;
  const int start = split * a.chunk;
  int32_t raw[kRowsPerThread];
  prefetch_entries<DENSE>(a, u, start, raw);
  const int nb = kv_seq_len(a.kv, b);
  if (!DENSE && unit_excluded(a, u)) return;
  const UnitSpan sp = unit_span<DENSE>(a, u, b, nb);
  const int L = sp.L;
  if (L == 0 && split == 0) {  // empty set: y = 0, lse = -inf
    for (int dim = threadIdx.x; dim < D; dim += blockDim.x)
      write_final(a, bh, D, dim, -INFINITY, 0.f, 0.f);
    return;
  }
  if (start >= L) return;
  const int n = min(L, start + a.chunk) - start;
  const int nwaves = blockDim.x >> 6;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rg = lane >> 4, c = lane & 15;
  const float* qp = (const float*)a.q + (size_t)bh * D + c * DPL;
  float qv[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) qv[i] = qp[i];
  stage_rows<DENSE, PAGED>(a, raw, start, n, sp, nb, b, g, s_row);
  const float* kb = (const float*)a.kv.k;
  const float* vb = (const float*)a.kv.v;
  float m_run = -INFINITY, l_run = 0.f, o[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) o[i] = 0.f;
  for (int t = wave * 4; t < n; t += 4 * nwaves) {
    const int r = t + rg;
    const int row = r < n ? s_row[r] : -1;
    const float* kp = kb + (int64_t)(row < 0 ? 0 : row) * D + c * DPL;
    const float* vp = vb + (int64_t)(row < 0 ? 0 : row) * D + c * DPL;
    float kx[DPL], vx[DPL];
#pragma unroll
    for (int i = 0; i < DPL; ++i) {
      kx[i] = kp[i];
      vx[i] = vp[i];
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < DPL; ++i) s = fmaf(qv[i], kx[i], s);
#pragma unroll
    for (int w = 1; w < 16; w <<= 1) s += __shfl_xor(s, w, 16);
    const float x = row >= 0 ? s * a.scale_log2 : -INFINITY;
    float mt = fmaxf(x, __shfl_xor(x, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    float alpha = 1.f, p = 0.f;
    if (m_new != -INFINITY) {
      alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      p = row >= 0 ? __builtin_amdgcn_exp2f(x - m_new) : 0.f;
    }
    l_run = l_run * alpha + p;
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] = o[i] * alpha + (row >= 0 ? p * vx[i] : 0.f);
    m_run = m_new;
  }
#pragma unroll
  for (int i = 0; i < DPL; ++i) {
    o[i] += __shfl_xor(o[i], 16);
    o[i] += __shfl_xor(o[i], 32);
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (lane < 16) {
#pragma unroll
    for (int i = 0; i < DPL; ++i) sm_o[wave][c * DPL + i] = o[i];
  }
  if (lane == 0) {
    sm_m[wave] = m_run;
    sm_l[wave] = l_run;
  }
  __syncthreads();
  const int nsp = (L + a.chunk - 1) / a.chunk;
  for (int dim = threadIdx.x; dim < D; dim += blockDim.x) {
    float M = -INFINITY;
    for (int w = 0; w < nwaves; ++w) M = fmaxf(M, sm_m[w]);
    float num = 0.f, den = 0.f;
    if (M != -INFINITY) {
      for (int w = 0; w < nwaves; ++w) {
        const float f = __builtin_amdgcn_exp2f(sm_m[w] - M);
        num += f * sm_o[w][dim];
        den += f * sm_l[w];
      }
    }
    if (nsp == 1) {
      write_final(a, bh, D, dim, M, num, den);
    } else {
      const size_t pidx = (size_t)bh * a.nsplit + split;
      a.part_o[pidx * D + dim] = num;
      if (dim == 0) {
        a.part_ml[pidx * 2] = M;
        a.part_ml[pidx * 2 + 1] = den;
      }
    }
  }
}

// Combines the split partials of one query head (grid: batch * num_q_heads,
// 256 threads).  Every thread first loads all it may need (the m, l and
// numerators of its first kMergePerThread split slots, for 256 / d split
// groups) together with the unit's lengths, before the number of splits in
// use is known, so the kernel costs one memory latency; slots past that
// number (stale values of earlier calls) are masked, never used in
// arithmetic.  The max, the weights and the sums follow in registers and
// LDS.  Units that fit one split were written by the split kernel and are
// skipped.
constexpr int kMergePerThread = 16;

template <int D, bool DENSE>
__global__ __launch_bounds__(256) void attn_merge(AttnArgs a) {
  constexpr int SG = 256 / D;
  __shared__ float s_red[SG][D];
  __shared__ float s_den[SG];
  __shared__ float s_max[4];
  const int bh = blockIdx.x;
  const int hkv = a.kv.hkv, hq = a.kv.hq, G = hq / hkv;
  const int b = bh / hq, h = bh % hq, u = b * hkv + h / G;
  const float* ml = a.part_ml + (size_t)bh * a.nsplit * 2;
  const float* po = a.part_o + (size_t)bh * a.nsplit * D;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sg = tid / D, dim = tid - sg * D;
  // the first batch of slots below nsplit (a launch argument: no load
  // waits for another)
  float m0[kMergePerThread], l0[kMergePerThread], o0[kMergePerThread];
#pragma unroll
  for (int k = 0; k < kMergePerThread; ++k) {
    const int s = sg + k * SG;
    const bool in = s < a.nsplit;
    m0[k] = in ? ml[2 * s] : -INFINITY;
    l0[k] = in ? ml[2 * s + 1] : 0.f;
    o0[k] = in ? po[(size_t)s * D + dim] : 0.f;
  }
  if (!DENSE && unit_excluded(a, u)) return;
  const int L = unit_span<DENSE>(a, u, b, kv_seq_len(a.kv, b)).L;
  const int nsp = (L + a.chunk - 1) / a.chunk;
  if (nsp <= 1) return;
  float mx = -INFINITY, num = 0.f, den = 0.f;
  for (int s0 = sg; s0 < nsp; s0 += SG * kMergePerThread) {
    float m[kMergePerThread], l[kMergePerThread], o[kMergePerThread];
#pragma unroll
    for (int k = 0; k < kMergePerThread; ++k) {
      const int s = s0 + k * SG;
      const bool ok = s < nsp;
      if (s0 == sg) {
        m[k] = ok ? m0[k] : -INFINITY;
        l[k] = ok ? l0[k] : 0.f;
        o[k] = ok ? o0[k] : 0.f;
      } else {
        m[k] = ok ? ml[2 * s] : -INFINITY;
        l[k] = ok ? ml[2 * s + 1] : 0.f;
        o[k] = ok ? po[(size_t)s * D + dim] : 0.f;
      }
    }
    // rescale the running sums to the new maximum of this thread
    float bm = mx;
#pragma unroll
    for (int k = 0; k < kMergePerThread; ++k) bm = fmaxf(bm, m[k]);
    if (bm != -INFINITY) {
      const float r = __builtin_amdgcn_exp2f(mx - bm);
      num *= r;
      den *= r;
#pragma unroll
      for (int k = 0; k < kMergePerThread; ++k) {
        const float f = __builtin_amdgcn_exp2f(m[k] - bm);
        num += f * o[k];
        den += f * l[k];
      }
      mx = bm;
    }
  }
  // block-wide maximum
  const float wm = wave_max(mx);
  if (lane == 0) s_max[wave] = wm;
  __syncthreads();
  const float M = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
  const float f = (mx == -INFINITY || M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mx - M);
  s_red[sg][dim] = num * f;
  if (dim == 0) s_den[sg] = den * f;
  __syncthreads();
  if (sg == 0) {
    float tot = 0.f, dt = 0.f;
#pragma unroll
    for (int k = 0; k < SG; ++k) {
      tot += s_red[k][dim];
      dt += s_den[k];
    }
    write_final(a, bh, D, dim, M, tot, dt);
  }
}

// Workgroups the split geometry aims for: few for the sparse path (one
// split per unit avoids the merge launch whenever the units alone fill the
// chip), many for the dense stream.  PRHS_ATTN_GROUPS and
// PRHS_ATTN_DENSE_GROUPS override them (tuning knobs, read once per process).
int env_int(const char* name, int dflt) {
  const char* e = getenv(name);
  const int x = e ? atoi(e) : 0;
  return x > 0 ? x : dflt;
}

int target_groups(bool dense) {
  static const int sparse_v = env_int("PRHS_ATTN_GROUPS", 256);
  static const int dense_v = env_int("PRHS_ATTN_DENSE_GROUPS", 1024);
  return dense ? dense_v : sparse_v;
}

// Waves per bf16 workgroup: PRHS_ATTN_WAVES overrides the default of 4.
int wave_limit() {
  static int v = [] {
    const char* e = getenv("PRHS_ATTN_WAVES");
    const int x = e ? atoi(e) : 0;
    return x >= 1 && x <= 8 ? x : 4;
  }();
  return v;
}

template <int D, bool DENSE, bool PAGED>
hipError_t launch_typed(const AttnArgs& a, int dtype, int units, int waves, hipStream_t stream) {
  if (dtype == 1) {
    const int G = a.kv.hq / a.kv.hkv;
    const size_t dyn = (size_t)waves * attn_wave_bytes(D, G) +
                       (size_t)64 * waves * kRowsPerThread * sizeof(int32_t);
    if (dyn > 65536) {
      const hipError_t e = hipFuncSetAttribute((const void*)attn_split_bf16<D, DENSE, PAGED>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((attn_split_bf16<D, DENSE, PAGED>), dim3(a.nsplit, units), dim3(64 * waves),
                       dyn, stream, a);
  } else {
    hipLaunchKernelGGL((attn_split_f32<D, DENSE, PAGED>), dim3(a.nsplit, units), dim3(256), 0,
                       stream, a);
  }
  if (a.nsplit > 1)
    hipLaunchKernelGGL((attn_merge<D, DENSE>), dim3(a.kv.batch * a.kv.hq), dim3(256), 0, stream,
                       a);
  return hipGetLastError();
}

struct AttnLayout {
  size_t part_o, part_ml, total;
};

AttnLayout attn_layout(int batch, int hq, int d, int nsplit) {
  const size_t parts = (size_t)batch * hq * nsplit;
  AttnLayout L;
  size_t off = 0;
  L.part_o = off;  off += (parts * d * 4 + 255) & ~(size_t)255;
  L.part_ml = off; off += parts * 2 * 4;
  L.total = off;
  return L;
}

int waves_for(int dtype, int chunk) {
  if (dtype != 1) return 4;
  int w = chunk / 32;
  const int lim = wave_limit();
  return w < 1 ? 1 : (w > lim ? lim : w);
}

}  // namespace

// Rows per workgroup: a multiple of the per-wave tile (32 rows for bf16, 16
// rows for fp32), sized so about target_groups() workgroups cover the
// largest unit, at most 8 staged rows per thread, at most kMaxSplits splits,
// and balanced so the splits of a full unit differ by at most one tile.
void attn_split_geometry(int dtype, bool dense, int batch, int hq, int hkv, int rows_cap,
                         int* chunk, int* nsplit) {
  const int gran = dtype == 1 ? 32 : 16;
  const long long units = dtype == 1 ? (long long)batch * hkv : (long long)batch * hq;
  const long long rows = rows_cap > 0 ? rows_cap : 1;
  const long long tg = target_groups(dense);
  long long c = (rows * (units > 0 ? units : 1) + tg - 1) / tg;
  const long long cmin = (rows + kMaxSplits - 1) / kMaxSplits;
  if (c < cmin) c = cmin;
  const long long threads = dtype == 1 ? 64LL * wave_limit() : 256;
  const long long cmax = threads * kRowsPerThread;
  if (!dense && rows <= kNoSplitRows && rows <= cmax) c = rows;
  if (c > cmax) c = cmax;
  if (c < gran) c = gran;
  const long long ns = (rows + c - 1) / c;
  c = (rows + ns - 1) / ns;
  c = ((c + gran - 1) / gran) * gran;
  if (c > cmax) c = cmax;
  *chunk = (int)c;
  *nsplit = (int)((rows + c - 1) / c);
}

// Scratch for the split-K partials of prhs_sparse_decode_attn_static, the
// entry point for callers that cannot allocate.  Every device that runs it
// holds its own copy until the process ends; calls on one device share it.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

hipError_t attn_static_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

size_t attn_workspace_bytes(int dtype, bool dense, int batch, int hq, int hkv, int d,
                            int rows_cap) {
  int chunk, nsplit;
  attn_split_geometry(dtype, dense, batch, hq, hkv, rows_cap, &chunk, &nsplit);
  return attn_layout(batch, hq, d, nsplit).total;
}

hipError_t launch_attention(const AttnLaunch& s, bool dense, hipStream_t stream) {
  if (s.kv.batch == 0) return hipSuccess;
  AttnArgs a;
  a.kv = s.kv;
  a.q = s.q;
  a.set_idx = s.set_idx;
  a.set_len = s.set_len;
  a.tail_start = dense ? nullptr : s.tail_start;
  a.unit_row = dense ? nullptr : s.unit_row;
  a.unit_tail = dense ? nullptr : s.unit_tail;
  a.pool_rows = s.pool_rows;
  a.unit_gate = dense ? nullptr : s.unit_gate;
  a.units_side = s.units_side;
  a.psaw = dense ? 0 : s.psaw;
  a.psaw_f = s.psaw_f;
  a.psaw_sink = s.psaw_sink;
  a.set_cap = s.set_cap;
  a.scale_log2 = s.scale * 1.44269504088896340736f;
  const int rows_cap = dense ? s.kv.max_seq_len : s.set_cap;
  attn_split_geometry(s.dtype, dense, s.kv.batch, s.kv.hq, s.kv.hkv, rows_cap, &a.chunk,
                      &a.nsplit);
  const AttnLayout L = attn_layout(s.kv.batch, s.kv.hq, s.kv.d, a.nsplit);
  char* ws = (char*)s.ws;
  a.part_o = (float*)(ws + L.part_o);
  a.part_ml = (float*)(ws + L.part_ml);
  a.out = s.out;
  a.lse = s.lse;
  const int waves = waves_for(s.dtype, a.chunk);
  const int units = s.dtype == 1 ? s.kv.batch * s.kv.hkv : s.kv.batch * s.kv.hq;
  const bool paged = s.kv.paged != 0;
#define PRHS_ATTN_DISPATCH(DV)                                                          \
  if (dense) {                                                                          \
    return paged ? launch_typed<DV, true, true>(a, s.dtype, units, waves, stream)       \
                 : launch_typed<DV, true, false>(a, s.dtype, units, waves, stream);     \
  }                                                                                     \
  return paged ? launch_typed<DV, false, true>(a, s.dtype, units, waves, stream)        \
               : launch_typed<DV, false, false>(a, s.dtype, units, waves, stream);
  if (s.kv.d == 128) {
    PRHS_ATTN_DISPATCH(128)
  }
  PRHS_ATTN_DISPATCH(64)
#undef PRHS_ATTN_DISPATCH
}

}  // namespace prhs

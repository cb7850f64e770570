// Causal prefill attention of a prompt under the progressive sliding
// attention window (Sec. 4.2, Eq. psaw: the window narrows during prefill
// as well as decoding).  The query at position i of sequence b (i < n_b)
// attends the keys p <= i with p < C_sink or p >= vis_start(i), the first
// visible position of Eq. psaw with the i + 1 tokens [0, i] in view (computed
// per query from the layer's factor); without PSAW every p <= i (plain
// causal attention, Eq. attn_eq per position).
//
// attn_prefill_bf16<D, QB, PAGED>: one workgroup per (QB = 192 or 256
// query positions, batch, query head), over a contiguous or paged cache;
// wave w takes the 16 queries q0 + 16w .. q0 + 16w + 15 as the 16 columns
// of its MFMA tiles, so a wave owns its queries' whole softmax and writes
// their outputs itself.  Key tiles of 64 rows are loaded once per workgroup
// (whole rows, one tile ahead of their use; the default cache policy, since
// the unit's other query blocks read the same rows) into two LDS buffers,
// K and V both row-major, and every wave computes
//   S^T (64 keys x 16 queries) = K_tile . Q^T   (v_mfma_f32_16x16x32_bf16, four 16-row blocks)
//   O^T (d x 16 queries)      += V_tile^T . P^T (P as bf16 hi + lo parts, 32 keys per product;
//                                                the V^T operand by transposing LDS reads)
// with an online softmax per query (rescaled lazily).  A block visits only
// the key tiles that meet its queries' visible ranges -- the sink
// [0, C_sink) and the band from the smallest vis_start of its queries to
// its last query -- so tiles that PSAW masks for every query of the block
// are never loaded: that is the prefill work PSAW saves.  Inside the block a
// wave skips the tiles masked for all of its queries and takes the
// per-(key, query) mask only on tiles that some of its queries see in part.
// Blocks are ordered per XCD: each XCD takes whole (batch, head) units, a
// unit's query blocks longest first (the last blocks see the most keys).
#include "prhs_internal.h"

namespace prhs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Query positions per workgroup, 16 per wave: 256 (16 waves) when the
// launch has at least kWideMinGroupsPerCu workgroups per CU, 192 (12 waves)
// otherwise, where the longer blocks would leave the last round of
// workgroups short of CUs.
constexpr int kQBlockWide = 256;
constexpr int kQBlockNarrow = 192;
constexpr int kWideMinGroupsPerCu = 4;
constexpr int kKTile = 64;    // key rows per tile
static_assert(kKTile % 32 == 0, "a tile is whole 32-key sub-tiles");
static_assert(kKTile <= 64, "wave 0 looks up one tile row per lane (paged caches)");
constexpr int kXcds = 8;      // accelerator dies, each with its own L2
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLazyLog2 = 8.f;  // log2 of the largest probability between rescales

struct PrefillArgs {
  KvView kv;
  const __bf16* q;        // [B][Hq][T][D]
  int T;
  int psaw;               // nonzero: row i attends [0, sink) U [first visible at i + 1, i]
  double psaw_f;          // Eq. psaw factor of the layer
  int sink;
  float scale_log2;
  float* out;             // [B][Hq][T][D]
  float* lse;             // [B][Hq][T] or null
};

// K tile in LDS: 16-byte chunk c of tile row r at slot c ^ (r mod D/8), so
// the whole-row writes and the MFMA-order reads (16 rows, one chunk each)
// hit distinct banks.
template <int D>
__device__ __forceinline__ int k_slot(int r, int c) {
  constexpr int CH = D / 8;
  return r * CH + (c ^ (r & (CH - 1)));
}

// Whole-row loads of tile rows [ks, ks + kKTile): each thread takes up to
// RPL 16-byte chunks of K and of V (threads past the tile's chunks take none).
// Rows at or past n (the prompt) read row n - 1.  A paged cache resolves
// every row through the block table (a row outside the table's valid pages
// reads element 0 of the cache instead: no access outside it).
template <int D, int NT>
struct TileRegs {
  static constexpr int RPL = (kKTile * (D / 8) + NT - 1) / NT;  // chunks per thread
  u32x4_t k[RPL], v[RPL];
};

// One thread's chunks of a tile: element offsets.  For a paged cache the
// row offsets of each tile come from LDS, where wave 0 stores them (one
// block-table read per row) two tiles ahead of the loads.
template <int D, int NT>
struct TileOffs {
  int64_t e[TileRegs<D, NT>::RPL];
};

// This thread's chunks of the tile at rows [ks, ks + kKTile) of a
// contiguous cache.
template <int D, int NT>
__device__ __forceinline__ void tile_offsets(TileOffs<D, NT>& off, int64_t unit_row0, int ks, int n) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int j = 0; j < TileRegs<D, NT>::RPL; ++j) {
    const int e = (int)threadIdx.x + j * NT;
    const int r = (e / CH) % kKTile, c = e % CH;
    off.e[j] = (unit_row0 + min(ks + r, n - 1)) * D + c * 8;
  }
}

// The same from the tile's row offsets in LDS (paged cache).
template <int D, int NT>
__device__ __forceinline__ void tile_offsets_lds(TileOffs<D, NT>& off, const int64_t* rows) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int j = 0; j < TileRegs<D, NT>::RPL; ++j) {
    const int e = (int)threadIdx.x + j * NT;
    off.e[j] = rows[(e / CH) % kKTile] + (e % CH) * 8;
  }
}

// Element offset of the row of position min(pos, n - 1) of (b, kv head g) in
// a paged cache (element 0 for a position outside the table's valid pages:
// no access outside the cache).
__device__ __forceinline__ int64_t paged_row(const KvView& kv, int b, int g, int pos, int n) {
  const int64_t row = kv_row_offset(kv, b, g, min(pos, n - 1));
  return row < 0 ? 0 : row;
}

template <int D, int NT>
__device__ __forceinline__ void tile_load(TileRegs<D, NT>& R, const KvView& kv,
                                          const TileOffs<D, NT>& off) {
  const __bf16* kb = (const __bf16*)kv.k;
  const __bf16* vb = (const __bf16*)kv.v;
  constexpr int CH = D / 8;
#pragma unroll
  for (int j = 0; j < TileRegs<D, NT>::RPL; ++j) {
    const int e = (int)threadIdx.x + j * NT;
    if (e >= kKTile * CH) break;
    R.k[j] = *(const u32x4_t*)(kb + off.e[j]);
    R.v[j] = *(const u32x4_t*)(vb + off.e[j]);
  }
}

// V tile in LDS: row-major, key rows of D * 2 bytes padded to
// vrow_bytes<D> (32 bytes more), so that the transposing operand reads below
// (4 key rows x 4 pieces of 8 bytes per 16 lanes) hit distinct banks and
// every read of a row's pieces is the lane's base address plus a constant.
template <int D>
constexpr int vrow_bytes() { return D * 2 + 32; }

template <int D, int NT>
__device__ __forceinline__ void tile_store(const TileRegs<D, NT>& R, u32x4_t* sk, u32x4_t* sv) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int j = 0; j < TileRegs<D, NT>::RPL; ++j) {
    const int e = (int)threadIdx.x + j * NT;
    if (e >= kKTile * CH) break;
    const int r = e / CH, c = e % CH;
    sk[k_slot<D>(r, c)] = R.k[j];
    *(u32x4_t*)((unsigned char*)sv + r * vrow_bytes<D>() + c * 16) = R.v[j];
  }
}

// Maximum over the lanes col, col + 16, col + 32 and col + 48 (one query's
// four lane groups), by the cross-half and cross-row lane swaps: each swap
// of a value with itself leaves a lane holding its own value and its
// partner's, one in each result.
__device__ __forceinline__ float max_over_groups(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// One key tile against one wave's 16 queries: S^T, the per-(key, query)
// mask, the online softmax and O^T += V^T P^T (as in the decode kernel, with
// the query positions in the columns).
template <int D>
__device__ __forceinline__ void prefill_tile(const u32x4_t* sk, const u32x4_t* svx, int ks,
                                             const bf16x8_t* qf, int qi, bool qvalid, int my_vis,
                                             int sink, float scale_log2, bool full, float& m_run,
                                             float& l_run, f32x4_t* o) {
  constexpr int KS = D / 32;       // products per 16-key block of S
  constexpr int DB = D / 16;       // 16-dim blocks of O^T
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  // the tile in 32-key sub-tiles u, each taken through the whole step
  // (scores, mask, softmax update, products) so that only its 8 scores per
  // lane are live at a time
#pragma unroll
  for (int u = 0; u < kKTile / 32; ++u) {
    // S^T for this wave's 16 queries: lane (col, grp) gets keys
    // ks + 32u + 16h + 4grp + e of 16-key block h
    float x[2][4];
    float mt = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int s = 2 * u + h;
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
      // raised issue priority around the MFMA runs, so that a wave ready to
      // issue products goes ahead of waves doing softmax work
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8_t kf = __builtin_bit_cast(bf16x8_t, sk[k_slot<D>(16 * s + col, 4 * kk + grp)]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[kk], acc, 0, 0, 0);
      }
      __builtin_amdgcn_s_setprio(0);
      // the MFMA output row is the key, the column the query: lane (col,
      // grp) holds query col of its wave for keys 4 grp + e of block s.
      // Raw products (scale_log2 > 0 is applied with the maximum's shift).
      if (full) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[h][e] = acc[e];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int p = ks + 16 * s + 4 * grp + e;
          const bool vis = qvalid && p <= qi && (p < sink || p >= my_vis);
          x[h][e] = vis ? acc[e] : -INFINITY;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) mt = fmaxf(mt, x[h][e]);
    }
    mt = max_over_groups(mt);
    // lazy rescaling: the reference m_run (and with it O and l) moves only
    // when some query of the wave sees its maximum rise by more than 2^8, so
    // the probabilities stay below 2^8; O / l does not depend on the reference
    const float m_new = fmaxf(m_run, mt * scale_log2);
    if (__builtin_amdgcn_ballot_w64(m_new > m_run + kLazyLog2)) {
      const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int blk = 0; blk < DB; ++blk) o[blk] *= alpha;
    }
    // P^T as bf16 hi + lo parts: lane (col, grp) holds keys 32u + 16h +
    // 4 grp + e, in the K-index order 8 grp + 4h + e of the products
    // while m_run is -inf every score is -inf too: a finite reference makes
    // every probability 0 without a branch
    const float mref = m_run == -INFINITY ? 0.f : m_run;
    uint32_t hi[4], lo[4];
    float psum = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      // probabilities of keys 2w and 2w + 1 of this lane's 8, converted
      // as a pair (round to nearest even), then the pair of remainders
      const int j0 = 2 * w, j1 = 2 * w + 1;
      const float p0 = __builtin_amdgcn_exp2f(fmaf(x[j0 >> 2][j0 & 3], scale_log2, -mref));
      const float p1 = __builtin_amdgcn_exp2f(fmaf(x[j1 >> 2][j1 & 3], scale_log2, -mref));
      psum += p0 + p1;
      const uint32_t hp = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{p0, p1}, bf16x2_t));
      const float r0 = p0 - __uint_as_float(hp << 16);
      const float r1 = p1 - __uint_as_float(hp & 0xFFFF0000u);
      hi[w] = hp;
      lo[w] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{r0, r1}, bf16x2_t));
    }
    l_run += psum;
    const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
    const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
    // V^T operand of product blk (16 dims x 32 keys; lane (col, grp) needs
    // dim 16 blk + col at its 8 keys, the keys of its probabilities) by two
    // transposing LDS loads from the row-major tile: in each 16-lane group,
    // lane 4e + q points at the 8-byte piece (dims 16 blk + 4q .. + 3) of
    // key row 32u + 16h + 4 grp + e, and the load hands lane col the values
    // of dim 16 blk + col at its group's 4 rows, e = 0 .. 3.
    const unsigned char* vrow = (const unsigned char*)svx +
                                (32 * u + 4 * grp + (col >> 2)) * vrow_bytes<D>() + 8 * (col & 3);
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int blk = 0; blk < DB; ++blk) {
      const v4i16_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) v4i16_t*)(vrow + 32 * blk));
      const v4i16_t a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) v4i16_t*)(vrow + 16 * vrow_bytes<D>() + 32 * blk));
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
      o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, phi, o[blk], 0, 0, 0);
      o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, plo, o[blk], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
  }
}

template <int D, int QB, bool PAGED>
__global__ __launch_bounds__(QB / 16 * 64) void attn_prefill_bf16(PrefillArgs a) {
  constexpr int kQBlock = QB;
  constexpr int kThreads = QB / 16 * 64;
  constexpr int KS = D / 32;   // products per 16-key block of S
  constexpr int DB = D / 16;   // output blocks of 16 dims per lane group
  constexpr int CH = D / 8;    // 16-byte chunks per row
  __shared__ u32x4_t s_k[2][kKTile * CH];
  __shared__ u32x4_t s_v[2][kKTile * vrow_bytes<D>() / 16];
  __shared__ int s_vmin;
  __shared__ int64_t s_rows[2][PAGED ? kKTile : 1];  // paged: row offsets of upcoming tiles
  // Workgroups go to the 8 XCDs round-robin by id; id L runs unit-major
  // slot (L mod 8) * (N / 8) + L / 8, so that each XCD works through its
  // own (batch, head) units one after another and a unit's K and V stay in
  // that XCD's L2.  Within a unit the longest query blocks come first.
  const int nqb = (a.T + kQBlock - 1) / kQBlock;
  const int N = (int)gridDim.x, L = (int)blockIdx.x;
  const int M = (N % kXcds == 0) ? (L % kXcds) * (N / kXcds) + L / kXcds : L;
  const int bh = M / nqb;
  const int qb = nqb - 1 - M % nqb;
  const int hq = a.kv.hq, G = hq / a.kv.hkv;
  const int b = bh / hq, h = bh % hq, g = h / G;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 15, grp = lane >> 4;
  const int n = min(kv_seq_len(a.kv, b), a.T);  // prompt positions with a query
  const int q0 = qb * kQBlock;
  const int qi = q0 + wave * 16 + col;            // this lane's query position
  const size_t qrow = ((size_t)b * hq + h) * a.T;
  const int qlast = min(q0 + kQBlock, n) - 1;      // last query of the block inside the prompt

  if (qlast < q0) {  // the whole block lies past the prompt: empty rows
    for (int e = tid; e < kQBlock * D; e += kThreads) {
      const int i = q0 + e / D;
      if (i < a.T) a.out[(qrow + i) * D + e % D] = 0.f;
    }
    if (a.lse)
      for (int i = q0 + tid; i < min(q0 + kQBlock, a.T); i += kThreads) a.lse[qrow + i] = -INFINITY;
    return;
  }

  // the block's key range: the sink, then the band from the smallest first
  // visible position of its queries to its last query
  const int sink_end = min(a.sink, qlast + 1);
  if (wave == 0) {
    int v = sink_end;
    if (a.psaw) {
      v = 0x7FFFFFFF;
      for (int i = q0 + lane; i <= qlast; i += 64) v = min(v, psaw_first_visible(a.psaw_f, a.sink, i + 1));
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off));
    }
    if (lane == 0) s_vmin = v;
  }
  // this lane's query and its first visible non-sink position
  const bool qvalid = qi <= qlast;
  const int my_vis = (a.psaw && qvalid) ? psaw_first_visible(a.psaw_f, a.sink, qi + 1) : 0;
  // a tile needs no mask for this wave when all 16 of its queries lie in
  // the prompt, the tile ends at or before the first of them, and it lies
  // inside the sink or at or past the largest of their vis_start
  const int qw0 = q0 + 16 * wave;
  const bool wave_all = qw0 + 15 <= qlast;
  int wvis = my_vis, wvmin = qvalid ? my_vis : 0x7FFFFFFF;
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) {
    wvis = max(wvis, __shfl_xor(wvis, off));
    wvmin = min(wvmin, __shfl_xor(wvmin, off));
  }
  // every 16-lane group holds the wave's 16 queries: the results are uniform
  wvis = __builtin_amdgcn_readfirstlane(wvis);
  wvmin = __builtin_amdgcn_readfirstlane(wvmin);
  // and it needs no work at all when it lies past the wave's last query or
  // between the sink and the smallest of their vis_start (every product
  // would be masked; skipping leaves O, m and l exactly as they are)
  const int wlast = min(qw0 + 15, qlast);
  bf16x8_t qf[KS];
  {
    const __bf16* qp = a.q + (qrow + (qvalid ? qi : q0)) * D + grp * 8;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = __builtin_bit_cast(bf16x8_t, *(const uint4*)(qp + 32 * kk));
  }
  __syncthreads();
  const int band_lo = min(max(s_vmin, sink_end), qlast + 1);
  const int nsink = (sink_end + kKTile - 1) / kKTile;
  const int tb0 = max(nsink, band_lo / kKTile), tb1 = qlast / kKTile;
  const int ntiles = nsink + (tb1 >= tb0 ? tb1 - tb0 + 1 : 0);

  const int64_t row0 = ((int64_t)b * a.kv.hkv + g) * a.kv.capacity;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  TileRegs<D, kThreads> R;
  auto tile_start = [&](int t) { return (t < nsink ? t : tb0 + (t - nsink)) * kKTile; };
  auto full_tile = [&](int ks) {
    return wave_all && ks + kKTile - 1 <= qw0 && (ks + kKTile <= a.sink || ks >= wvis);
  };
  auto masked_tile = [&](int ks) {
    return ks > wlast || (ks >= a.sink && ks + kKTile - 1 < wvmin);
  };
  // chunk offsets one tile ahead of the loads (contiguous cache); for a
  // paged cache wave 0 reads the block table for tile t + 2 while tile t is
  // multiplied and stores the row offsets in LDS
  TileOffs<D, kThreads> offs;
  if constexpr (PAGED) {
    if (ntiles > 0 && wave == 0) {
      s_rows[0][lane] = paged_row(a.kv, b, g, tile_start(0) + lane, n);
      s_rows[1][lane] = paged_row(a.kv, b, g, tile_start(min(1, ntiles - 1)) + lane, n);
    }
    __syncthreads();
    if (ntiles > 0) {
      tile_offsets_lds<D, kThreads>(offs, s_rows[0]);
      tile_load<D, kThreads>(R, a.kv, offs);
    }
  } else if (ntiles > 0) {
    tile_offsets<D, kThreads>(offs, row0, tile_start(0), n);
    tile_load<D, kThreads>(R, a.kv, offs);
    tile_offsets<D, kThreads>(offs, row0, tile_start(min(1, ntiles - 1)), n);
  }
  for (int t = 0; t < ntiles; ++t) {
    tile_store<D, kThreads>(R, s_k[t & 1], s_v[t & 1]);
    __syncthreads();
    int64_t prow = 0;
    if constexpr (PAGED) {
      // the table read is issued before the tile loads, so waiting for it
      // later does not wait for them
      if (wave == 0) prow = paged_row(a.kv, b, g, tile_start(min(t + 2, ntiles - 1)) + lane, n);
      tile_offsets_lds<D, kThreads>(offs, s_rows[(t + 1) & 1]);
    }
    tile_load<D, kThreads>(R, a.kv, offs);  // tile t + 1 (the last one again at the end)
    if constexpr (!PAGED)
      tile_offsets<D, kThreads>(offs, row0, tile_start(min(t + 2, ntiles - 1)), n);
    const int ks = tile_start(t);
    if (!masked_tile(ks))
      prefill_tile<D>(s_k[t & 1], s_v[t & 1], ks, qf, qi, qvalid, my_vis, a.sink, a.scale_log2,
                      full_tile(ks), m_run, l_run, o);
    if constexpr (PAGED)
      if (wave == 0) s_rows[t & 1][lane] = prow;  // tile t + 2, read after the next barrier
  }

  // lane (col, grp) holds dims 16 blk + 4 grp .. 16 blk + 4 grp + 3 of query col
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (qi < a.T) {
    float* op = a.out + (qrow + qi) * D + 4 * grp;
    const float inv = (qvalid && l_run > 0.f) ? 1.f / l_run : 0.f;
#pragma unroll
    for (int blk = 0; blk < DB; ++blk)
      *(float4*)(op + 16 * blk) =
          make_float4(o[blk][0] * inv, o[blk][1] * inv, o[blk][2] * inv, o[blk][3] * inv);
    if (a.lse && grp == 0)
      a.lse[qrow + qi] = (qvalid && l_run > 0.f) ? (m_run + log2f(l_run)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillLaunch& s, hipStream_t stream) {
  if (s.kv.batch == 0 || s.T == 0) return hipSuccess;
  PrefillArgs a;
  a.kv = s.kv;
  a.q = (const __bf16*)s.q;
  a.T = s.T;
  a.psaw = s.psaw;
  a.psaw_f = s.psaw_f;
  a.sink = s.sink;
  a.scale_log2 = s.scale * 1.44269504088896340736f;
  a.out = s.out;
  a.lse = s.lse;
  const long long units = (long long)s.kv.batch * s.kv.hq;
  const int cus = device_cus();
  const bool wide = cus > 0 && ((s.T + kQBlockWide - 1) / kQBlockWide) * units >=
                                   (long long)kWideMinGroupsPerCu * cus;
  const int qb = wide ? kQBlockWide : kQBlockNarrow;
  const dim3 grid((unsigned)(((s.T + qb - 1) / qb) * units));
  const dim3 block(qb / 16 * 64);
#define PRHS_PREFILL_LAUNCH(DV, PG)                                                           \
  do {                                                                                       \
    if (wide)                                                                                \
      hipLaunchKernelGGL((attn_prefill_bf16<DV, kQBlockWide, PG>), grid, block, 0, stream, a); \
    else                                                                                     \
      hipLaunchKernelGGL((attn_prefill_bf16<DV, kQBlockNarrow, PG>), grid, block, 0, stream, a); \
  } while (0)
  if (s.kv.d == 128) {
    if (s.kv.paged) PRHS_PREFILL_LAUNCH(128, true);
    else PRHS_PREFILL_LAUNCH(128, false);
  } else {
    if (s.kv.paged) PRHS_PREFILL_LAUNCH(64, true);
    else PRHS_PREFILL_LAUNCH(64, false);
  }
#undef PRHS_PREFILL_LAUNCH
  return hipGetLastError();
}

}  // namespace prhs

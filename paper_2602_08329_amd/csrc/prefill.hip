// Causal prefill attention of a prompt under the progressive sliding
// attention window (Sec. 4.2, Eq. psaw: the window narrows during prefill
// as well as decoding).  The query at position i of sequence b (i < n_b)
// attends the keys p <= i with p < C_sink or p >= vis_start[i]; without
// vis_start every p <= i (plain causal attention, Eq. attn_eq per position).
//
// attn_prefill_bf16<D>: one workgroup per (64 query positions, batch, query
// head); wave w takes the 16 queries q0 + 16w .. q0 + 16w + 15 as the 16
// columns of its MFMA tiles, so a wave owns its queries' whole softmax and
// writes their outputs itself.  Key tiles of 32 rows are loaded once per
// workgroup (whole rows, streaming cache policy) into LDS, double-buffered,
// and every wave computes
//   S^T (32 keys x 16 queries) = K_tile . Q^T   (v_mfma_f32_16x16x32_bf16, two 16-row halves)
//   O^T (d x 16 queries)      += V_tile^T . P^T (P as bf16 hi + lo parts)
// with an online softmax per query.  A block visits only the key tiles that
// meet its queries' visible ranges -- the sink [0, C_sink) and the band from
// the smallest vis_start of its queries to its last query -- so tiles that
// PSAW masks for every query of the block are never loaded: that is the
// prefill work PSAW saves.  Inside a tile the mask is per (key, query).
// Blocks are issued longest first (the last query blocks see the most keys).
#include "prhs_internal.h"

namespace prhs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kQBlock = 64;   // query positions per workgroup (4 waves x 16)
constexpr int kKTile = 32;    // key rows per tile
constexpr float kLn2 = 0.69314718055994530942f;

struct PrefillArgs {
  KvView kv;
  const __bf16* q;        // [B][Hq][T][D]
  int T;
  const int32_t* vis;     // [T] or null
  int sink;
  float scale_log2;
  float* out;             // [B][Hq][T][D]
  float* lse;             // [B][Hq][T] or null
};

__device__ __forceinline__ uint32_t bf16_bits_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// K tile in LDS: 16-byte chunk c of tile row r at slot c ^ (r mod D/8), so
// the whole-row writes and the MFMA-order reads (16 rows, one chunk each)
// hit distinct banks.
template <int D>
__device__ __forceinline__ int k_slot(int r, int c) {
  constexpr int CH = D / 8;
  return r * CH + (c ^ (r & (CH - 1)));
}

// Whole-row loads of tile rows [ks, ks + 32): each thread takes RPL 16-byte
// chunks of K and of V.  Rows at or past n (the prompt) read row n - 1.
template <int D>
struct TileRegs {
  static constexpr int RPL = kKTile * (D / 8) / 256;  // chunks per thread
  u32x4_t k[RPL], v[RPL];
};

template <int D>
__device__ __forceinline__ void tile_load(TileRegs<D>& R, const __bf16* kb, const __bf16* vb,
                                          int64_t unit_row0, int ks, int n) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int j = 0; j < TileRegs<D>::RPL; ++j) {
    const int e = (int)threadIdx.x + j * 256;
    const int r = e / CH, c = e % CH;
    const int p = min(ks + r, n - 1);
    const int64_t off = (unit_row0 + p) * D + c * 8;
    R.k[j] = stream_load16(kb + off);
    R.v[j] = stream_load16(vb + off);
  }
}

template <int D>
__device__ __forceinline__ void tile_store(const TileRegs<D>& R, u32x4_t* sk, u32x4_t* sv) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int j = 0; j < TileRegs<D>::RPL; ++j) {
    const int e = (int)threadIdx.x + j * 256;
    const int r = e / CH, c = e % CH;
    sk[k_slot<D>(r, c)] = R.k[j];
    sv[e] = R.v[j];  // row-major: row r, chunk c
  }
}

template <int D>
__global__ __launch_bounds__(256) void attn_prefill_bf16(PrefillArgs a) {
  constexpr int KS = D / 32;   // products per 16-key half of S
  constexpr int DB = D / 16;   // output blocks of 16 dims per lane group
  constexpr int CH = D / 8;    // 16-byte chunks per row
  __shared__ u32x4_t s_k[2][kKTile * CH];
  __shared__ u32x4_t s_v[2][kKTile * CH];
  __shared__ int s_vmin;
  const int qb = (int)gridDim.x - 1 - (int)blockIdx.x;  // longest blocks first
  const int bh = blockIdx.y;
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
    for (int e = tid; e < kQBlock * D; e += 256) {
      const int i = q0 + e / D;
      if (i < a.T) a.out[(qrow + i) * D + e % D] = 0.f;
    }
    if (a.lse)
      for (int i = q0 + tid; i < min(q0 + kQBlock, a.T); i += 256) a.lse[qrow + i] = -INFINITY;
    return;
  }

  // the block's key range: the sink, then the band from the smallest first
  // visible position of its queries to its last query
  const int sink_end = min(a.sink, qlast + 1);
  if (wave == 0) {
    int v = sink_end;
    if (a.vis) {
      const int i = q0 + lane;
      v = i <= qlast ? a.vis[i] : 0x7FFFFFFF;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off));
    }
    if (lane == 0) s_vmin = v;
  }
  // this lane's query and its first visible non-sink position
  const bool qvalid = qi <= qlast;
  const int my_vis = (a.vis && qvalid) ? a.vis[qi] : 0;
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

  const __bf16* kb = (const __bf16*)a.kv.k;
  const __bf16* vb = (const __bf16*)a.kv.v;
  const int64_t row0 = ((int64_t)b * a.kv.hkv + g) * a.kv.capacity;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  TileRegs<D> R;
  auto tile_start = [&](int t) { return (t < nsink ? t : tb0 + (t - nsink)) * kKTile; };
  if (ntiles > 0) tile_load<D>(R, kb, vb, row0, tile_start(0), n);
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    const int ks = tile_start(t);
    tile_store<D>(R, s_k[buf], s_v[buf]);
    __syncthreads();
    if (t + 1 < ntiles) tile_load<D>(R, kb, vb, row0, tile_start(t + 1), n);
    // S^T for this wave's 16 queries: lane (col, grp) gets keys ks + 16s + 4grp + e
    float x[2][4];
    float mt = -INFINITY;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8_t kf = __builtin_bit_cast(bf16x8_t, s_k[buf][k_slot<D>(16 * s + col, 4 * kk + grp)]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[kk], acc, 0, 0, 0);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int p = ks + 16 * s + 4 * grp + e;
        // the MFMA output row is the key, the column the query: lane (col,
        // grp) holds query col of its wave for keys 4 grp + e of half s
        const bool vis = qvalid && p <= qi && (p < a.sink || p >= my_vis);
        x[s][e] = vis ? acc[e] * a.scale_log2 : -INFINITY;
        mt = fmaxf(mt, x[s][e]);
      }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    float alpha = 1.f, psum = 0.f;
    uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
    if (m_new != -INFINITY) {
      alpha = exp2f(m_run - m_new);
      uint32_t hb[8], lb[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float pr = exp2f(x[j >> 2][j & 3] - m_new);
        psum += pr;
        hb[j] = bf16_bits_rne(pr);
        lb[j] = bf16_bits_rne(pr - __uint_as_float(hb[j] << 16));
      }
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        hi[w] = hb[2 * w] | (hb[2 * w + 1] << 16);
        lo[w] = lb[2 * w] | (lb[2 * w + 1] << 16);
      }
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
    const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
    // V operand: lane (col, grp) takes dims col DB .. col DB + DB - 1 of the
    // 8 rows 16s + 4grp + j, the rows of its probabilities
    const uint32_t* sv = (const uint32_t*)s_v[buf];
    uint32_t vw[2][4][DB / 2];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int w = 0; w < DB / 2; ++w)
          vw[s][j][w] = sv[((16 * s + 4 * grp + j) * D + col * DB) / 2 + w];
#pragma unroll
    for (int blk = 0; blk < DB; ++blk) {
      o[blk] *= alpha;
      uint32_t aw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int j0 = 2 * w, j1 = 2 * w + 1;
        const uint32_t e0 = vw[j0 >> 2][j0 & 3][blk >> 1], e1 = vw[j1 >> 2][j1 & 3][blk >> 1];
        const uint32_t v0 = (blk & 1) ? (e0 >> 16) : (e0 & 0xFFFFu);
        const uint32_t v1 = (blk & 1) ? (e1 >> 16) : (e1 & 0xFFFFu);
        aw[w] = v0 | (v1 << 16);
      }
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, make_uint4(aw[0], aw[1], aw[2], aw[3]));
      o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, phi, o[blk], 0, 0, 0);
      o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, plo, o[blk], 0, 0, 0);
    }
  }

  // lane (col, grp) holds dims (4 grp + i) DB + blk of query col
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (qi < a.T) {
    float* op = a.out + (qrow + qi) * D;
    const float inv = (qvalid && l_run > 0.f) ? 1.f / l_run : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v[DB];
#pragma unroll
      for (int blk = 0; blk < DB; ++blk) v[blk] = o[blk][i] * inv;
      float* dst = op + (grp * 4 + i) * DB;
#pragma unroll
      for (int blk = 0; blk < DB; blk += 4)
        *(float4*)(dst + blk) = make_float4(v[blk], v[blk + 1], v[blk + 2], v[blk + 3]);
    }
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
  a.vis = s.vis_start;
  a.sink = s.sink;
  a.scale_log2 = s.scale * 1.44269504088896340736f;
  a.out = s.out;
  a.lse = s.lse;
  const dim3 grid((s.T + kQBlock - 1) / kQBlock, s.kv.batch * s.kv.hq);
  if (s.kv.d == 128)
    hipLaunchKernelGGL(attn_prefill_bf16<128>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_prefill_bf16<64>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace prhs

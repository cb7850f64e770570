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
// bf16 inputs use MFMA for both products of a wave's 32-row tile:
//   S^T (32 keys x 16 heads) = K_tile . Q^T  (v_mfma_f32_16x16x32_bf16, two 16-row halves)
//   O^T (d x 16 heads)      += V_tile^T . P^T, P split into bf16 hi + lo parts so
//                              the probabilities keep ~16 significant bits.
// The key order inside a tile and the dimension order inside a row are
// permuted identically on both operands of each product, so every lane loads
// contiguous bytes: K rows as d/2-byte runs of one key, V rows as full
// 256-byte rows across 16 lanes (coalesced), and no LDS transpose is needed.
// fp32 inputs take a vector-ALU path (16 lanes per row, one query head per
// workgroup).
#include <stdlib.h>

#include "prhs_internal.h"

namespace prhs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;

struct AttnArgs {
  KvView kv;
  const void* q;
  const int32_t* set_idx;
  const int32_t* set_len;
  int set_cap;
  float scale_log2;
  int chunk, nsplit;
  float* part_o;    // [B*Hq][nsplit][D]
  float* part_ml;   // [B*Hq][nsplit][2]
  float* out;
  float* lse;
};

template <bool DENSE>
__device__ __forceinline__ int unit_rows(const AttnArgs& a, int b, int u) {
  if (DENSE) return kv_seq_len(a.kv, b);
  int L = a.set_len[u];
  L = L < 0 ? 0 : L;
  return L > a.set_cap ? a.set_cap : L;
}

// Element offset of the cached row at list position r, or -1 if r is past the
// list end or names a position outside [0, nb) or outside the cache.
template <bool DENSE>
__device__ __forceinline__ int64_t list_row(const AttnArgs& a, const int32_t* idx, int r, int end,
                                            int nb, int b, int g) {
  if (r >= end) return -1;
  const int pos = DENSE ? r : idx[r];
  if (pos < 0 || pos >= nb) return -1;
  return kv_row_offset(a.kv, b, g, pos);
}

__device__ __forceinline__ uint32_t bf16_bits_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
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
    const uint4 x = *(const uint4*)p;
    v.w[0] = x.x; v.w[1] = x.y; v.w[2] = x.z; v.w[3] = x.w;
  } else {
    const uint2 x = *(const uint2*)p;
    v.w[0] = x.x; v.w[1] = x.y;
  }
  return v;
}

template <int DB>
__device__ __forceinline__ uint32_t vrow_elem(const VRow<DB>& v, int e) {
  const uint32_t w = v.w[e >> 1];
  return (e & 1) ? (w >> 16) : (w & 0xFFFFu);
}

template <int D, bool DENSE>
__global__ __launch_bounds__(256) void attn_split_bf16(AttnArgs a) {
  constexpr int KS = D / 32;
  constexpr int DB = D / 16;
  __shared__ float sm_m[4][16];
  __shared__ float sm_l[4][16];
  __shared__ float sm_o[4][16][D + 1];
  const int split = blockIdx.x, u = blockIdx.y;
  const int hkv = a.kv.hkv, hq = a.kv.hq, G = hq / hkv;
  const int b = u / hkv, g = u % hkv;
  const int L = unit_rows<DENSE>(a, b, u);
  const int start = split * a.chunk;
  if (L == 0 && split == 0) {  // empty set: y = 0, lse = -inf
    for (int e = threadIdx.x; e < G * D; e += blockDim.x) {
      const size_t bh = (size_t)b * hq + g * G + e / D;
      a.out[bh * D + e % D] = 0.f;
      if (a.lse && e % D == 0) a.lse[bh] = -INFINITY;
    }
    return;
  }
  if (start >= L) return;
  const int end = min(L, start + a.chunk);
  const int nb = kv_seq_len(a.kv, b);
  const int nwaves = blockDim.x >> 6;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;

  const __bf16* qb = (const __bf16*)a.q;
  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    if (col < G) {
      const uint4* qp = (const uint4*)(qb + ((size_t)b * hq + g * G + col) * D + grp * (D / 4));
      qf[kk] = __builtin_bit_cast(bf16x8_t, qp[kk]);
    } else {
      qf[kk] = __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
    }
  }
  const __bf16* kb = (const __bf16*)a.kv.k;
  const __bf16* vb = (const __bf16*)a.kv.v;
  const int32_t* idx = DENSE ? nullptr : a.set_idx + (size_t)u * a.set_cap;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int t = start + wave * 32; t < end; t += 32 * nwaves) {
    bf16x8_t kf[2][KS];
    VRow<DB> vf[2][4];
    bool vok[2][4];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int64_t off = list_row<DENSE>(a, idx, t + 16 * s + col, end, nb, b, g);
      const uint4* kp = (const uint4*)(kb + (off < 0 ? 0 : off) + grp * (D / 4));
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        kf[s][kk] = __builtin_bit_cast(bf16x8_t, off < 0 ? make_uint4(0, 0, 0, 0) : kp[kk]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t vo = list_row<DENSE>(a, idx, t + 16 * s + grp * 4 + j, end, nb, b, g);
        vok[s][j] = vo >= 0;
        if (vo >= 0) {
          vf[s][j] = load_vrow<DB>(vb + vo + col * DB);
        } else {
#pragma unroll
          for (int w = 0; w < DB / 2; ++w) vf[s][j].w[w] = 0u;
        }
      }
    }
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
        x[s][e] = vok[s][e] ? acc[e] * a.scale_log2 : -INFINITY;
        mt = fmaxf(mt, x[s][e]);
      }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    float alpha = 1.f, psum = 0.f;
    uint32_t hi[4], lo[4];
    if (m_new == -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) hi[w] = lo[w] = 0u;
    } else {
      alpha = exp2f(m_run - m_new);
      uint32_t hb[8], lb[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float p = exp2f(x[j >> 2][j & 3] - m_new);
        psum += p;
        hb[j] = bf16_bits_rne(p);
        lb[j] = bf16_bits_rne(p - __uint_as_float(hb[j] << 16));
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
#pragma unroll
    for (int blk = 0; blk < DB; ++blk) {
      o[blk] *= alpha;
      uint32_t aw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int j0 = 2 * w, j1 = 2 * w + 1;
        aw[w] = vrow_elem<DB>(vf[j0 >> 2][j0 & 3], blk) | (vrow_elem<DB>(vf[j1 >> 2][j1 & 3], blk) << 16);
      }
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, make_uint4(aw[0], aw[1], aw[2], aw[3]));
      o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, phi, o[blk], 0, 0, 0);
      o[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, plo, o[blk], 0, 0, 0);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (grp == 0) {
    sm_m[wave][col] = m_run;
    sm_l[wave][col] = l_run;
  }
  if (col < G) {
#pragma unroll
    for (int blk = 0; blk < DB; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) sm_o[wave][col][(grp * 4 + i) * DB + blk] = o[blk][i];
  }
  __syncthreads();
  const int nsp = (L + a.chunk - 1) / a.chunk;
  const bool direct = nsp == 1;
  for (int e = threadIdx.x; e < G * D; e += blockDim.x) {
    const int h = e / D, dim = e - h * D;
    float M = -INFINITY;
    for (int w = 0; w < nwaves; ++w) M = fmaxf(M, sm_m[w][h]);
    float num = 0.f, den = 0.f;
    if (M != -INFINITY) {
      for (int w = 0; w < nwaves; ++w) {
        const float f = exp2f(sm_m[w][h] - M);
        num += f * sm_o[w][h][dim];
        den += f * sm_l[w][h];
      }
    }
    const size_t bh = (size_t)b * hq + g * G + h;
    if (direct) {
      a.out[bh * D + dim] = den > 0.f ? num / den : 0.f;
      if (a.lse && dim == 0) a.lse[bh] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
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

template <int D, bool DENSE>
__global__ __launch_bounds__(256) void attn_split_f32(AttnArgs a) {
  constexpr int DPL = D / 16;
  __shared__ float sm_m[4], sm_l[4];
  __shared__ float sm_o[4][D];
  const int split = blockIdx.x, bh = blockIdx.y;
  const int hkv = a.kv.hkv, hq = a.kv.hq, G = hq / hkv;
  const int b = bh / hq, h = bh % hq, g = h / G, u = b * hkv + g;
  const int L = unit_rows<DENSE>(a, b, u);
  const int start = split * a.chunk;
  if (L == 0 && split == 0) {  // empty set: y = 0, lse = -inf
    for (int dim = threadIdx.x; dim < D; dim += blockDim.x) a.out[(size_t)bh * D + dim] = 0.f;
    if (a.lse && threadIdx.x == 0) a.lse[bh] = -INFINITY;
    return;
  }
  if (start >= L) return;
  const int end = min(L, start + a.chunk);
  const int nb = kv_seq_len(a.kv, b);
  const int nwaves = blockDim.x >> 6;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rg = lane >> 4, c = lane & 15;
  const float* qp = (const float*)a.q + (size_t)bh * D + c * DPL;
  float qv[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) qv[i] = qp[i];
  const float* kb = (const float*)a.kv.k;
  const float* vb = (const float*)a.kv.v;
  const int32_t* idx = DENSE ? nullptr : a.set_idx + (size_t)u * a.set_cap;
  float m_run = -INFINITY, l_run = 0.f, o[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) o[i] = 0.f;
  for (int t = start + wave * 4; t < end; t += 4 * nwaves) {
    const int64_t off = list_row<DENSE>(a, idx, t + rg, end, nb, b, g);
    float kx[DPL], vx[DPL];
#pragma unroll
    for (int i = 0; i < DPL; ++i) {
      kx[i] = off >= 0 ? kb[off + c * DPL + i] : 0.f;
      vx[i] = off >= 0 ? vb[off + c * DPL + i] : 0.f;
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < DPL; ++i) s = fmaf(qv[i], kx[i], s);
#pragma unroll
    for (int w = 1; w < 16; w <<= 1) s += __shfl_xor(s, w, 16);
    const float x = off >= 0 ? s * a.scale_log2 : -INFINITY;
    float mt = fmaxf(x, __shfl_xor(x, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    float alpha = 1.f, p = 0.f;
    if (m_new != -INFINITY) {
      alpha = exp2f(m_run - m_new);
      p = exp2f(x - m_new);
    }
    l_run = l_run * alpha + p;
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] = o[i] * alpha + p * vx[i];
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
  const bool direct = nsp == 1;
  for (int dim = threadIdx.x; dim < D; dim += blockDim.x) {
    float M = -INFINITY;
    for (int w = 0; w < nwaves; ++w) M = fmaxf(M, sm_m[w]);
    float num = 0.f, den = 0.f;
    if (M != -INFINITY) {
      for (int w = 0; w < nwaves; ++w) {
        const float f = exp2f(sm_m[w] - M);
        num += f * sm_o[w][dim];
        den += f * sm_l[w];
      }
    }
    if (direct) {
      a.out[(size_t)bh * D + dim] = den > 0.f ? num / den : 0.f;
      if (a.lse && dim == 0) a.lse[bh] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
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
// block: d threads).  Units that fit one split were written by the split
// kernel and are skipped.
template <int D, bool DENSE>
__global__ __launch_bounds__(D) void attn_merge(AttnArgs a) {
  const int bh = blockIdx.x;
  const int hkv = a.kv.hkv, hq = a.kv.hq, G = hq / hkv;
  const int b = bh / hq, h = bh % hq, u = b * hkv + h / G;
  const int L = unit_rows<DENSE>(a, b, u);
  const int nsp = (L + a.chunk - 1) / a.chunk;
  if (nsp <= 1) return;
  const int dim = threadIdx.x;
  const float* ml = a.part_ml + (size_t)bh * a.nsplit * 2;
  const float* po = a.part_o + (size_t)bh * a.nsplit * D;
  float M = -INFINITY;
  for (int s = 0; s < nsp; ++s) M = fmaxf(M, ml[2 * s]);
  float num = 0.f, den = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < nsp; ++s) {
      const float f = exp2f(ml[2 * s] - M);
      num += f * po[(size_t)s * D + dim];
      den += f * ml[2 * s + 1];
    }
  }
  a.out[(size_t)bh * D + dim] = den > 0.f ? num / den : 0.f;
  if (a.lse && dim == 0) a.lse[bh] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
}

constexpr int kDefaultTargetGroups = 1024;

// Workgroups the split geometry aims for; PRHS_ATTN_GROUPS overrides it (a
// tuning knob, read once per process).
int target_groups() {
  static int v = [] {
    const char* e = getenv("PRHS_ATTN_GROUPS");
    const int x = e ? atoi(e) : 0;
    return x > 0 ? x : kDefaultTargetGroups;
  }();
  return v;
}

template <int D, bool DENSE>
void launch_typed(const AttnArgs& a, int dtype, int units, int waves, hipStream_t stream) {
  if (dtype == 1) {
    hipLaunchKernelGGL((attn_split_bf16<D, DENSE>), dim3(a.nsplit, units), dim3(64 * waves), 0,
                       stream, a);
  } else {
    hipLaunchKernelGGL((attn_split_f32<D, DENSE>), dim3(a.nsplit, units), dim3(64 * waves), 0,
                       stream, a);
  }
  if (a.nsplit > 1)
    hipLaunchKernelGGL((attn_merge<D, DENSE>), dim3(a.kv.batch * a.kv.hq), dim3(D), 0, stream, a);
}

struct AttnLayout {
  size_t part_o, part_ml, total;
};

AttnLayout attn_layout(int dtype, int batch, int hq, int hkv, int d, int nsplit) {
  const size_t parts = (size_t)batch * hq * nsplit;
  AttnLayout L;
  size_t off = 0;
  L.part_o = off;  off += (parts * d * 4 + 255) & ~(size_t)255;
  L.part_ml = off; off += parts * 2 * 4;
  L.total = off;
  return L;
}

}  // namespace

// Rows per workgroup: a multiple of the per-wave tile (32 rows for bf16, 16
// rows for fp32), sized so about target_groups() workgroups cover the
// largest unit, with up to 4 waves per workgroup.
void attn_split_geometry(int dtype, int batch, int hq, int hkv, int rows_cap, int* chunk,
                         int* nsplit) {
  const int gran = dtype == 1 ? 32 : 16;
  const long long units = dtype == 1 ? (long long)batch * hkv : (long long)batch * hq;
  const long long rows = rows_cap > 0 ? rows_cap : 1;
  const long long tg = target_groups();
  long long c = (rows * (units > 0 ? units : 1) + tg - 1) / tg;
  c = ((c + gran - 1) / gran) * gran;
  if (c < gran) c = gran;
  if (c > rows) c = ((rows + gran - 1) / gran) * gran;
  *chunk = (int)c;
  *nsplit = (int)((rows + c - 1) / c);
}

size_t attn_workspace_bytes(int dtype, int batch, int hq, int hkv, int d, int rows_cap) {
  int chunk, nsplit;
  attn_split_geometry(dtype, batch, hq, hkv, rows_cap, &chunk, &nsplit);
  return attn_layout(dtype, batch, hq, hkv, d, nsplit).total;
}

hipError_t launch_attention(const AttnLaunch& s, bool dense, hipStream_t stream) {
  if (s.kv.batch == 0) return hipSuccess;
  AttnArgs a;
  a.kv = s.kv;
  a.q = s.q;
  a.set_idx = s.set_idx;
  a.set_len = s.set_len;
  a.set_cap = s.set_cap;
  a.scale_log2 = s.scale * 1.44269504088896340736f;
  const int rows_cap = dense ? s.kv.max_seq_len : s.set_cap;
  attn_split_geometry(s.dtype, s.kv.batch, s.kv.hq, s.kv.hkv, rows_cap, &a.chunk, &a.nsplit);
  const AttnLayout L = attn_layout(s.dtype, s.kv.batch, s.kv.hq, s.kv.hkv, s.kv.d, a.nsplit);
  char* ws = (char*)s.ws;
  a.part_o = (float*)(ws + L.part_o);
  a.part_ml = (float*)(ws + L.part_ml);
  a.out = s.out;
  a.lse = s.lse;
  const int gran = s.dtype == 1 ? 32 : 16;
  int waves = s.dtype == 1 ? a.chunk / gran : 4;
  waves = waves < 1 ? 1 : (waves > 4 ? 4 : waves);
  const int units = s.dtype == 1 ? s.kv.batch * s.kv.hkv : s.kv.batch * s.kv.hq;
  if (s.kv.d == 128) {
    if (dense) launch_typed<128, true>(a, s.dtype, units, waves, stream);
    else launch_typed<128, false>(a, s.dtype, units, waves, stream);
  } else {
    if (dense) launch_typed<64, true>(a, s.dtype, units, waves, stream);
    else launch_typed<64, false>(a, s.dtype, units, waves, stream);
  }
  return hipGetLastError();
}

}  // namespace prhs

// Workgroup-level ordered set construction in LDS.
//
// compact_marked() appends, in ascending order, every position of [lo, hi)
// that a marker sets in an LDS bitmap, one segment of seg_bits positions at a
// time (clear, mark with atomicOr, popcount + workgroup prefix sum, write).
//
// build_index_set() uses it for an ascending, duplicate-free
//   [0, sink_end) U S* U {p + j : p in first m of S*, |j| <= r} U [w0, n)
// with w0 = max(win_start, sink_end), as used by the critical set (Sec. 4.1)
// and the dilated shared set (Eq. neighboring).  Every S* entry lies in the
// middle range [sink_end, win_start).  A neighbour that leaves the middle
// range lands either in the sink, in [w0, n), or outside [0, n); so only the
// middle range needs de-duplication.  Cost is O(|middle| / 32 + segments *
// (k + m(2r+1))) and independent of head_dim.
#pragma once

#include "prhs_internal.h"

namespace prhs {

constexpr int kSegBits = 262144;
constexpr int kSegWords = kSegBits / 32;

// Writes base + b for every set bit b of the LDS bitmap bm[0, nwords), in
// ascending order, to out[pos ...] (entries at or past cap are dropped) and
// returns pos plus the number of set bits.  `scan` holds BLOCK/64 + 1 words.
// Every thread of the workgroup must call it; bm must be complete (a barrier
// after the last mark).
template <int BLOCK>
__device__ int compact_bitmap(const uint32_t* bm, int nwords, int base, int32_t* out, int cap,
                              int pos, uint32_t* scan) {
  const int tid = threadIdx.x;
  // thread t owns words [t*wpt, (t+1)*wpt)
  const int wpt = (nwords + BLOCK - 1) / BLOCK;
  const int w_begin = min(nwords, tid * wpt);
  const int w_end = min(nwords, w_begin + wpt);
  uint32_t cnt = 0;
  for (int w = w_begin; w < w_end; ++w) cnt += __popc(bm[w]);
  uint32_t total = 0;
  const uint32_t off = block_exclusive_scan<BLOCK>(cnt, scan, &total);
  int o = pos + (int)off;
  for (int w = w_begin; w < w_end; ++w) {
    uint32_t bits = bm[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      bits &= bits - 1u;
      if (o < cap) out[o] = base + (w << 5) + bit;
      ++o;
    }
  }
  return pos + (int)total;
}

// `bm` holds seg_bits / 32 words of LDS, `scan` BLOCK/64 + 1 words.  Writes
// out[pos ...] (entries at or past cap are dropped) and returns the new pos.
// Every thread of the workgroup must call it.
template <int BLOCK, typename Mark>
__device__ int compact_marked(int lo, int hi, int seg_bits, Mark mark, int32_t* out, int cap,
                              int pos, uint32_t* bm, uint32_t* scan) {
  const int tid = threadIdx.x;
  for (int seg_lo = lo; seg_lo < hi; seg_lo += seg_bits) {
    const int seg_hi = min(hi, seg_lo + seg_bits);
    const int nwords = (seg_hi - seg_lo + 31) >> 5;
    for (int w = tid; w < nwords; w += BLOCK) bm[w] = 0u;
    lds_barrier();
    mark(seg_lo, seg_hi, bm);
    lds_barrier();
    pos = compact_bitmap<BLOCK>(bm, nwords, seg_lo, out, cap, pos, scan);
    lds_barrier();
  }
  return pos;
}

__device__ __forceinline__ void mark_bit(uint32_t* bm, int seg_lo, int p) {
  atomicOr(&bm[(p - seg_lo) >> 5], 1u << ((p - seg_lo) & 31));
}

// `topk` may point to global or LDS memory.  Writes at most set_cap entries
// of `out`; *out_len receives min(size, set_cap).
template <int BLOCK>
__device__ void build_index_set(const int32_t* topk, int klen, int m, int r, int sink_end,
                                int win_start, int n, int32_t* out, int set_cap, int32_t* out_len,
                                uint32_t* bm, uint32_t* scan, int seg_bits) {
  const int tid = threadIdx.x;
  for (int i = tid; i < sink_end; i += BLOCK)
    if (i < set_cap) out[i] = i;
  const int span = 2 * r + 1;
  auto mark = [&](int seg_lo, int seg_hi, uint32_t* b) {
    for (int j = tid; j < klen; j += BLOCK) {
      const int p = topk[j];
      if (p >= seg_lo && p < seg_hi) mark_bit(b, seg_lo, p);
    }
    const int nd = m * span;
    for (int j = tid; j < nd; j += BLOCK) {
      const int p = topk[j / span] + (j % span) - r;
      if (p >= seg_lo && p < seg_hi) mark_bit(b, seg_lo, p);
    }
  };
  int pos = compact_marked<BLOCK>(sink_end, win_start, seg_bits, mark, out, set_cap, sink_end, bm,
                                  scan);
  const int w0 = max(win_start, sink_end);
  const int nw = n - w0;
  for (int i = tid; i < nw; i += BLOCK) {
    const int o = pos + i;
    if (o < set_cap) out[o] = w0 + i;
  }
  if (nw > 0) pos += nw;
  if (tid == 0) *out_len = pos < set_cap ? pos : set_cap;
}

}  // namespace prhs

// Workgroup-level construction of an ascending, duplicate-free index set
//   [0, sink_end) U S* U {p + j : p in first m of S*, |j| <= r} U [w0, n)
// with w0 = max(win_start, sink_end), as used by the critical set (Sec. 4.1)
// and the dilated shared set (Eq. neighboring).
//
// Every S* entry lies in the middle range [sink_end, win_start).  A neighbour
// that leaves the middle range lands either in the sink, in [w0, n), or
// outside [0, n); so only the middle range needs de-duplication.  It is done
// with an LDS bitmap, one segment of kSegBits positions at a time, followed by
// an ordered compaction (popcount + workgroup prefix sum).  Cost is
// O(|middle| / 32 + segments * (k + m(2r+1))) and independent of head_dim.
#pragma once

#include "prhs_internal.h"

namespace prhs {

constexpr int kSegBits = 32768;
constexpr int kSegWords = kSegBits / 32;

// `topk` may point to global or LDS memory (flat address).  `bm` needs
// kSegWords words of LDS, `scan` BLOCK/64 + 1 words.  Writes at most set_cap
// entries of `out`; *out_len receives min(size, set_cap).
template <int BLOCK>
__device__ void build_index_set(const int32_t* topk, int klen, int m, int r, int sink_end,
                                int win_start, int n, int32_t* out, int set_cap, int32_t* out_len,
                                uint32_t* bm, uint32_t* scan) {
  const int tid = threadIdx.x;
  int pos = 0;
  for (int i = tid; i < sink_end; i += BLOCK)
    if (i < set_cap) out[i] = i;
  pos = sink_end;

  const int span = 2 * r + 1;
  for (int seg_lo = sink_end; seg_lo < win_start; seg_lo += kSegBits) {
    const int seg_hi = min(win_start, seg_lo + kSegBits);
    const int nwords = (seg_hi - seg_lo + 31) >> 5;
    for (int w = tid; w < nwords; w += BLOCK) bm[w] = 0u;
    __syncthreads();
    for (int j = tid; j < klen; j += BLOCK) {
      const int p = topk[j];
      if (p >= seg_lo && p < seg_hi) atomicOr(&bm[(p - seg_lo) >> 5], 1u << ((p - seg_lo) & 31));
    }
    const int nd = m * span;
    for (int j = tid; j < nd; j += BLOCK) {
      const int p = topk[j / span] + (j % span) - r;
      if (p >= seg_lo && p < seg_hi) atomicOr(&bm[(p - seg_lo) >> 5], 1u << ((p - seg_lo) & 31));
    }
    __syncthreads();
    // ordered compaction: thread t owns words [t*wpt, (t+1)*wpt)
    const int wpt = (nwords + BLOCK - 1) / BLOCK;
    const int w_begin = min(nwords, tid * wpt);
    const int w_end = min(nwords, w_begin + wpt);
    uint32_t cnt = 0;
    for (int w = w_begin; w < w_end; ++w) cnt += __popc(bm[w]);
    uint32_t total = 0;
    uint32_t off = block_exclusive_scan<BLOCK>(cnt, scan, &total);
    int o = pos + (int)off;
    for (int w = w_begin; w < w_end; ++w) {
      uint32_t bits = bm[w];
      while (bits) {
        const int bit = __ffs(bits) - 1;
        bits &= bits - 1u;
        if (o < set_cap) out[o] = seg_lo + (w << 5) + bit;
        ++o;
      }
    }
    pos += (int)total;
    __syncthreads();
  }

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

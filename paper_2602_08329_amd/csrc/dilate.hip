// Reuse step: the dilated shared set of a later decode step or of another
// layer in the anchor's group (Def. 3.2 key-value sharing; Eq. neighboring,
// neighbours clipped to the valid positions as in the CIS parameterisation
// appendix).  One workgroup per (batch, kv head); the set is built in LDS by
// build_index_set and depends only on the anchor's top-k and the lengths.
#include "prhs.h"
#include "prhs_internal.h"
#include "setops.h"

namespace prhs {
namespace {

constexpr int kDilateBlock = 1024;

__global__ __launch_bounds__(kDilateBlock) void dilate_reuse_kernel(DilateLaunch a) {
  extern __shared__ int32_t s_topk[];  // [k_cap] the row's top-k, staged once
  __shared__ uint32_t bm[kSegWords];
  __shared__ uint32_t scan[kDilateBlock / 64 + 1];
  const int row = blockIdx.x;
  const int b = row / a.hkv;
  int n = a.seq_lens[b];
  n = n < 0 ? 0 : n;
  int n0 = a.anchor_lens[b];
  n0 = n0 < 0 ? 0 : (n0 > n ? n : n0);
  const int sink_end = min(a.sink, n0);
  const int win_start = max(sink_end, n0 - a.window);
  // m = floor(k_b / 3) of the budget before clamping to the middle range
  // (or dilate_m), then clamped to the selected count
  long long kb = a.k_den > 0 ? ((long long)a.k_num * n0) / a.k_den : (long long)a.k;
  kb = kb < 0 ? 0 : kb;
  // prhs_select never selects more than PRHS_MAX_TOPK, the staging capacity
  const int stage_cap = a.k_cap < PRHS_MAX_TOPK ? a.k_cap : PRHS_MAX_TOPK;
  int klen = a.topk_len[row];
  klen = klen < 0 ? 0 : (klen > stage_cap ? stage_cap : klen);
  long long m = a.dilate_m < 0 ? kb / 3 : a.dilate_m;
  m = m > klen ? klen : m;
  const int32_t* topk = a.topk_idx + (size_t)row * a.k_cap;
  for (int j = threadIdx.x; j < klen; j += kDilateBlock) s_topk[j] = topk[j];
  __syncthreads();
  build_index_set<kDilateBlock>(s_topk, klen, (int)m, a.dilate_r,
                                sink_end, win_start, n, a.set_idx + (size_t)row * a.set_cap,
                                a.set_cap, a.set_len + row, bm, scan, kSegBits);
}

}  // namespace

hipError_t launch_dilate_reuse(const DilateLaunch& a, hipStream_t stream) {
  const int rows = a.batch * a.hkv;
  if (rows == 0) return hipSuccess;
  const int stage_cap = a.k_cap < PRHS_MAX_TOPK ? a.k_cap : PRHS_MAX_TOPK;
  const size_t dyn = (size_t)(stage_cap > 0 ? stage_cap : 1) * sizeof(int32_t);
  if (dyn + (size_t)kSegWords * 4 > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)dilate_reuse_kernel,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(dilate_reuse_kernel, dim3(rows), dim3(kDilateBlock), dyn, stream, a);
  return hipGetLastError();
}

}  // namespace prhs

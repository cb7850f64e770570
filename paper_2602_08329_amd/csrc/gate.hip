// Similarity gate of CIS (Sec. 4.1, Similarity Criteria; Eq. cos_sim).
//
// One wave per (batch, kv head) unit.  At block step `slot` > 0 a unit shares
// the selection of the most recent earlier step j of its block that
// retrieved for it and whose queries are similar to the current ones for
// every query head of the group; otherwise it retrieves now.  sim > tau is
// decided as dot > 0 and dot^2 > (tau^2 |q|^2) |q_j|^2 in binary64, from dot
// products and squared norms summed in fp32 (exact for inputs on a coarse
// grid, so the decision is reproducible).
//
// The kernel also records the step: the current queries become reference
// slot `slot`, ref_valid[slot] marks the units that retrieve, slot_lens[slot]
// the sequence lengths; and it resolves, per unit, which row of the set pool
// each layer attends and from which position the decoded tail starts.
#include "prhs.h"
#include "prhs_internal.h"

namespace prhs {
namespace {

template <typename T>
__device__ __forceinline__ float to_f32(T x);
template <>
__device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f32<__bf16>(__bf16 x) { return (float)x; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

template <typename T>
__global__ __launch_bounds__(64) void gate_kernel(GateLaunch a) {
  const int u = blockIdx.x;
  const int lane = threadIdx.x;
  const int units = a.batch * a.hkv;
  const int b = u / a.hkv, g = u % a.hkv;
  const int G = a.hq / a.hkv;
  const size_t qstride = (size_t)a.batch * a.hq * a.d;  // one slot of ref_q
  const T* q = (const T*)a.q;
  T* ref = (T*)a.ref_q;
  int choice = -1;
  for (int j = a.slot - 1; j >= 0 && choice < 0; --j) {
    if (a.ref_valid[(size_t)j * units + u] == 0) continue;
    bool all = true;
    for (int h = 0; h < G && all; ++h) {
      const size_t off = ((size_t)b * a.hq + g * G + h) * a.d;
      float dot = 0.f, nn = 0.f, nr = 0.f;
      for (int e = lane; e < a.d; e += 64) {
        const float x = to_f32(q[off + e]);
        const float y = to_f32(ref[(size_t)j * qstride + off + e]);
        dot = fmaf(x, y, dot);
        nn = fmaf(x, x, nn);
        nr = fmaf(y, y, nr);
      }
      const double dd = (double)wave_sum(dot);
      const double n1 = (double)wave_sum(nn), n2 = (double)wave_sum(nr);
      all = dd > 0.0 && dd * dd > (a.tau * a.tau) * n1 * n2;
    }
    if (all) choice = j;
  }
  // the current queries become reference slot `slot`
  for (int h = 0; h < G; ++h) {
    const size_t off = ((size_t)b * a.hq + g * G + h) * a.d;
    for (int e = lane; e < a.d; e += 64) ref[(size_t)a.slot * qstride + off + e] = q[off + e];
  }
  if (lane == 0) {
    const int src = choice < 0 ? a.slot : choice;
    a.ref_valid[(size_t)a.slot * units + u] = choice < 0 ? 1 : 0;
    a.choice[u] = choice;
    // pool rows: [kind][slot][unit] with kind 0 the critical set, 1 the
    // dilated shared set
    const int S = a.num_slots;
    a.row_anchor[u] = (choice < 0 ? a.slot : S + choice) * units + u;
    a.row_other[u] = (S + src) * units + u;
    int n = a.seq_lens[b];
    a.tail[u] = choice < 0 ? n : a.slot_lens[(size_t)choice * a.batch + b];
    if (g == 0) a.slot_lens[(size_t)a.slot * a.batch + b] = n;
  }
}

}  // namespace

hipError_t launch_gate(const GateLaunch& a, hipStream_t stream) {
  const int units = a.batch * a.hkv;
  if (units == 0) return hipSuccess;
  if (a.dtype == 1)
    hipLaunchKernelGGL(gate_kernel<__bf16>, dim3(units), dim3(64), 0, stream, a);
  else
    hipLaunchKernelGGL(gate_kernel<float>, dim3(units), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace prhs

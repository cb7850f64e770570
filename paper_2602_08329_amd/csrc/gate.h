// The similarity gate of CIS (Sec. 4.1, Similarity Criteria; Eq. cos_sim)
// for one (batch, kv head) unit, taken by one whole wave: shared by the gate
// kernel and the refresh kernels that take the decision themselves.
//
// At block step `slot` > 0 a unit shares the selection of the most recent
// earlier step j of its block that retrieved for it and whose queries are
// similar to the current ones for every query head of the group; otherwise
// it retrieves now.  sim > tau is decided as dot > 0 and dot^2 > (tau^2
// |q|^2) |q_j|^2 in binary64, from dot products and squared norms summed in
// fp32 (exact for inputs on a coarse grid, so the decision is reproducible).
//
// The decision resolves, per unit, which row of the set pool each layer
// attends and from which position the decoded tail starts.  With
// a.record the step is also recorded: the current queries become reference
// slot `slot`, ref_valid[slot] marks the units that retrieve, slot_lens[slot]
// the sequence lengths.
#pragma once

#include "prhs_internal.h"

namespace prhs {

template <typename T>
__device__ __forceinline__ float gate_to_f32(T x);
template <>
__device__ __forceinline__ float gate_to_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ float gate_to_f32<__bf16>(__bf16 x) { return (float)x; }

__device__ __forceinline__ float gate_wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Decides unit u and writes its choice, pool rows and tail start (and the
// step record with a.record).  Every lane of one wave must call it; returns
// the choice (the shared slot, or -1 to retrieve) in every lane.
template <typename T>
__device__ int gate_unit(const GateLaunch& a, int u, int lane) {
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
        const float x = gate_to_f32(q[off + e]);
        const float y = gate_to_f32(ref[(size_t)j * qstride + off + e]);
        dot = fmaf(x, y, dot);
        nn = fmaf(x, x, nn);
        nr = fmaf(y, y, nr);
      }
      const double dd = (double)gate_wave_sum(dot);
      const double n1 = (double)gate_wave_sum(nn), n2 = (double)gate_wave_sum(nr);
      all = dd > 0.0 && dd * dd > (a.tau * a.tau) * n1 * n2;
    }
    if (all) choice = j;
  }
  if (a.record) {
    for (int h = 0; h < G; ++h) {
      const size_t off = ((size_t)b * a.hq + g * G + h) * a.d;
      for (int e = lane; e < a.d; e += 64) ref[(size_t)a.slot * qstride + off + e] = q[off + e];
    }
  }
  if (lane == 0) {
    const int src = choice < 0 ? a.slot : choice;
    a.choice[u] = choice;
    // pool rows: [kind][slot][unit] with kind 0 the critical set, 1 the
    // dilated shared set
    const int S = a.num_slots;
    a.row_anchor[u] = (choice < 0 ? a.slot : S + choice) * units + u;
    a.row_other[u] = (S + src) * units + u;
    const int n = a.seq_lens[b];
    a.tail[u] = choice < 0 ? n : a.slot_lens[(size_t)choice * a.batch + b];
    if (a.record) {
      a.ref_valid[(size_t)a.slot * units + u] = choice < 0 ? 1 : 0;
      if (g == 0) a.slot_lens[(size_t)a.slot * a.batch + b] = n;
    }
  }
  return choice;
}

}  // namespace prhs

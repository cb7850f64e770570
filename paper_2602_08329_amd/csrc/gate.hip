// Similarity gate of CIS (Sec. 4.1, Similarity Criteria; Eq. cos_sim): one
// wave per (batch, kv head) unit takes the decision of gate.h.
#include "gate.h"
#include "prhs.h"

namespace prhs {
namespace {

template <typename T>
__global__ __launch_bounds__(64) void gate_kernel(GateLaunch a) {
  gate_unit<T>(a, blockIdx.x, threadIdx.x);
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

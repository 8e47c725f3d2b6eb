// Threshold gate of the meter loop (Sec. 6): a query head is gated when its
// certified meter exceeds tau (tau < 1), or its raw risk score does (tau >= 1,
// Sec. 4.3); a KV head is routed to the exact path when any of its G query
// heads is gated (the any-of-G statistic, Sec. 5).  One thread per (sequence,
// KV head); counts are reduced per wave before one atomic add.
#include "wc_device.h"
#include "wc_launch.h"

namespace wc {

namespace {

__global__ __launch_bounds__(256) void gate_kernel(GateArgs a) {
  const int item = blockIdx.x * blockDim.x + threadIdx.x;
  const int n_kv = a.n_q / a.group;
  int nq = 0, nk = 0;
  if (item < a.batch * n_kv) {
    const int b = item / n_kv, g = item % n_kv;
    const bool use_raw = a.tau >= 1.0f;
    int any = 0;
    for (int j = 0; j < a.group; ++j) {
      const int idx = b * a.n_q + g * a.group + j;
      const float v = use_raw ? a.raw[idx] : a.meter[idx];
      const int m = v > a.tau ? 1 : 0;
      a.mask_q[idx] = (uint8_t)m;
      nq += m;
      any |= m;
    }
    a.mask_kv[item] = (uint8_t)any;
    nk = any;
  }
  if (a.n_gated != nullptr) {
    for (int o = 32; o > 0; o >>= 1) {
      nq += __shfl_xor(nq, o, 64);
      nk += __shfl_xor(nk, o, 64);
    }
    if ((threadIdx.x & 63) == 0 && (nq | nk)) {
      atomicAdd(&a.n_gated[0], nq);
      atomicAdd(&a.n_gated[1], nk);
    }
  }
}

}  // namespace

hipError_t launch_gate(const GateArgs& a, hipStream_t st) {
  const int items = a.batch * (a.n_q / a.group);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(gate_kernel, dim3((items + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace wc

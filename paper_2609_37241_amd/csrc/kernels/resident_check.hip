// The check of the LDS channel of argument-free fused-chain launches: a
// kernel with the fused chain's largest static LDS reports the slot it reads
// back (the same decoding the chain uses) for launches that request
// slot * kLdsGranule bytes of dynamic LDS.
#include <hip/hip_runtime.h>

#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

namespace {
constexpr uint32_t kPadWords = 2052;   // 8208 bytes of static LDS

__global__ __launch_bounds__(64) void k_resident_check(uint32_t *out, uint32_t i) {
  __shared__ uint32_t pad[kPadWords];
  for (uint32_t j = threadIdx.x; j < kPadWords; j += 64) pad[j] = j;
  __syncthreads();
  // pad's last word keeps the array (and so the static LDS) alive
  if (threadIdx.x == 0) out[i] = resident_slot() + (pad[kPadWords - 1] - (kPadWords - 1));
}
}  // namespace

// Launches the check at slots 0, 1, 2 and the last one on the current
// device (synchronously, on a private stream). 0 when each launch read its
// own slot back, else TRI_E_RUNTIME.
int resident_check() {
  constexpr uint32_t kN = 4;
  const uint32_t slots[kN] = {0, 1, 2, kResidentSlots - 1};
  uint32_t *d = nullptr;
  if (hipMalloc(&d, kN * sizeof(uint32_t)) != hipSuccess) return TRI_E_RUNTIME;
  hipStream_t s = nullptr;
  bool ok = hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess;
  uint32_t h[kN] = {};
  ok = ok && hipMemsetAsync(d, 0xff, kN * sizeof(uint32_t), s) == hipSuccess;
  for (uint32_t i = 0; ok && i < kN; ++i) {
    hipLaunchKernelGGL(k_resident_check, dim3(1), dim3(64), slots[i] * kLdsGranule, s, d, i);
    ok = hipGetLastError() == hipSuccess;
  }
  ok = ok && hipMemcpyAsync(h, d, sizeof h, hipMemcpyDeviceToHost, s) == hipSuccess &&
       hipStreamSynchronize(s) == hipSuccess;
  if (s) (void)hipStreamDestroy(s);
  (void)hipFree(d);
  for (uint32_t i = 0; ok && i < kN; ++i) ok = h[i] == slots[i];
  return ok ? 0 : TRI_E_RUNTIME;
}

}  // namespace tri

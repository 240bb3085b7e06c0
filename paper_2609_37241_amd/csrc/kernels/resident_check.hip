// The check of the LDS channel of launches without kernel arguments: kernels
// with no static LDS, with a few bytes of it (the norm kernels' reductions)
// and with the fused chain's 8208 bytes report the slot they read back (the
// decoding every argument-free kernel uses) for launches that request
// slot * kLdsGranule bytes of dynamic LDS.
#include <hip/hip_runtime.h>

#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

namespace {
template <uint32_t W>
__global__ __launch_bounds__(64) void k_resident_check(uint32_t *out, uint32_t i) {
  if constexpr (W == 0) {
    if (threadIdx.x == 0) out[i] = resident_slot();
  } else {
    __shared__ uint32_t pad[W];
    for (uint32_t j = threadIdx.x; j < W; j += 64) pad[j] = j;
    __syncthreads();
    // pad's last word keeps the array (and so the static LDS) alive
    if (threadIdx.x == 0) out[i] = resident_slot() + (pad[W - 1] - (W - 1));
  }
}
}  // namespace

// Launches each check kernel at slots 0, 1, 2 and the last one on the
// current device (synchronously, on a private stream). 0 when every launch
// read its own slot back, else TRI_E_RUNTIME.
int resident_check() {
  constexpr uint32_t kSlotsChecked = 4, kForms = 3, kN = kSlotsChecked * kForms;
  const uint32_t slots[kSlotsChecked] = {0, 1, 2, kResidentSlots - 1};
  uint32_t *d = nullptr;
  if (hipMalloc(&d, kN * sizeof(uint32_t)) != hipSuccess) return TRI_E_RUNTIME;
  hipStream_t s = nullptr;
  bool ok = hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess;
  uint32_t h[kN] = {};
  ok = ok && hipMemsetAsync(d, 0xff, kN * sizeof(uint32_t), s) == hipSuccess;
  for (uint32_t k = 0; ok && k < kSlotsChecked; ++k) {
    const uint32_t dyn = slots[k] * kLdsGranule;
    hipLaunchKernelGGL(k_resident_check<0>, dim3(1), dim3(64), dyn, s, d, k);
    hipLaunchKernelGGL(k_resident_check<4>, dim3(1), dim3(64), dyn, s, d, kSlotsChecked + k);
    hipLaunchKernelGGL(k_resident_check<2052>, dim3(1), dim3(64), dyn, s, d,
                       2 * kSlotsChecked + k);
    ok = hipGetLastError() == hipSuccess;
  }
  ok = ok && hipMemcpyAsync(h, d, sizeof h, hipMemcpyDeviceToHost, s) == hipSuccess &&
       hipStreamSynchronize(s) == hipSuccess;
  if (s) (void)hipStreamDestroy(s);
  (void)hipFree(d);
  for (uint32_t i = 0; ok && i < kN; ++i) ok = h[i] == slots[i % kSlotsChecked];
  return ok ? 0 : TRI_E_RUNTIME;
}

}  // namespace tri

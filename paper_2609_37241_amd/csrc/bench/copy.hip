// Reference streaming copy for the benchmark: the practical HBM ceiling
// reported beside the path's kernels (a kernel that only moves bytes, with
// the same 16-byte vector access and 256-work-item workgroups).
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// U vectors per work-item per step, grid-stride; NT: nontemporal loads and
// stores. Every access is guarded by i < n.
template <int U, bool NT>
__global__ __launch_bounds__(256) void k_copy(const u32x4 *__restrict__ a, u32x4 *__restrict__ o,
                                              int64_t n) {
  const int64_t step = int64_t(gridDim.x) * 256 * U;
  for (int64_t base = int64_t(blockIdx.x) * 256 * U + threadIdx.x; base < n; base += step) {
    u32x4 v[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < n) v[k] = NT ? __builtin_nontemporal_load(a + i) : a[i];
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < n) {
        if (NT)
          __builtin_nontemporal_store(v[k], o + i);
        else
          o[i] = v[k];
      }
    }
  }
}

template <int U, bool NT>
int launch(const void *src, void *dst, int64_t n, hipStream_t s) {
  int64_t g = (n + 256 * U - 1) / (256 * U);
  if (g > (int64_t(1) << 20)) g = int64_t(1) << 20;
  k_copy<U, NT><<<dim3(uint32_t(g)), dim3(256), 0, s>>>(static_cast<const u32x4 *>(src),
                                                        static_cast<u32x4 *>(dst), n);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

extern "C" {

// Copy n16 16-byte vectors from src to dst (both 16-byte aligned) on
// `stream`. form 0: one vector per work-item; 1: two; 2: four,
// nontemporal. Returns 0, or -1 for bad arguments or a failed launch.
int trib_copy(const void *src, void *dst, int64_t n16, int form, void *stream) {
  if (!src || !dst || n16 < 1 || (uintptr_t(src) | uintptr_t(dst)) % 16) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (form) {
    case 0: return launch<1, false>(src, dst, n16, s);
    case 1: return launch<2, false>(src, dst, n16, s);
    case 2: return launch<4, true>(src, dst, n16, s);
    default: return -1;
  }
}

}  // extern "C"

// SwiGLU kernels, one per install-policy variant and dtype.
#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

template <int DT, int U, bool NT>
__global__ __launch_bounds__(256) void k_sw_flat(SwArgs a) {
  body_sw_flat<DT, U, NT>(a);
}

template <int DT>
__global__ __launch_bounds__(256) void k_sw_rows(SwArgs a) {
  body_sw_rows<DT>(a);
}

template <int DT>
__global__ __launch_bounds__(256) void k_sw_scalar(SwArgs a) {
  body_sw_scalar<DT>(a);
}

namespace {
template <int DT>
const void *sw_pick(int32_t variant) {
  switch (variant) {
    case SW_SCALAR: return reinterpret_cast<const void *>(&k_sw_scalar<DT>);
    case SW_FLAT: return reinterpret_cast<const void *>(&k_sw_flat<DT, 1, false>);
    case SW_FLAT_NT: return reinterpret_cast<const void *>(&k_sw_flat<DT, 1, true>);
    case SW_ROWS: return reinterpret_cast<const void *>(&k_sw_rows<DT>);
    default: return nullptr;
  }
}
}  // namespace

const void *sw_kernel(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return sw_pick<kF32>(variant);
  if (dtype == TRI_BF16) return sw_pick<kBF16>(variant);
  return nullptr;
}

}  // namespace tri

// SwiGLU kernels, one per install-policy variant and dtype, each also
// without kernel arguments (its block read from this device's resident
// table).
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

// Resident argument blocks of the SwiGLU kernels: one table per GPU, dtype
// major, zero at load. In host code the name stands for a host-side shadow;
// the host writes the table through its device address.
static __device__ __align__(256) ResidentBlock resident_swiglu[2 * kResidentSlots];

template <int DT, int U, bool NT>
__global__ __launch_bounds__(256) void k_sw_flat_res() {
  SwArgs a;
  uint32_t g;
  if (resident_args(resident_swiglu + DT * kResidentSlots, a, g)) body_sw_flat<DT, U, NT>(a, g);
}

template <int DT>
__global__ __launch_bounds__(256) void k_sw_rows_res() {
  SwArgs a;
  uint32_t g;
  if (resident_args(resident_swiglu + DT * kResidentSlots, a, g)) body_sw_rows<DT>(a, g);
}

template <int DT>
__global__ __launch_bounds__(256) void k_sw_scalar_res() {
  SwArgs a;
  uint32_t g;
  if (resident_args(resident_swiglu + DT * kResidentSlots, a, g)) body_sw_scalar<DT>(a, g);
}

namespace {
template <class F>
const void *sym(F *f) {
  return reinterpret_cast<const void *>(f);
}

template <int DT, bool R>
const void *sw_pick(int32_t variant) {
  if constexpr (R) {
    switch (variant) {
      case SW_SCALAR: return sym(&k_sw_scalar_res<DT>);
      case SW_FLAT: return sym(&k_sw_flat_res<DT, 1, false>);
      case SW_FLAT_NT: return sym(&k_sw_flat_res<DT, 1, true>);
      case SW_ROWS: return sym(&k_sw_rows_res<DT>);
      default: return nullptr;
    }
  } else {
    switch (variant) {
      case SW_SCALAR: return sym(&k_sw_scalar<DT>);
      case SW_FLAT: return sym(&k_sw_flat<DT, 1, false>);
      case SW_FLAT_NT: return sym(&k_sw_flat<DT, 1, true>);
      case SW_ROWS: return sym(&k_sw_rows<DT>);
      default: return nullptr;
    }
  }
}
}  // namespace

const void *sw_kernel(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return sw_pick<kF32, false>(variant);
  if (dtype == TRI_BF16) return sw_pick<kBF16, false>(variant);
  return nullptr;
}

// The same kernel without kernel arguments.
const void *sw_kernel_resident(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return sw_pick<kF32, true>(variant);
  if (dtype == TRI_BF16) return sw_pick<kBF16, true>(variant);
  return nullptr;
}

// Host shadow of the SwiGLU kernels' resident table (dtype-major).
const void *resident_symbol_swiglu() { return reinterpret_cast<const void *>(&resident_swiglu); }

}  // namespace tri

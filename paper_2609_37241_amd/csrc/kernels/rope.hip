// RoPE-on-Q-and-K kernels (in place), with and without the per-head QK
// RMSNorm, rotate-half or GPT-J pairs, one per install-policy variant and
// dtype (the scalar kernels take the pairing, position width and angle
// source at run time), each also without kernel arguments (its block read
// from this device's resident table).
#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

// QKN: per-head RMSNorm of Q and K before the rotation; INTER: GPT-J pairs.
template <int DT, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_rope_vec(RopeArgs a) {
  body_rope_vec<DT, QKN, INTER>(a);
}

template <int DT, bool QKN>
__global__ __launch_bounds__(256) void k_rope_scalar(RopeArgs a) {
  body_rope_scalar<DT, QKN>(a);
}

// Resident argument blocks of the RoPE kernels: one table per GPU, dtype
// major, zero at load. In host code the name stands for a host-side shadow;
// the host writes the table through its device address.
static __device__ __align__(256) ResidentBlock resident_rope[2 * kResidentSlots];

template <int DT, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_rope_vec_res() {
  RopeArgs a;
  uint32_t g;
  if (resident_args(resident_rope + DT * kResidentSlots, a, g)) body_rope_vec<DT, QKN, INTER>(a);
}

template <int DT, bool QKN>
__global__ __launch_bounds__(256) void k_rope_scalar_res() {
  RopeArgs a;
  uint32_t g;
  if (resident_args(resident_rope + DT * kResidentSlots, a, g)) body_rope_scalar<DT, QKN>(a);
}

namespace {
template <class F>
const void *sym(F *f) {
  return reinterpret_cast<const void *>(f);
}

template <int DT, bool R>
const void *rope_pick(int32_t variant) {
  if constexpr (R) {
    switch (variant) {
      case ROPE_SCALAR: return sym(&k_rope_scalar_res<DT, false>);
      case ROPE_VEC: return sym(&k_rope_vec_res<DT, false, false>);
      case ROPE_VEC_I: return sym(&k_rope_vec_res<DT, false, true>);
      case ROPE_QKN_SCALAR: return sym(&k_rope_scalar_res<DT, true>);
      case ROPE_QKN_VEC: return sym(&k_rope_vec_res<DT, true, false>);
      case ROPE_QKN_VEC_I: return sym(&k_rope_vec_res<DT, true, true>);
      default: return nullptr;
    }
  } else {
    switch (variant) {
      case ROPE_SCALAR: return sym(&k_rope_scalar<DT, false>);
      case ROPE_VEC: return sym(&k_rope_vec<DT, false, false>);
      case ROPE_VEC_I: return sym(&k_rope_vec<DT, false, true>);
      case ROPE_QKN_SCALAR: return sym(&k_rope_scalar<DT, true>);
      case ROPE_QKN_VEC: return sym(&k_rope_vec<DT, true, false>);
      case ROPE_QKN_VEC_I: return sym(&k_rope_vec<DT, true, true>);
      default: return nullptr;
    }
  }
}
}  // namespace

const void *rope_kernel(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return rope_pick<kF32, false>(variant);
  if (dtype == TRI_BF16) return rope_pick<kBF16, false>(variant);
  return nullptr;
}

// The same kernel without kernel arguments.
const void *rope_kernel_resident(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return rope_pick<kF32, true>(variant);
  if (dtype == TRI_BF16) return rope_pick<kBF16, true>(variant);
  return nullptr;
}

// Host shadow of the RoPE kernels' resident table (dtype-major).
const void *resident_symbol_rope() { return reinterpret_cast<const void *>(&resident_rope); }

}  // namespace tri

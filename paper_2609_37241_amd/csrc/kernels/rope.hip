// RoPE-on-Q-and-K kernels (in place), with and without the per-head QK
// RMSNorm, rotate-half or GPT-J pairs, one per install-policy variant and
// dtype (the scalar kernels take the pairing, position width and angle
// source at run time).
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

namespace {
template <int DT>
const void *rope_pick(int32_t variant) {
  switch (variant) {
    case ROPE_SCALAR: return reinterpret_cast<const void *>(&k_rope_scalar<DT, false>);
    case ROPE_VEC: return reinterpret_cast<const void *>(&k_rope_vec<DT, false, false>);
    case ROPE_VEC_I: return reinterpret_cast<const void *>(&k_rope_vec<DT, false, true>);
    case ROPE_QKN_SCALAR: return reinterpret_cast<const void *>(&k_rope_scalar<DT, true>);
    case ROPE_QKN_VEC: return reinterpret_cast<const void *>(&k_rope_vec<DT, true, false>);
    case ROPE_QKN_VEC_I: return reinterpret_cast<const void *>(&k_rope_vec<DT, true, true>);
    default: return nullptr;
  }
}
}  // namespace

const void *rope_kernel(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return rope_pick<kF32>(variant);
  if (dtype == TRI_BF16) return rope_pick<kBF16>(variant);
  return nullptr;
}

}  // namespace tri

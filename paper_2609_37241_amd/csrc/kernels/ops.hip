// Short ops of the paper's operator suite: silu, add and masked_fill over
// [T, W] and embedding rows, one kernel per install-policy variant, op and
// dtype.
#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

template <int DT, int OP, int U>
__global__ __launch_bounds__(256) void k_elt_flat(EltArgs a) {
  body_elt_flat<DT, OP, U>(a);
}

template <int DT, int OP>
__global__ __launch_bounds__(256) void k_elt_rows(EltArgs a) {
  body_elt_rows<DT, OP>(a);
}

template <int DT, int OP>
__global__ __launch_bounds__(256) void k_elt_scalar(EltArgs a) {
  body_elt_scalar<DT, OP>(a);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(256) void k_emb(EmbArgs a) {
  body_emb<DT, VEC>(a);
}

namespace {
template <int DT, int OP>
const void *elt_pick(int32_t variant) {
  switch (variant) {
    case ELT_SCALAR: return reinterpret_cast<const void *>(&k_elt_scalar<DT, OP>);
    case ELT_FLAT: return reinterpret_cast<const void *>(&k_elt_flat<DT, OP, 1>);
    case ELT_FLAT_U2: return reinterpret_cast<const void *>(&k_elt_flat<DT, OP, 2>);
    case ELT_ROWS: return reinterpret_cast<const void *>(&k_elt_rows<DT, OP>);
    default: return nullptr;
  }
}

template <int DT>
const void *elt_pick_op(int32_t variant, int32_t op) {
  switch (op) {
    case kOpSilu: return elt_pick<DT, kOpSilu>(variant);
    case kOpAdd: return elt_pick<DT, kOpAdd>(variant);
    case kOpMaskedFill: return elt_pick<DT, kOpMaskedFill>(variant);
    default: return nullptr;
  }
}
}  // namespace

// op: TRI_OP_SILU, TRI_OP_ADD or TRI_OP_MASKED_FILL.
const void *elt_kernel(int32_t variant, uint32_t dtype, int32_t op) {
  if (dtype == TRI_F32) return elt_pick_op<kF32>(variant, op);
  if (dtype == TRI_BF16) return elt_pick_op<kBF16>(variant, op);
  return nullptr;
}

const void *emb_kernel(int32_t variant, uint32_t dtype) {
  const bool vec = variant == EMB_VEC;
  if (variant != EMB_VEC && variant != EMB_SCALAR) return nullptr;
  if (dtype == TRI_F32)
    return vec ? reinterpret_cast<const void *>(&k_emb<kF32, true>)
               : reinterpret_cast<const void *>(&k_emb<kF32, false>);
  if (dtype == TRI_BF16)
    return vec ? reinterpret_cast<const void *>(&k_emb<kBF16, true>)
               : reinterpret_cast<const void *>(&k_emb<kBF16, false>);
  return nullptr;
}

}  // namespace tri

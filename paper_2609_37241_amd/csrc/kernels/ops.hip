// Short ops of the paper's operator suite: silu, add and masked_fill over
// [T, W] and embedding rows, one kernel per install-policy variant, op and
// dtype, each also without kernel arguments (its block read from this
// device's resident table of its family).
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

// Resident argument blocks of the element-wise and embedding kernels: one
// table per family and GPU, dtype major, zero at load. In host code the
// names stand for host-side shadows; the host writes the tables through
// their device addresses.
static __device__ __align__(256) ResidentBlock resident_elt[2 * kResidentSlots];
static __device__ __align__(256) ResidentBlock resident_emb[2 * kResidentSlots];

template <int DT, int OP, int U>
__global__ __launch_bounds__(256) void k_elt_flat_res() {
  EltArgs a;
  uint32_t g;
  if (resident_args(resident_elt + DT * kResidentSlots, a, g)) body_elt_flat<DT, OP, U>(a, g);
}

template <int DT, int OP>
__global__ __launch_bounds__(256) void k_elt_rows_res() {
  EltArgs a;
  uint32_t g;
  if (resident_args(resident_elt + DT * kResidentSlots, a, g)) body_elt_rows<DT, OP>(a, g);
}

template <int DT, int OP>
__global__ __launch_bounds__(256) void k_elt_scalar_res() {
  EltArgs a;
  uint32_t g;
  if (resident_args(resident_elt + DT * kResidentSlots, a, g)) body_elt_scalar<DT, OP>(a, g);
}

template <int DT, bool VEC>
__global__ __launch_bounds__(256) void k_emb_res() {
  EmbArgs a;
  uint32_t g;
  if (resident_args(resident_emb + DT * kResidentSlots, a, g)) body_emb<DT, VEC>(a, g);
}

namespace {
template <class F>
const void *sym(F *f) {
  return reinterpret_cast<const void *>(f);
}

template <int DT, int OP, bool R>
const void *elt_pick(int32_t variant) {
  if constexpr (R) {
    switch (variant) {
      case ELT_SCALAR: return sym(&k_elt_scalar_res<DT, OP>);
      case ELT_FLAT: return sym(&k_elt_flat_res<DT, OP, 1>);
      case ELT_FLAT_U2: return sym(&k_elt_flat_res<DT, OP, 2>);
      case ELT_ROWS: return sym(&k_elt_rows_res<DT, OP>);
      default: return nullptr;
    }
  } else {
    switch (variant) {
      case ELT_SCALAR: return sym(&k_elt_scalar<DT, OP>);
      case ELT_FLAT: return sym(&k_elt_flat<DT, OP, 1>);
      case ELT_FLAT_U2: return sym(&k_elt_flat<DT, OP, 2>);
      case ELT_ROWS: return sym(&k_elt_rows<DT, OP>);
      default: return nullptr;
    }
  }
}

template <int DT, bool R>
const void *elt_pick_op(int32_t variant, int32_t op) {
  switch (op) {
    case kOpSilu: return elt_pick<DT, kOpSilu, R>(variant);
    case kOpAdd: return elt_pick<DT, kOpAdd, R>(variant);
    case kOpMaskedFill: return elt_pick<DT, kOpMaskedFill, R>(variant);
    default: return nullptr;
  }
}

template <int DT, bool R>
const void *emb_pick(int32_t variant) {
  if (variant != EMB_VEC && variant != EMB_SCALAR) return nullptr;
  const bool vec = variant == EMB_VEC;
  if constexpr (R)
    return vec ? sym(&k_emb_res<DT, true>) : sym(&k_emb_res<DT, false>);
  else
    return vec ? sym(&k_emb<DT, true>) : sym(&k_emb<DT, false>);
}
}  // namespace

// op: TRI_OP_SILU, TRI_OP_ADD or TRI_OP_MASKED_FILL.
const void *elt_kernel(int32_t variant, uint32_t dtype, int32_t op) {
  if (dtype == TRI_F32) return elt_pick_op<kF32, false>(variant, op);
  if (dtype == TRI_BF16) return elt_pick_op<kBF16, false>(variant, op);
  return nullptr;
}

const void *elt_kernel_resident(int32_t variant, uint32_t dtype, int32_t op) {
  if (dtype == TRI_F32) return elt_pick_op<kF32, true>(variant, op);
  if (dtype == TRI_BF16) return elt_pick_op<kBF16, true>(variant, op);
  return nullptr;
}

const void *emb_kernel(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return emb_pick<kF32, false>(variant);
  if (dtype == TRI_BF16) return emb_pick<kBF16, false>(variant);
  return nullptr;
}

const void *emb_kernel_resident(int32_t variant, uint32_t dtype) {
  if (dtype == TRI_F32) return emb_pick<kF32, true>(variant);
  if (dtype == TRI_BF16) return emb_pick<kBF16, true>(variant);
  return nullptr;
}

// Host shadows of the element-wise and embedding kernels' resident tables
// (dtype-major).
const void *resident_symbol_elt() { return reinterpret_cast<const void *>(&resident_elt); }
const void *resident_symbol_emb() { return reinterpret_cast<const void *>(&resident_emb); }

}  // namespace tri

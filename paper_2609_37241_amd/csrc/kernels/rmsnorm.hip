// RMSNorm and residual-add + RMSNorm kernels, one per install-policy variant
// and dtype, each also without kernel arguments (its block read from this
// device's resident table). Row bodies live in device.h (shared with the
// fused chain).
#include <mutex>

#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

// The fixed exchange scratch of tri_residual_rmsnorm_noalloc: one copy per
// GPU, zero at load, left zero by every split call. In host code the name
// stands for a host-side shadow, not for device memory: kernels receive the
// device address looked up below, never the name.
static __device__ __align__(256) uint64_t scratch[kNoAllocScratchWords];

namespace {
std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
void *g_scratch_ptr[kMaxDevices];
int g_scratch_status[kMaxDevices];   // 0: not looked up; 1: found; -1: failed
}  // namespace

// Device address of `device`'s copy of `scratch`, looked up once per device
// with that device current (the caller's contract: cache creation).
int be_noalloc_scratch(int device, void **ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return TRI_E_RUNTIME;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_status[device] == 0) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_status[device] = e == hipSuccess && p ? 1 : -1;
    g_scratch_ptr[device] = g_scratch_status[device] == 1 ? p : nullptr;
  }
  *ptr = g_scratch_ptr[device];
  return g_scratch_status[device] == 1 ? 0 : TRI_E_RUNTIME;
}

template <int DT, int NV, bool RES>
__global__ __launch_bounds__(256) void k_rn_wave(RnArgs a) {
  body_rn_wave<DT, NV, RES>(a);
}

template <int DT, int NB, bool RES>
__global__ __launch_bounds__(256) void k_rn_block(RnArgs a) {
  body_rn_block<DT, NB, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(256) void k_rn_loop(RnArgs a) {
  body_rn_loop<DT, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(kWideLanes) void k_rn_wide(RnArgs a) {
  body_rn_wide<DT, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(256) void k_rn_split(RnSplitArgs a) {
  body_rn_split<DT, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(256) void k_rn_scalar(RnArgs a) {
  body_rn_scalar<DT, RES>(a);
}

// Resident argument blocks of the norm kernels: one table per GPU, dtype
// major, zero at load. In host code the name stands for a host-side shadow;
// the host writes the table through its device address.
static __device__ __align__(256) ResidentBlock resident_norm[2 * kResidentSlots];

template <int DT>
__device__ __forceinline__ const ResidentBlock *norm_table() {
  return resident_norm + DT * kResidentSlots;
}

template <int DT, int NV, bool RES>
__global__ __launch_bounds__(256) void k_rn_wave_res() {
  RnArgs a;
  uint32_t g;
  if (resident_args(norm_table<DT>(), a, g)) body_rn_wave<DT, NV, RES>(a);
}

template <int DT, int NB, bool RES>
__global__ __launch_bounds__(256) void k_rn_block_res() {
  RnArgs a;
  uint32_t g;
  if (resident_args(norm_table<DT>(), a, g)) body_rn_block<DT, NB, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(256) void k_rn_loop_res() {
  RnArgs a;
  uint32_t g;
  if (resident_args(norm_table<DT>(), a, g)) body_rn_loop<DT, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(kWideLanes) void k_rn_wide_res() {
  RnArgs a;
  uint32_t g;
  if (resident_args(norm_table<DT>(), a, g)) body_rn_wide<DT, RES>(a, g);
}

template <int DT, bool RES>
__global__ __launch_bounds__(256) void k_rn_split_res() {
  RnSplitArgs a;
  uint32_t g;
  if (resident_args(norm_table<DT>(), a, g)) body_rn_split<DT, RES>(a);
}

template <int DT, bool RES>
__global__ __launch_bounds__(256) void k_rn_scalar_res() {
  RnArgs a;
  uint32_t g;
  if (resident_args(norm_table<DT>(), a, g)) body_rn_scalar<DT, RES>(a);
}

namespace {
template <class F>
const void *sym(F *f) {
  return reinterpret_cast<const void *>(f);
}

template <int DT, bool RES>
const void *rn_pick(int32_t variant) {
  switch (variant) {
    case RN_SCALAR: return sym(&k_rn_scalar<DT, RES>);
    case RN_WAVE_1: return sym(&k_rn_wave<DT, 1, RES>);
    case RN_WAVE_2: return sym(&k_rn_wave<DT, 2, RES>);
    case RN_BLOCK_1: return sym(&k_rn_block<DT, 1, RES>);
    case RN_BLOCK_2: return sym(&k_rn_block<DT, 2, RES>);
    case RN_BLOCK_4: return sym(&k_rn_block<DT, 4, RES>);
    case RN_BLOCK_8: return sym(&k_rn_block<DT, 8, RES>);
    case RN_BLOCK_16: return sym(&k_rn_block<DT, 16, RES>);
    case RN_LOOP: return sym(&k_rn_loop<DT, RES>);
    case RN_WIDE: return sym(&k_rn_wide<DT, RES>);
    case RN_SPLIT: return sym(&k_rn_split<DT, RES>);
    default: return nullptr;
  }
}

template <int DT, bool RES>
const void *rn_pick_resident(int32_t variant) {
  switch (variant) {
    case RN_SCALAR: return sym(&k_rn_scalar_res<DT, RES>);
    case RN_WAVE_1: return sym(&k_rn_wave_res<DT, 1, RES>);
    case RN_WAVE_2: return sym(&k_rn_wave_res<DT, 2, RES>);
    case RN_BLOCK_1: return sym(&k_rn_block_res<DT, 1, RES>);
    case RN_BLOCK_2: return sym(&k_rn_block_res<DT, 2, RES>);
    case RN_BLOCK_4: return sym(&k_rn_block_res<DT, 4, RES>);
    case RN_BLOCK_8: return sym(&k_rn_block_res<DT, 8, RES>);
    case RN_BLOCK_16: return sym(&k_rn_block_res<DT, 16, RES>);
    case RN_LOOP: return sym(&k_rn_loop_res<DT, RES>);
    // the plain wide form holds its weights in 128 KiB of static LDS,
    // which leaves too little for the slot channel: kernel arguments only
    case RN_WIDE:
      if constexpr (RES) return sym(&k_rn_wide_res<DT, RES>);
      else return nullptr;
    case RN_SPLIT: return sym(&k_rn_split_res<DT, RES>);
    default: return nullptr;
  }
}
}  // namespace

// Host stub of the kernel for (variant, dtype, residual flavour).
const void *rn_kernel(int32_t variant, uint32_t dtype, int32_t res) {
  if (dtype == TRI_F32) return res ? rn_pick<kF32, true>(variant) : rn_pick<kF32, false>(variant);
  if (dtype == TRI_BF16) return res ? rn_pick<kBF16, true>(variant) : rn_pick<kBF16, false>(variant);
  return nullptr;
}

// The same kernel without kernel arguments.
const void *rn_kernel_resident(int32_t variant, uint32_t dtype, int32_t res) {
  if (dtype == TRI_F32)
    return res ? rn_pick_resident<kF32, true>(variant) : rn_pick_resident<kF32, false>(variant);
  if (dtype == TRI_BF16)
    return res ? rn_pick_resident<kBF16, true>(variant) : rn_pick_resident<kBF16, false>(variant);
  return nullptr;
}

// Host shadow of the norm kernels' resident table (dtype-major).
const void *resident_symbol_norm() { return reinterpret_cast<const void *>(&resident_norm); }

}  // namespace tri

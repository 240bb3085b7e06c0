// The fused decode-chain kernel (f32): one launch whose workgroups take the
// residual-RMSNorm, RoPE-QK and SwiGLU roles by blockIdx range. Instantiated
// for every (norm role variant, SwiGLU role) the install policy can pick, in
// two forms: with the argument block as the kernel argument, and without
// kernel arguments, reading the block from this device's resident table.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

// Resident argument blocks of this dtype's fused chain: one table per GPU,
// zero at load (every tag unset). In host code the name stands for a
// host-side shadow, not for device memory: the host writes the table through
// the device address looked up below, never through the name.
static __device__ __align__(256) ResidentChain resident_f32[kResidentSlots];

// RNV: RN_WAVE_1/2 (one wavefront per row) or RN_BLOCK_1..16 (one
// workgroup per row); SWV: SW_FLAT or SW_FLAT_NT; QKN: QK norm before the
// rotation; INTER: GPT-J pairs.
template <int DT, int RNV, int SWV, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_chain(ChainArgs a) {
  constexpr bool wave = RNV <= RN_WAVE_2;
  constexpr int n = wave ? 1 << (RNV - RN_WAVE_1) : 1 << (RNV - RN_BLOCK_1);
  body_chain<DT, wave, n, SWV == SW_FLAT_NT, QKN, INTER>(a, gridDim.x);
}

template <int DT, int RNV, int SWV, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_chain_res() {
  constexpr bool wave = RNV <= RN_WAVE_2;
  constexpr int n = wave ? 1 << (RNV - RN_WAVE_1) : 1 << (RNV - RN_BLOCK_1);
  body_chain_resident<DT, wave, n, SWV == SW_FLAT_NT, QKN, INTER>(resident_f32);
}

namespace {
template <bool RES, int RNV, bool QKN, bool INTER>
const void *chain_pick_sw(bool nt) {
  if constexpr (RES)
    return nt ? reinterpret_cast<const void *>(&k_chain_res<kF32, RNV, SW_FLAT_NT, QKN, INTER>)
              : reinterpret_cast<const void *>(&k_chain_res<kF32, RNV, SW_FLAT, QKN, INTER>);
  else
    return nt ? reinterpret_cast<const void *>(&k_chain<kF32, RNV, SW_FLAT_NT, QKN, INTER>)
              : reinterpret_cast<const void *>(&k_chain<kF32, RNV, SW_FLAT, QKN, INTER>);
}

template <bool RES, int RNV>
const void *chain_pick_rn(int32_t rope_bits, bool nt) {
  switch (rope_bits) {
    case 0: return chain_pick_sw<RES, RNV, false, false>(nt);
    case 1: return chain_pick_sw<RES, RNV, true, false>(nt);
    case 2: return chain_pick_sw<RES, RNV, false, true>(nt);
    default: return chain_pick_sw<RES, RNV, true, true>(nt);
  }
}

template <bool RES>
const void *chain_pick(int32_t sub) {
  const bool nt = sub & 1;
  const int32_t rb = (sub >> 1) & 3;   // bit 0: QK norm, bit 1: GPT-J pairs
  switch (RN_WAVE_1 + (sub >> 3)) {
    case RN_WAVE_1: return chain_pick_rn<RES, RN_WAVE_1>(rb, nt);
    case RN_WAVE_2: return chain_pick_rn<RES, RN_WAVE_2>(rb, nt);
    case RN_BLOCK_1: return chain_pick_rn<RES, RN_BLOCK_1>(rb, nt);
    case RN_BLOCK_2: return chain_pick_rn<RES, RN_BLOCK_2>(rb, nt);
    case RN_BLOCK_4: return chain_pick_rn<RES, RN_BLOCK_4>(rb, nt);
    case RN_BLOCK_8: return chain_pick_rn<RES, RN_BLOCK_8>(rb, nt);
    case RN_BLOCK_16: return chain_pick_rn<RES, RN_BLOCK_16>(rb, nt);
    default: return nullptr;
  }
}

std::mutex g_table_mu;
constexpr int kMaxDevices = 64;
void *g_table_ptr[kMaxDevices];
int g_table_status[kMaxDevices];   // 0: not looked up; 1: found; -1: failed
}  // namespace

// sub = (norm role - RN_WAVE_1) * 8 + 4 * (GPT-J pairs) + 2 * (QK norm)
//       + (SwiGLU role streams nontemporally).
const void *chain_kernel_f32(int32_t sub) { return chain_pick<false>(sub); }
const void *chain_kernel_resident_f32(int32_t sub) { return chain_pick<true>(sub); }

// Device address of `device`'s copy of the resident table, looked up once
// per device with that device current.
int chain_resident_table_f32(int device, void **ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return TRI_E_RUNTIME;
  std::lock_guard<std::mutex> lock(g_table_mu);
  if (g_table_status[device] == 0) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(resident_f32));
    g_table_status[device] = e == hipSuccess && p ? 1 : -1;
    g_table_ptr[device] = g_table_status[device] == 1 ? p : nullptr;
  }
  *ptr = g_table_ptr[device];
  return g_table_status[device] == 1 ? 0 : TRI_E_RUNTIME;
}

}  // namespace tri

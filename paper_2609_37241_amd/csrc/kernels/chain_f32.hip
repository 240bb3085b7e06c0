// The fused decode-chain kernel (f32): one launch whose workgroups take the
// residual-RMSNorm, RoPE-QK and SwiGLU roles by blockIdx range. Instantiated
// for every (norm role variant, SwiGLU role) the install policy can pick, in
// two forms: with the argument block as the kernel argument, and without
// kernel arguments, reading the block from this device's resident table.
#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

// RNV: RN_WAVE_1/2 (one wavefront per row) or RN_BLOCK_1..16 (one
// workgroup per row); SWV: SW_FLAT or SW_FLAT_NT; QKN: QK norm before the
// rotation; INTER: GPT-J pairs.
template <int DT, int RNV, int SWV, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_chain(ChainArgs a) {
  constexpr bool wave = RNV <= RN_WAVE_2;
  constexpr int n = wave ? 1 << (RNV - RN_WAVE_1) : 1 << (RNV - RN_BLOCK_1);
  body_chain<DT, wave, n, SWV == SW_FLAT_NT, QKN, INTER>(a, gridDim.x);
}

// Resident argument blocks of this dtype's fused chain: one table per GPU,
// zero at load (every tag unset). In host code the name stands for a
// host-side shadow, not for device memory: the host writes the table through
// its device address, never through the name.
static __device__ __align__(256) ResidentBlock resident_chain_f32[kResidentSlots];

template <int DT, int RNV, int SWV, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_chain_res() {
  constexpr bool wave = RNV <= RN_WAVE_2;
  constexpr int n = wave ? 1 << (RNV - RN_WAVE_1) : 1 << (RNV - RN_BLOCK_1);
  ChainArgs a;
  uint32_t g;
  if (resident_args(resident_chain_f32, a, g))
    body_chain<DT, wave, n, SWV == SW_FLAT_NT, QKN, INTER>(a, g);
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
}  // namespace

// sub = (norm role - RN_WAVE_1) * 8 + 4 * (GPT-J pairs) + 2 * (QK norm)
//       + (SwiGLU role streams nontemporally).
const void *chain_kernel_f32(int32_t sub) { return chain_pick<false>(sub); }
const void *chain_kernel_resident_f32(int32_t sub) { return chain_pick<true>(sub); }

// Host shadow of this dtype's resident table.
const void *resident_symbol_chain_f32() {
  return reinterpret_cast<const void *>(&resident_chain_f32);
}

}  // namespace tri

// The fused decode-chain kernel (bf16): one launch whose workgroups take the
// residual-RMSNorm, RoPE-QK and SwiGLU roles by blockIdx range. Instantiated
// for every (norm role variant, SwiGLU role) the install policy can pick.
#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

// RNV: RN_WAVE_1/2 (one wavefront per row) or RN_BLOCK_1..16 (one
// workgroup per row); the RoPE role takes one token per workgroup, with the
// per-head QK RMSNorm first when QKN and GPT-J pairs when INTER; SWV: SW_FLAT
// (one vector per work-item, cached) or SW_FLAT_U4_NT (four, streaming).
template <int DT, int RNV>
__device__ __forceinline__ void chain_norm_role(const ChainArgs &a, uint32_t blk) {
  if constexpr (RNV <= RN_WAVE_2) {
    rn_wave_block<DT, 1 << (RNV - RN_WAVE_1), true, false>(a.rn, blk);
  } else {
    __shared__ float red[4];
    rn_row_regs<DT, 1 << (RNV - RN_BLOCK_1), true, 256, false>(a.rn, blk, threadIdx.x, red);
  }
}

// Role order by blockIdx. Decode sizes (SW_FLAT): norm rows, RoPE tokens,
// then SwiGLU -- the norm and RoPE roles take about as long as SwiGLU but
// have far fewer workgroups, so dispatching them first shortens the critical
// path (2.75 vs 3.1 µs device time at 1 token). Streaming sizes
// (SW_FLAT_U4_NT): SwiGLU first, then norm, then RoPE (about 1 % faster at
// 8192 tokens than norm first).
template <int DT, int RNV, int SWV, bool QKN, bool INTER>
__global__ __launch_bounds__(256) void k_chain(ChainArgs a) {
  __shared__ float lds[2 * 256];
  const uint32_t b = blockIdx.x;
  const uint32_t R = a.rn_blocks, P = a.rope_blocks, S = gridDim.x - R - P;
  if constexpr (SWV == SW_FLAT_U4_NT) {
    if (b < S) {
      sw_flat_part<DT, 4, true>(a.sw, b, S);
    } else if (b < S + R) {
      chain_norm_role<DT, RNV>(a, b - S);
    } else {
      rope_vec_block<DT, 1, false, 4, QKN, INTER>(a.rope, b - S - R, lds);
    }
  } else {
    if (b < R) {
      chain_norm_role<DT, RNV>(a, b);
    } else if (b < R + P) {
      rope_vec_block<DT, 1, false, 4, QKN, INTER>(a.rope, b - R, lds);
    } else {
      sw_flat_part<DT, 1, false>(a.sw, b - R - P, S);
    }
  }
}

namespace {
template <int RNV, bool QKN, bool INTER>
const void *chain_pick_sw(bool u4) {
  return u4 ? reinterpret_cast<const void *>(&k_chain<kBF16, RNV, SW_FLAT_U4_NT, QKN, INTER>)
            : reinterpret_cast<const void *>(&k_chain<kBF16, RNV, SW_FLAT, QKN, INTER>);
}

template <int RNV>
const void *chain_pick_rn(int32_t rope_bits, bool u4) {
  switch (rope_bits) {
    case 0: return chain_pick_sw<RNV, false, false>(u4);
    case 1: return chain_pick_sw<RNV, true, false>(u4);
    case 2: return chain_pick_sw<RNV, false, true>(u4);
    default: return chain_pick_sw<RNV, true, true>(u4);
  }
}
}  // namespace

// sub = (norm role - RN_WAVE_1) * 8 + 4 * (GPT-J pairs) + 2 * (QK norm)
//       + (SwiGLU role streams four vectors per work-item).
const void *chain_kernel_bf16(int32_t sub) {
  const bool u4 = sub & 1;
  const int32_t rb = (sub >> 1) & 3;   // bit 0: QK norm, bit 1: GPT-J pairs
  switch (RN_WAVE_1 + (sub >> 3)) {
    case RN_WAVE_1: return chain_pick_rn<RN_WAVE_1>(rb, u4);
    case RN_WAVE_2: return chain_pick_rn<RN_WAVE_2>(rb, u4);
    case RN_BLOCK_1: return chain_pick_rn<RN_BLOCK_1>(rb, u4);
    case RN_BLOCK_2: return chain_pick_rn<RN_BLOCK_2>(rb, u4);
    case RN_BLOCK_4: return chain_pick_rn<RN_BLOCK_4>(rb, u4);
    case RN_BLOCK_8: return chain_pick_rn<RN_BLOCK_8>(rb, u4);
    case RN_BLOCK_16: return chain_pick_rn<RN_BLOCK_16>(rb, u4);
    default: return nullptr;
  }
}

}  // namespace tri

// The fused decode-chain kernel (f32): one launch whose workgroups take the
// residual-RMSNorm, RoPE-QK and SwiGLU roles by blockIdx range. Instantiated
// for every (rows per lane, RoPE tokens per workgroup, SwiGLU unroll) the
// install policy can pick.
#include "../internal.h"
#include "device.h"

namespace tri {
using namespace dev;

template <int DT, int NV, int TPB, int U>
__global__ __launch_bounds__(256) void k_chain(ChainArgs a) {
  __shared__ float lds[2 * TPB * 256];
  const uint32_t b = blockIdx.x;
  if (b < a.rn_blocks) {
    rn_wave_block<DT, NV, true>(a.rn, b);
    return;
  }
  const uint32_t b1 = b - a.rn_blocks;
  if (b1 < a.rope_blocks) {
    rope_vec_block<DT, TPB>(a.rope, b1, lds);
    return;
  }
  sw_flat_part<DT, U>(a.sw, b1 - a.rope_blocks, gridDim.x - a.rn_blocks - a.rope_blocks);
}

namespace {
template <int DT, int NV>
const void *chain_pick_nv(bool t4, bool u4) {
  if (t4) return u4 ? reinterpret_cast<const void *>(&k_chain<DT, NV, 4, 4>)
                    : reinterpret_cast<const void *>(&k_chain<DT, NV, 4, 1>);
  return u4 ? reinterpret_cast<const void *>(&k_chain<DT, NV, 1, 4>)
            : reinterpret_cast<const void *>(&k_chain<DT, NV, 1, 1>);
}
}  // namespace

// sub = (index of NV in 1,2,4,8,16) * 4 + (4 RoPE tokens per block) * 2 + (SwiGLU unroll 4).
const void *chain_kernel_f32(int32_t sub) {
  const bool t4 = (sub >> 1) & 1, u4 = sub & 1;
  switch (sub >> 2) {
    case 0: return chain_pick_nv<kF32, 1>(t4, u4);
    case 1: return chain_pick_nv<kF32, 2>(t4, u4);
    case 2: return chain_pick_nv<kF32, 4>(t4, u4);
    case 3: return chain_pick_nv<kF32, 8>(t4, u4);
    case 4: return chain_pick_nv<kF32, 16>(t4, u4);
    default: return nullptr;
  }
}

}  // namespace tri

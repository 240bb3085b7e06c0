// Device-side building blocks shared by the standalone kernels and the fused
// decode-chain kernel: 16-byte packed element access, wavefront / workgroup
// reductions, and the per-role bodies. A role body is the same inlined code
// in both places, so the fused chain computes exactly what the three
// separate launches compute.
//
// Layout conventions: every workgroup has 256 work-items (4 wavefronts of
// 64). A "vector" is 16 bytes: 4 float32 or 8 bfloat16 elements, loaded and
// stored with one global_load/store_dwordx4 per lane.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../kernargs.h"

namespace tri {
namespace dev {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kF32 = 0, kBF16 = 1;
constexpr int kThreads = 256;

template <int DT>
struct Elt;

template <>
struct Elt<kF32> {
  static constexpr int V = 4;
  static constexpr int ES = 4;
  __device__ static inline void unpack(const u32x4 &p, float *f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(p[i]);
  }
  __device__ static inline u32x4 pack(const float *f) {
    u32x4 p;
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = __float_as_uint(f[i]);
    return p;
  }
  __device__ static inline float ld(const void *b, int64_t i) {
    return static_cast<const float *>(b)[i];
  }
  __device__ static inline void st(void *b, int64_t i, float v) { static_cast<float *>(b)[i] = v; }
  __device__ static inline float round(float v) { return v; }
};

template <>
struct Elt<kBF16> {
  static constexpr int V = 8;
  static constexpr int ES = 2;
  // bf16 -> f32 is exact: the bf16 bits are the upper half of the f32 bits.
  __device__ static inline void unpack(const u32x4 &p, float *f) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f[2 * j] = __uint_as_float(p[j] << 16);
      f[2 * j + 1] = __uint_as_float(p[j] & 0xFFFF0000u);
    }
  }
  // f32 -> bf16 round-to-nearest-even, two at a time (v_cvt_pk_bf16_f32).
  __device__ static inline uint32_t pack2(float a, float b) {
    const f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
  }
  __device__ static inline u32x4 pack(const float *f) {
    u32x4 p;
#pragma unroll
    for (int j = 0; j < 4; ++j) p[j] = pack2(f[2 * j], f[2 * j + 1]);
    return p;
  }
  __device__ static inline float ld(const void *b, int64_t i) {
    return __uint_as_float(uint32_t(static_cast<const uint16_t *>(b)[i]) << 16);
  }
  __device__ static inline void st(void *b, int64_t i, float v) {
    static_cast<uint16_t *>(b)[i] = uint16_t(pack2(v, 0.0f) & 0xFFFFu);
  }
  __device__ static inline float round(float v) {
    return __uint_as_float(pack2(v, 0.0f) << 16);
  }
};

// 16-byte global access; NT marks streaming data (nontemporal: the line is
// not kept in the caches for reuse), used where the working set is far larger
// than the caches.
template <bool NT>
__device__ inline u32x4 ld16(const u32x4 *p) {
  if constexpr (NT)
    return __builtin_nontemporal_load(p);
  else
    return *p;
}

template <bool NT>
__device__ inline void st16(u32x4 *p, const u32x4 &v) {
  if constexpr (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

// ---- reductions ----------------------------------------------------------------
// DPP move within a row of 16 lanes (every source lane is in range for the
// controls used here, so no lane reads an out-of-row value).
template <int CTRL>
__device__ inline float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes of a wavefront (all lanes active). Within each row of
// 16 lanes: exchange with lane^1 and lane^2 (quad permutes), then with the
// mirrored lane in each half row and in the row, so every lane holds its
// row's sum; the four row sums are read from lanes 0, 16, 32, 48 and added in
// a fixed order. Every lane returns the same, bitwise equal total.
__device__ inline float wave_sum(float v) {
  v += dpp_mov<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);   // row_half_mirror
  v += dpp_mov<0x140>(v);   // row_mirror
  const int b = __float_as_int(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(b, 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(b, 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(b, 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(b, 48));
  return (r0 + r1) + (r2 + r3);
}

// float64 butterfly over the 64 lanes (long-row and scalar norm paths).
__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over aligned groups of n consecutive lanes (n a power of two, at most
// 64, the same for the whole wavefront); every lane of a group returns the
// same, bitwise equal sum. Lanes of one group must be active together.
__device__ inline float group_sum(float v, int n) {
  if (n >= 2) v += dpp_mov<0xB1>(v);    // lane ^ 1
  if (n >= 4) v += dpp_mov<0x4E>(v);    // lane ^ 2
  if (n >= 8) v += dpp_mov<0x141>(v);   // the other quad of the half row
  if (n >= 16) v += dpp_mov<0x140>(v);  // the other half row
  if (n >= 32) v += __shfl_xor(v, 16, 64);
  if (n >= 64) v += __shfl_xor(v, 32, 64);
  return v;
}

// Sum over the NW wavefronts of a workgroup (256 work-items by default);
// `red` is NW words of LDS. The wavefront sums are added in a fixed order.
template <int NW = 4, typename T>
__device__ inline T block_sum(T v, T *red) {
  v = wave_sum(v);
  const int wid = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wid] = v;
  __syncthreads();
  T s;
  if constexpr (NW == 4) {
    s = (red[0] + red[1]) + (red[2] + red[3]);
  } else {
    s = red[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) s += red[i];
  }
  __syncthreads();
  return s;
}

// ---- RMSNorm / residual RMSNorm --------------------------------------------------
// One row held in registers: lane `lane` of LANES owns vectors lane + LANES*k,
// k < NV. With RES, h = RN(x + r) is written to res_out and normalised.
// LANES = 64: one wavefront per row, no barrier. LANES = 256 or kWideLanes:
// one workgroup of that many work-items.
// Without NT (decode sizes) the weight vectors are requested together with the
// row, so the row costs one memory round trip; with NT (streaming sizes) they
// are loaded after the reduction to keep fewer registers live.
template <int DT, int NV, bool RES, int LANES, bool NT>
__device__ __forceinline__ void rn_row_regs(const RnArgs &a, int64_t row, int lane, float *red) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  const int nvec = a.H / V;
  const u32x4 *xr = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.x) +
                                                     row * a.x_rs * E::ES);
  const u32x4 *wr = static_cast<const u32x4 *>(a.w);
  u32x4 xv[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int vi = lane + LANES * k;
    xv[k] = vi < nvec ? ld16<NT>(xr + vi) : u32x4{0, 0, 0, 0};
  }
  u32x4 rv[RES ? NV : 1];
  if constexpr (RES) {
    const u32x4 *rr = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.res) +
                                                       row * a.res_rs * E::ES);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int vi = lane + LANES * k;
      rv[k] = vi < nvec ? ld16<NT>(rr + vi) : u32x4{0, 0, 0, 0};
    }
  }
  u32x4 wv[NT ? 1 : NV];
  if constexpr (!NT) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int vi = lane + LANES * k;
      wv[k] = vi < nvec ? wr[vi] : u32x4{0, 0, 0, 0};
    }
  }
  if constexpr (RES) {
    u32x4 *orow = reinterpret_cast<u32x4 *>(static_cast<char *>(a.res_out) + row * a.ro_rs * E::ES);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      float f[V], g[V];
      E::unpack(xv[k], f);
      E::unpack(rv[k], g);
#pragma unroll
      for (int e = 0; e < V; ++e) f[e] += g[e];
      xv[k] = E::pack(f);
      const int vi = lane + LANES * k;
      if (vi < nvec) st16<NT>(orow + vi, xv[k]);
    }
  }
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float f[V];
    E::unpack(xv[k], f);
#pragma unroll
    for (int e = 0; e < V; ++e) ss = __builtin_fmaf(f[e], f[e], ss);
  }
  if constexpr (LANES == 64)
    ss = wave_sum(ss);
  else
    ss = block_sum<LANES / 64>(ss, red);
  const float inv = rsqrtf(ss / float(a.H) + a.eps);
  u32x4 *yr = reinterpret_cast<u32x4 *>(static_cast<char *>(a.y) + row * a.y_rs * E::ES);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int vi = lane + LANES * k;
    if (vi < nvec) {
      float f[V], w[V];
      E::unpack(xv[k], f);
      if constexpr (NT)
        E::unpack(wr[vi], w);
      else
        E::unpack(wv[k], w);
#pragma unroll
      for (int e = 0; e < V; ++e) f[e] = (f[e] * inv) * w[e];
      st16<NT>(yr + vi, E::pack(f));
    }
  }
}

// Workgroup `blk` of the one-wavefront-per-row layout: rows 4*blk .. 4*blk+3.
template <int DT, int NV, bool RES, bool NT>
__device__ __forceinline__ void rn_wave_block(const RnArgs &a, int64_t blk) {
  const int64_t row = blk * 4 + (threadIdx.x >> 6);
  if (row >= a.T) return;
  rn_row_regs<DT, NV, RES, 64, NT>(a, row, threadIdx.x & 63, nullptr);
}

// ---- split rows -------------------------------------------------------------------
// A row of nvec vectors is split over S = ceil(nvec / kSplitSpan)
// consecutive workgroups (workgroup b: row b / S, slice b % S of
// kSplitVecs vectors per work-item). Each holds its slice in registers,
// reduces its partial sum of squares, publishes it in the row's slot of the
// scratch buffer and waits until all S slots of the row are full; every
// workgroup of the row then adds the S partials in the same order (one
// wavefront, lanes 0..S-1), so all of them normalise with the same total.
// The row is read once and written once: nothing is re-read.
//
// Slots carry their own "full" bit, so the exchange needs no memory fence:
// a slot is one relaxed device-scope 64-bit atomic, and nothing else is
// communicated. The row's last reader (a per-row counter reaching S)
// clears the row's slots and counter, so the scratch is all zero again when
// the kernel ends, ready for the next call on the stream. No counter is
// shared between rows: atomics on one address serialise, and a ticket or
// completion counter for the whole grid measured 5-20x slower.
//
// The wait relies on the S workgroups of a row being resident together:
// they are consecutive in dispatch order, so once the earlier ones run the
// later ones are next in line (S <= 64, far below the workgroups the GPU
// holds). As a guard against anything else occupying the GPU indefinitely,
// the wait is bounded (kSplitSpinMax polls, several hundred milliseconds):
// a row whose partials do not all arrive is written as NaN and sets the
// sticky failure flag in header word 0, after which every call on that
// scratch writes NaN rows instead of trusting the exchange. A failure is
// therefore loud and never silent.
constexpr int kSplitSpinMax = 1 << 18;
constexpr uint64_t kSlotFull = uint64_t(1) << 63;

template <int DT, bool RES>
__device__ __forceinline__ void rn_split_row(const RnArgs &a, uint64_t *scratch) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  constexpr int NB = kSplitVecs;
  __shared__ float red[4];
  __shared__ float total;
  const int nvec = a.H / V;
  const int S = (nvec + kSplitSpan - 1) / kSplitSpan;
  const int64_t row = int64_t(blockIdx.x) / S;
  const int s = int(int64_t(blockIdx.x) - row * S);
  uint64_t *slots = scratch + kSplitHeaderWords + row * S;
  uint64_t *count = scratch + kSplitHeaderWords + a.T * S + row;
  const int v0 = s * kSplitSpan + int(threadIdx.x);
  const u32x4 *xr = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.x) +
                                                     row * a.x_rs * E::ES);
  const u32x4 *wr = static_cast<const u32x4 *>(a.w);
  u32x4 xv[NB], wv[NB];
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    const int vi = v0 + 256 * k;
    xv[k] = vi < nvec ? xr[vi] : u32x4{0, 0, 0, 0};
  }
  if constexpr (RES) {
    const u32x4 *rr = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.res) +
                                                       row * a.res_rs * E::ES);
    u32x4 *orow = reinterpret_cast<u32x4 *>(static_cast<char *>(a.res_out) + row * a.ro_rs * E::ES);
    u32x4 rv[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int vi = v0 + 256 * k;
      rv[k] = vi < nvec ? rr[vi] : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      float f[V], g[V];
      E::unpack(xv[k], f);
      E::unpack(rv[k], g);
#pragma unroll
      for (int e = 0; e < V; ++e) f[e] += g[e];
      xv[k] = E::pack(f);
      const int vi = v0 + 256 * k;
      if (vi < nvec) orow[vi] = xv[k];
    }
  }
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    const int vi = v0 + 256 * k;
    wv[k] = vi < nvec ? wr[vi] : u32x4{0, 0, 0, 0};
  }
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    float f[V];
    E::unpack(xv[k], f);
#pragma unroll
    for (int e = 0; e < V; ++e) ss = __builtin_fmaf(f[e], f[e], ss);
  }
  ss = block_sum(ss, red);
  if (threadIdx.x < 64) {   // one whole wavefront: the exchange
    const int lane = int(threadIdx.x);
    float sum = __builtin_nanf("");
    if (scratch[0] == 0) {
      if (lane == 0)
        __hip_atomic_store(&slots[s], kSlotFull | __float_as_uint(ss), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      bool have = lane >= S;
      float part = 0.0f;
      bool late = false;
      for (int it = 0;; ++it) {
        if (!have) {
          const uint64_t w = __hip_atomic_load(&slots[lane], __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
          if (w & kSlotFull) {
            have = true;
            part = __uint_as_float(uint32_t(w));
          }
        }
        if (__all(have)) break;
        if (it >= kSplitSpinMax) {
          late = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      sum = wave_sum(part);
      if (lane == 0) {
        if (late) {
          sum = __builtin_nanf("");
          __hip_atomic_store(&scratch[0], uint64_t(1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        const uint64_t c = __hip_atomic_fetch_add(count, uint64_t(1), __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        if (c == uint64_t(S) - 1) {   // the row's last reader: clear for the next call
          for (int j = 0; j < S; ++j)
            __hip_atomic_store(&slots[j], uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(count, uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
    if (lane == 0) total = sum;
  }
  __syncthreads();
  const float inv = rsqrtf(total / float(a.H) + a.eps);
  u32x4 *yr = reinterpret_cast<u32x4 *>(static_cast<char *>(a.y) + row * a.y_rs * E::ES);
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    const int vi = v0 + 256 * k;
    if (vi < nvec) {
      float f[V], w[V];
      E::unpack(xv[k], f);
      E::unpack(wv[k], w);
#pragma unroll
      for (int e = 0; e < V; ++e) f[e] = (f[e] * inv) * w[e];
      yr[vi] = E::pack(f);
    }
  }
}

// Vectors a work-item keeps in flight in the long-row kernels' streaming
// passes (one 16-byte load each, all issued before any is used).
constexpr int kRnBatch = 8;

// Long rows: two passes over global memory with float64 accumulation (each
// thread sums up to H/256 elements, so a float32 running sum would lose
// accuracy at the largest H). Vector form (16-byte aligned rows). Both passes
// keep kRnBatch vectors per work-item in flight; pass 2 re-reads x (or h from
// res_out: the thread's own writes).
template <int DT, bool RES>
__device__ __forceinline__ void rn_loop_row(const RnArgs &a, int64_t row, double *red) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  constexpr int B = kRnBatch;
  const int nvec = a.H / V;
  const u32x4 *xr = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.x) +
                                                     row * a.x_rs * E::ES);
  const u32x4 *src = xr;
  double ss = 0.0;
  if constexpr (RES) {
    const u32x4 *rr = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.res) +
                                                       row * a.res_rs * E::ES);
    u32x4 *orow = reinterpret_cast<u32x4 *>(static_cast<char *>(a.res_out) + row * a.ro_rs * E::ES);
    for (int base = threadIdx.x; base < nvec; base += kThreads * B) {
      u32x4 xv[B], rv[B];
#pragma unroll
      for (int k = 0; k < B; ++k) {
        const int vi = base + k * kThreads;
        if (vi < nvec) {
          xv[k] = xr[vi];
          rv[k] = rr[vi];
        }
      }
#pragma unroll
      for (int k = 0; k < B; ++k) {
        const int vi = base + k * kThreads;
        if (vi < nvec) {
          float f[V], g[V];
          E::unpack(xv[k], f);
          E::unpack(rv[k], g);
#pragma unroll
          for (int e = 0; e < V; ++e) f[e] += g[e];
          const u32x4 h = E::pack(f);
          orow[vi] = h;
          E::unpack(h, f);
#pragma unroll
          for (int e = 0; e < V; ++e) ss += double(f[e]) * double(f[e]);
        }
      }
    }
    src = orow;
  } else {
    for (int base = threadIdx.x; base < nvec; base += kThreads * B) {
      u32x4 xv[B];
#pragma unroll
      for (int k = 0; k < B; ++k) {
        const int vi = base + k * kThreads;
        if (vi < nvec) xv[k] = xr[vi];
      }
#pragma unroll
      for (int k = 0; k < B; ++k) {
        const int vi = base + k * kThreads;
        if (vi < nvec) {
          float f[V];
          E::unpack(xv[k], f);
#pragma unroll
          for (int e = 0; e < V; ++e) ss += double(f[e]) * double(f[e]);
        }
      }
    }
  }
  ss = block_sum(ss, red);
  const float inv = float(1.0 / sqrt(ss / double(a.H) + double(a.eps)));
  const u32x4 *wr = static_cast<const u32x4 *>(a.w);
  u32x4 *yr = reinterpret_cast<u32x4 *>(static_cast<char *>(a.y) + row * a.y_rs * E::ES);
  for (int base = threadIdx.x; base < nvec; base += kThreads * B) {
    u32x4 hv[B], wv[B];
#pragma unroll
    for (int k = 0; k < B; ++k) {
      const int vi = base + k * kThreads;
      if (vi < nvec) {
        hv[k] = src[vi];
        wv[k] = wr[vi];
      }
    }
#pragma unroll
    for (int k = 0; k < B; ++k) {
      const int vi = base + k * kThreads;
      if (vi < nvec) {
        float f[V], w[V];
        E::unpack(hv[k], f);
        E::unpack(wv[k], w);
#pragma unroll
        for (int e = 0; e < V; ++e) f[e] = (f[e] * inv) * w[e];
        yr[vi] = E::pack(f);
      }
    }
  }
}

// Any alignment: element-wise two-pass row, float64 accumulation.
template <int DT, bool RES>
__device__ __forceinline__ void rn_scalar_row(const RnArgs &a, int64_t row, double *red) {
  using E = Elt<DT>;
  const int H = a.H;
  const char *xr = static_cast<const char *>(a.x) + row * a.x_rs * E::ES;
  const char *src = xr;
  double ss = 0.0;
  if constexpr (RES) {
    const char *rr = static_cast<const char *>(a.res) + row * a.res_rs * E::ES;
    char *orow = static_cast<char *>(a.res_out) + row * a.ro_rs * E::ES;
    for (int j = threadIdx.x; j < H; j += kThreads) {
      const float h = E::round(E::ld(xr, j) + E::ld(rr, j));
      E::st(orow, j, h);
      ss += double(h) * double(h);
    }
    src = orow;
  } else {
    for (int j = threadIdx.x; j < H; j += kThreads) {
      const float v = E::ld(xr, j);
      ss += double(v) * double(v);
    }
  }
  ss = block_sum(ss, red);
  const float inv = float(1.0 / sqrt(ss / double(H) + double(a.eps)));
  char *yr = static_cast<char *>(a.y) + row * a.y_rs * E::ES;
  for (int j = threadIdx.x; j < H; j += kThreads)
    E::st(yr, j, (E::ld(src, j) * inv) * E::ld(a.w, j));
}

// ---- RoPE ---------------------------------------------------------------------
// Angles: theta = float(pos) * inv_i (one float32 product; int64 positions
// convert with one rounding) and cos / sin of it, or cos / sin read from the
// caller's cache row min(max(pos, 0), cs_len - 1). They are computed once per
// (token, pair) into LDS; every head of the token reuses them.
__device__ __forceinline__ int64_t rope_pos(const RopeArgs &a, int64_t t) {
  return (a.mode & kRopePos64) ? static_cast<const int64_t *>(a.pos)[t]
                               : int64_t(static_cast<const int32_t *>(a.pos)[t]);
}

__device__ __forceinline__ void rope_cos_sin(const RopeArgs &a, int64_t t, int i, float &c,
                                             float &s) {
  const int64_t p = rope_pos(a, t);
  if (a.mode & kRopeCache) {
    const int64_t r = p < 0 ? 0 : (p >= a.cs_len ? a.cs_len - 1 : p);
    const float *row = a.cos_sin + r * a.rd;
    c = row[i];
    s = row[(a.rd >> 1) + i];
  } else {
    sincosf(float(p) * a.inv_freq[i], &s, &c);
  }
}

// The rotation of a pair (x, y) by (c, s): x c - y s and y c + x s, each one
// fused multiply-add on a rounded product (device code is compiled without
// contraction, so these are the only fused operations and their rounding
// does not depend on the surrounding code).
__device__ __forceinline__ float rot_a(float x, float y, float c, float s) {
  return __builtin_fmaf(x, c, -(y * s));
}
__device__ __forceinline__ float rot_b(float x, float y, float c, float s) {
  return __builtin_fmaf(y, c, x * s);
}

__device__ __forceinline__ char *rope_head(const RopeArgs &a, int64_t t, int h, int es) {
  return h < a.nq ? static_cast<char *>(a.q) + (t * a.q_ts + int64_t(h) * a.hd) * es
                  : static_cast<char *>(a.k) + (t * a.k_ts + int64_t(h - a.nq) * a.hd) * es;
}

// tpb tokens per workgroup (mode bits 16..23, at most kRopeTokensMax; `lds`
// holds 2 * 256 * kRopeTokensMax floats); with one token per workgroup a
// token's heads may instead be split round-robin over S = slices workgroups
// (mode bits 8..15: workgroup blk takes token blk / S and heads s, s + S,
// s + 2S, ... with s = blk % S). P2 = rd/2 angle
// pairs per token (a power of two). Rotate-half (INTER false): each half of the rotated span is
// cpb = P2/V 16-byte vectors and a work-item holds chunk c of both halves;
// GPT-J pairs (INTER true): the span is cpb = rd/V vectors of V/2 adjacent
// pairs each and a work-item holds one. Work-item `tid` owns chunk tid % cpb
// of heads tid / cpb, tid / cpb + 256 / cpb, ... of every token of the
// block. Its (token, head) items are processed PF at a time with all loads
// issued before any use, and the first batch is requested before the angle
// math and the barrier, so at decode sizes the block costs one memory round
// trip. Elements past rd are not touched.
//
// QKN (requires rd == hd): each head is first RMS-normalised over its hd
// elements with the Q or K head-norm weight. The cpb work-items of a head
// hold the whole head in registers, so the sum of squares is a reduction
// over cpb adjacent lanes and the head is read and written once. Whether an
// item is valid depends only on the work-item's head group, so the lanes of
// a group skip or process an item together and every lane a reduction reads
// from is active. cpb <= 64 (the policy guarantees it).
template <int DT, bool NT, int PF = 4, bool QKN = false, bool INTER = false>
__device__ __forceinline__ void rope_vec_block(const RopeArgs &a, int64_t blk, float *lds) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  const int P2 = a.rd >> 1;
  const int lp = __builtin_ctz(unsigned(P2));
  const int cpb = (INTER ? a.rd : P2) / V;
  const int shift = __builtin_ctz(unsigned(cpb));
  const int chunk = threadIdx.x & (cpb - 1);
  const int nh = a.nq + a.nk;
  const int tb = int((a.mode >> kRopeTokensShift) & 0xFFu);
  const int tpb = tb < 1 ? 1 : (tb > kRopeTokensMax ? kRopeTokensMax : tb);
  const int sb = int((a.mode >> kRopeSliceShift) & 0xFFu);
  const int S = tpb == 1 && sb > 1 ? sb : 1;
  const int64_t tok_blk = S > 1 ? blk / S : blk;
  const int hg = int(blk - tok_blk * S) + S * int(threadIdx.x >> shift);   // first head
  const int hstep = S * (kThreads >> shift);
  const int64_t t0 = tok_blk * tpb;
  const int64_t tlast = a.T - 1;
  float *cs = lds;
  float *sn = lds + kRopeTokensMax * 256;
  const int na = tpb * P2;
  // byte offset of the second vector of an item (rotate-half: the other half)
  const int off2 = P2 * E::ES;

  // Head-norm weight chunks of this work-item (Q and K; both halves).
  u32x4 wq1, wq2, wk1, wk2;
  if constexpr (QKN) {
    const char *qw = static_cast<const char *>(a.qw);
    const char *kw = a.kw ? static_cast<const char *>(a.kw) : qw;
    wq1 = reinterpret_cast<const u32x4 *>(qw)[chunk];
    wk1 = reinterpret_cast<const u32x4 *>(kw)[chunk];
    if constexpr (!INTER) {
      wq2 = reinterpret_cast<const u32x4 *>(qw + off2)[chunk];
      wk2 = reinterpret_cast<const u32x4 *>(kw + off2)[chunk];
    }
  }

  // Operands of this work-item's angle slot (token t0 + tid / P2, pair
  // tid % P2); indices are clamped so the loads are always in bounds. The
  // plain mode (int32 positions, computed angles) requests them before the
  // gather.
  const int ia = threadIdx.x & (P2 - 1);
  const int64_t ta = t0 + (threadIdx.x >> lp);
  const uint32_t vbits = a.mode & 0xFFu;
  const bool plain = vbits == 0 || vbits == kRopeInterleaved;
  int32_t pa = 0;
  float ina = 0.0f;
  if (plain) {
    pa = static_cast<const int32_t *>(a.pos)[ta <= tlast ? ta : tlast];
    ina = a.inv_freq[ia];
  }

  int tt = 0, h = hg;
  const int hfirst = hg < nh ? hg : nh - 1;
  u32x4 x1[PF], x2[PF];
  int it[PF], ih[PF];
  bool ok[PF];
  auto gather = [&]() {
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      ok[j] = tt < tpb && t0 + tt <= tlast && h < nh;
      it[j] = ok[j] ? tt : 0;
      ih[j] = ok[j] ? h : hfirst;
      const char *b = rope_head(a, t0 + it[j], ih[j], E::ES);
      x1[j] = ld16<NT>(reinterpret_cast<const u32x4 *>(b) + chunk);
      if constexpr (!INTER) x2[j] = ld16<NT>(reinterpret_cast<const u32x4 *>(b + off2) + chunk);
      if (ok[j]) {
        h += hstep;
        if (h >= nh) {
          h = hg;
          ++tt;
        }
      }
    }
  };
  gather();

  if (na <= kThreads) {
    if (threadIdx.x < na) {
      float c = 1.0f, s = 0.0f;
      if (ta <= tlast) {
        if (plain)
          sincosf(float(pa) * ina, &s, &c);
        else
          rope_cos_sin(a, ta, ia, c, s);
      }
      cs[threadIdx.x] = c;
      sn[threadIdx.x] = s;
    }
  } else {
    for (int e = threadIdx.x; e < na; e += kThreads) {
      const int64_t t = t0 + (e >> lp);
      float c = 1.0f, s = 0.0f;
      if (t <= tlast) rope_cos_sin(a, t, e & (P2 - 1), c, s);
      cs[e] = c;
      sn[e] = s;
    }
  }
  __syncthreads();

  for (;;) {
#pragma unroll
    for (int j = 0; j < PF; ++j) {
      if (!ok[j]) continue;   // uniform over the lanes of a head group
      float f1[V], f2[V];
      E::unpack(x1[j], f1);
      if constexpr (!INTER) E::unpack(x2[j], f2);
      if constexpr (QKN) {
        float ss = 0.0f;
#pragma unroll
        for (int e = 0; e < V; ++e) ss = __builtin_fmaf(f1[e], f1[e], ss);
        if constexpr (!INTER) {
#pragma unroll
          for (int e = 0; e < V; ++e) ss = __builtin_fmaf(f2[e], f2[e], ss);
        }
        ss = group_sum(ss, cpb);
        const float inv = rsqrtf(ss / float(a.hd) + a.eps);
        const bool isq = ih[j] < a.nq;
        float w1[V];
        E::unpack(isq ? wq1 : wk1, w1);
#pragma unroll
        for (int e = 0; e < V; ++e) f1[e] = (f1[e] * inv) * w1[e];
        if constexpr (!INTER) {
          float w2[V];
          E::unpack(isq ? wq2 : wk2, w2);
#pragma unroll
          for (int e = 0; e < V; ++e) f2[e] = (f2[e] * inv) * w2[e];
        }
      }
      char *b = rope_head(a, t0 + it[j], ih[j], E::ES);
      if constexpr (INTER) {
        const int base = it[j] * P2 + ((chunk * V) >> 1);
        float o[V];
#pragma unroll
        for (int e = 0; e < V; e += 2) {
          const float c = cs[base + (e >> 1)], s = sn[base + (e >> 1)];
          o[e] = rot_a(f1[e], f1[e + 1], c, s);
          o[e + 1] = rot_b(f1[e], f1[e + 1], c, s);
        }
        st16<NT>(reinterpret_cast<u32x4 *>(b) + chunk, E::pack(o));
      } else {
        const int base = it[j] * P2 + chunk * V;
        float o1[V], o2[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
          const float c = cs[base + e], s = sn[base + e];
          o1[e] = rot_a(f1[e], f2[e], c, s);
          o2[e] = rot_b(f1[e], f2[e], c, s);
        }
        st16<NT>(reinterpret_cast<u32x4 *>(b) + chunk, E::pack(o1));
        st16<NT>(reinterpret_cast<u32x4 *>(b + off2) + chunk, E::pack(o2));
      }
    }
    if (!(tt < tpb && t0 + tt <= tlast && hg < nh)) break;
    gather();
  }
}

// Any alignment / head size / variant: one token per workgroup, element
// pairs. `lds` holds 2 * 256 floats (cos, sin), and 256 more for QKN. Pairs
// are (i, i + rd/2), or (2i, 2i + 1) with kRopeInterleaved.
//
// QKN: heads are taken 256 at a time; wavefront w reduces the squares of
// heads w, w + 4, ... of the slice (element-wise loads, any alignment) and
// leaves 1/rms in LDS, then all work-items normalise and rotate the slice,
// and normalise the elements past rd.
template <int DT, bool QKN = false>
__device__ __forceinline__ void rope_scalar_block(const RopeArgs &a, int64_t t, float *lds) {
  using E = Elt<DT>;
  const int P2 = a.rd >> 1;
  const bool inter = a.mode & kRopeInterleaved;
  float *cs = lds;
  float *sn = lds + 256;
  for (int i = threadIdx.x; i < P2; i += kThreads) {
    float c, s;
    rope_cos_sin(a, t, i, c, s);
    cs[i] = c;
    sn[i] = s;
  }
  __syncthreads();
  const int nh = a.nq + a.nk;
  if constexpr (!QKN) {
    const int total = nh * P2;
    for (int e = threadIdx.x; e < total; e += kThreads) {
      const int h = e / P2;
      const int i = e - h * P2;
      const int i0 = inter ? 2 * i : i, i1 = inter ? 2 * i + 1 : i + P2;
      char *base = rope_head(a, t, h, E::ES);
      const float v1 = E::ld(base, i0), v2 = E::ld(base, i1);
      E::st(base, i0, rot_a(v1, v2, cs[i], sn[i]));
      E::st(base, i1, rot_b(v1, v2, cs[i], sn[i]));
    }
  } else {
    float *rinv = lds + 512;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const void *kw = a.kw ? a.kw : a.qw;
    const int pass = a.hd - a.rd;
    for (int h0 = 0; h0 < nh; h0 += kThreads) {
      const int hn = nh - h0 < kThreads ? nh - h0 : kThreads;
      for (int hl = wid; hl < hn; hl += kThreads / 64) {
        const char *base = rope_head(a, t, h0 + hl, E::ES);
        float ss = 0.0f;
        for (int i = lane; i < a.hd; i += 64) {
          const float v = E::ld(base, i);
          ss = __builtin_fmaf(v, v, ss);
        }
        ss = wave_sum(ss);
        if (lane == 0) rinv[hl] = rsqrtf(ss / float(a.hd) + a.eps);
      }
      __syncthreads();
      const int total = hn * P2;
      for (int e = threadIdx.x; e < total; e += kThreads) {
        const int hl = e / P2;
        const int i = e - hl * P2;
        const int i0 = inter ? 2 * i : i, i1 = inter ? 2 * i + 1 : i + P2;
        const int h = h0 + hl;
        const void *w = h < a.nq ? a.qw : kw;
        char *base = rope_head(a, t, h, E::ES);
        const float r = rinv[hl];
        const float n1 = (E::ld(base, i0) * r) * E::ld(w, i0);
        const float n2 = (E::ld(base, i1) * r) * E::ld(w, i1);
        E::st(base, i0, rot_a(n1, n2, cs[i], sn[i]));
        E::st(base, i1, rot_b(n1, n2, cs[i], sn[i]));
      }
      const int tp = hn * pass;
      for (int e = threadIdx.x; e < tp; e += kThreads) {
        const int hl = e / pass;
        const int j = a.rd + (e - hl * pass);
        const int h = h0 + hl;
        const void *w = h < a.nq ? a.qw : kw;
        char *base = rope_head(a, t, h, E::ES);
        E::st(base, j, (E::ld(base, j) * rinv[hl]) * E::ld(w, j));
      }
      __syncthreads();
    }
  }
}

// ---- SwiGLU ----------------------------------------------------------------------
// silu(g) = g / (1 + exp(-g)), evaluated as g * rcp(1 + exp(-g)) with the
// hardware reciprocal (v_rcp_f32, 1 ulp): the correctly rounded float32
// division costs about ten vector instructions per element, which made the
// streaming SwiGLU and silu kernels bound by vector ALU throughput rather
// than by HBM. Below g = -80, 1 + exp(g) is 1 in float32 and silu(g) is
// g * exp(g); that form keeps the tail where exp(-g) overflows (from
// g = -88.7 on) and would flush the product to zero although the value is
// still a normal float32 down to about g = -91.5. The tail is recomputed
// only where a lane is in it: a select of both forms costs three more
// vector instructions per element, which the streaming silu kernel
// measured as 7 % (it sits close to its vector ALU limit), while the
// branch is skipped whenever no lane of the wavefront is that negative.
// At g = -inf the tail gives -inf * 0 = NaN, as -inf / (1 + inf) does.
//
// exp(-g) itself is 2^th * 2^tl with th = RN(-g * hi), tl = the rest of
// -g * log2(e) (an fma recovers the product's rounding error, lo carries
// log2(e) - hi), and 2^tl = 1 + tl ln 2 to first order (|tl| < 2^-17): the
// hardware exp2 (v_exp_f32, 1 ulp) and four more instructions instead of
// the library expf's range reduction. The relative error of silu stays
// below 2.4e-7 for |g| <= 80 (checked against the float64 value over
// 3 million arguments, as expf's form gives 1.9e-7). At one token the
// SwiGLU role is the chain's critical path and runs its instructions back
// to back on one wavefront per SIMD: the shorter sequence measured 2.37
// against 2.56 us of device time for the standalone 1-token SwiGLU
// (rocprofv3, 3000 launches each). g is capped at 100 for the exponent
// (exp(-100) is far below float32's resolution next to 1), which keeps
// th and tl finite at g = +inf, where silu is +inf.
__device__ __forceinline__ float silu(float g) {
  constexpr float kLog2eHi = 1.44269502162933349609375f;   // RN_f32(log2 e)
  constexpr float kLog2eLo = 1.925963e-08f;                // log2 e - kLog2eHi
  constexpr float kLn2 = 0.693147180559945309f;
  const float ng = -__builtin_fminf(g, 100.0f);
  const float th = ng * kLog2eHi;
  const float tl = __builtin_fmaf(ng, kLog2eHi, -th) + ng * kLog2eLo;
  const float e = __builtin_amdgcn_exp2f(th);
  float r = g * __builtin_amdgcn_rcpf(1.0f + __builtin_fmaf(e * tl, kLn2, e));
  if (__builtin_expect(g < -80.0f, 0)) r = g * expf(g);
  return r;
}

__device__ __forceinline__ float silu_mul(float g, float u) {
  return silu(g) * u;
}

// Flat contiguous [T*I]: workgroup `blk` of `nblk` handles U vectors per
// work-item per step; workgroup 0 also does the < V element tail.
template <int DT, int U, bool NT>
__device__ __forceinline__ void sw_flat_part(const SwArgs &a, int64_t blk, int64_t nblk) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  const u32x4 *g = static_cast<const u32x4 *>(a.gate);
  const u32x4 *u = static_cast<const u32x4 *>(a.up);
  u32x4 *o = static_cast<u32x4 *>(a.out);
  const int64_t nvec = a.nvec;
  const int64_t step = nblk * kThreads * U;
  for (int64_t base = blk * kThreads * U + threadIdx.x; base < nvec; base += step) {
    u32x4 gv[U], uv[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t idx = base + int64_t(k) * kThreads;
      if (idx < nvec) {
        gv[k] = ld16<NT>(g + idx);
        uv[k] = ld16<NT>(u + idx);
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t idx = base + int64_t(k) * kThreads;
      if (idx < nvec) {
        float fg[V], fu[V];
        E::unpack(gv[k], fg);
        E::unpack(uv[k], fu);
#pragma unroll
        for (int e = 0; e < V; ++e) fg[e] = silu_mul(fg[e], fu[e]);
        st16<NT>(o + idx, E::pack(fg));
      }
    }
  }
  if (blk == 0) {
    const int64_t i = nvec * V + threadIdx.x;
    if (i < a.n) E::st(a.out, i, silu_mul(E::ld(a.gate, i), E::ld(a.up, i)));
  }
}

// Aligned rows with padded strides: (row, 256-vector chunk) items.
template <int DT>
__device__ __forceinline__ void sw_rows_part(const SwArgs &a, int64_t blk, int64_t nblk) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  const int64_t nvr = a.I / V;
  const int64_t cb = (nvr + kThreads - 1) / kThreads;
  const int64_t total = a.T * cb;
  for (int64_t it = blk; it < total; it += nblk) {
    const int64_t row = it / cb;
    const int64_t vi = (it - row * cb) * kThreads + threadIdx.x;
    if (vi < nvr) {
      const u32x4 gv = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.gate) +
                                                        row * a.g_rs * E::ES)[vi];
      const u32x4 uv = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.up) +
                                                        row * a.u_rs * E::ES)[vi];
      float fg[V], fu[V];
      E::unpack(gv, fg);
      E::unpack(uv, fu);
#pragma unroll
      for (int e = 0; e < V; ++e) fg[e] = silu_mul(fg[e], fu[e]);
      reinterpret_cast<u32x4 *>(static_cast<char *>(a.out) + row * a.o_rs * E::ES)[vi] =
          E::pack(fg);
    }
  }
}

// Any alignment: element-wise over T*I.
template <int DT>
__device__ __forceinline__ void sw_scalar_part(const SwArgs &a, int64_t blk, int64_t nblk) {
  using E = Elt<DT>;
  const int64_t n = a.T * a.I;
  for (int64_t e = blk * kThreads + threadIdx.x; e < n; e += nblk * kThreads) {
    const int64_t row = e / a.I;
    const int64_t j = e - row * a.I;
    const float r = silu_mul(E::ld(a.gate, row * a.g_rs + j), E::ld(a.up, row * a.u_rs + j));
    E::st(a.out, row * a.o_rs + j, r);
  }
}

// ---- element-wise ops (silu, add, masked_fill) and embedding -------------------------
constexpr int kOpSilu = 8, kOpAdd = 9, kOpMaskedFill = 10;   // the ABI's op ids

// One element of an element-wise op on float values (masked_fill works on
// bit patterns instead, see below).
template <int OP>
__device__ __forceinline__ float elt_value(float a, float b) {
  if constexpr (OP == kOpAdd)
    return a + b;
  else
    return silu(a);
}

// masked_fill on one 16-byte vector: element e takes `fill` (the fill
// value's bit pattern) where mask byte e is nonzero, else keeps its bits.
template <int DT>
__device__ __forceinline__ u32x4 mask_select(u32x4 x, uint64_t m, uint32_t fill) {
  u32x4 o;
  if constexpr (DT == kF32) {
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = ((m >> (8 * e)) & 0xFF) ? fill : x[e];
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo = ((m >> (16 * j)) & 0xFF) ? fill : (x[j] & 0xFFFFu);
      const uint32_t hi = ((m >> (16 * j + 8)) & 0xFF) ? fill : (x[j] >> 16);
      o[j] = lo | (hi << 16);
    }
  }
  return o;
}

template <int DT>
__device__ __forceinline__ uint32_t fill_bits(float value) {
  if constexpr (DT == kF32)
    return __float_as_uint(value);
  else
    return Elt<kBF16>::pack2(value, 0.0f) & 0xFFFFu;   // round to nearest even
}

// The V mask bytes of vector vi of a row starting at `m` (aligned to V).
template <int DT>
__device__ __forceinline__ uint64_t mask_bytes(const uint8_t *m, int64_t vi) {
  if constexpr (DT == kF32)
    return reinterpret_cast<const uint32_t *>(m)[vi];
  else
    return reinterpret_cast<const uint64_t *>(m)[vi];
}

template <int DT, int OP>
__device__ __forceinline__ u32x4 elt_vector(u32x4 x, const void *b, int64_t vi,
                                            const uint8_t *mrow, uint32_t fill, bool nt) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  if constexpr (OP == kOpMaskedFill) {
    return mask_select<DT>(x, mask_bytes<DT>(mrow, vi), fill);
  } else {
    float fa[V], fb[V];
    E::unpack(x, fa);
    if constexpr (OP == kOpAdd) {
      const u32x4 y = nt ? ld16<true>(static_cast<const u32x4 *>(b) + vi)
                         : ld16<false>(static_cast<const u32x4 *>(b) + vi);
      E::unpack(y, fb);
    }
#pragma unroll
    for (int e = 0; e < V; ++e) fa[e] = elt_value<OP>(fa[e], OP == kOpAdd ? fb[e] : 0.0f);
    return E::pack(fa);
  }
}

// Flat contiguous [T*W]: U vectors per work-item per step (all loads
// issued before any use); workgroup 0 also does the < V element tail.
template <int DT, int OP, bool NT, int U = 1>
__device__ __forceinline__ void elt_flat_part(const EltArgs &a, int64_t blk, int64_t nblk) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  const u32x4 *x = static_cast<const u32x4 *>(a.a);
  u32x4 *o = static_cast<u32x4 *>(a.out);
  const uint8_t *m = static_cast<const uint8_t *>(a.b);
  const uint32_t fill = fill_bits<DT>(a.value);
  const int64_t step = nblk * kThreads * U;
  for (int64_t base = blk * kThreads * U + threadIdx.x; base < a.nvec; base += step) {
    u32x4 xv[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * kThreads;
      if (i < a.nvec) xv[k] = ld16<NT>(x + i);
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * kThreads;
      if (i < a.nvec) st16<NT>(o + i, elt_vector<DT, OP>(xv[k], a.b, i, m, fill, NT));
    }
  }
  if (blk == 0) {
    const int64_t i = a.nvec * V + threadIdx.x;
    if (i < a.n) {
      if constexpr (OP == kOpMaskedFill) {
        if (m[i]) E::st(a.out, i, a.value);   // st rounds to the dtype
        else E::st(a.out, i, E::ld(a.a, i));
      } else {
        E::st(a.out, i, elt_value<OP>(E::ld(a.a, i), OP == kOpAdd ? E::ld(a.b, i) : 0.0f));
      }
    }
  }
}

// Aligned rows with padded strides: (row, 256-vector chunk) items.
template <int DT, int OP>
__device__ __forceinline__ void elt_rows_part(const EltArgs &a, int64_t blk, int64_t nblk) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  const int64_t nvr = a.W / V;
  const int64_t cb = (nvr + kThreads - 1) / kThreads;
  const uint32_t fill = fill_bits<DT>(a.value);
  for (int64_t it = blk; it < a.T * cb; it += nblk) {
    const int64_t row = it / cb;
    const int64_t vi = (it - row * cb) * kThreads + threadIdx.x;
    if (vi < nvr) {
      const u32x4 *x = reinterpret_cast<const u32x4 *>(static_cast<const char *>(a.a) +
                                                       row * a.a_rs * E::ES);
      const char *brow = static_cast<const char *>(a.b) +
                         row * a.b_rs * (OP == kOpMaskedFill ? 1 : E::ES);
      u32x4 *o = reinterpret_cast<u32x4 *>(static_cast<char *>(a.out) + row * a.o_rs * E::ES);
      o[vi] = elt_vector<DT, OP>(x[vi], brow, vi, reinterpret_cast<const uint8_t *>(brow), fill,
                                 false);
    }
  }
}

// Any alignment: element-wise over T*W (masked_fill copies bit patterns).
template <int DT, int OP>
__device__ __forceinline__ void elt_scalar_part(const EltArgs &a, int64_t blk, int64_t nblk) {
  using E = Elt<DT>;
  const int64_t n = a.T * a.W;
  for (int64_t e = blk * kThreads + threadIdx.x; e < n; e += nblk * kThreads) {
    const int64_t row = e / a.W;
    const int64_t j = e - row * a.W;
    if constexpr (OP == kOpMaskedFill) {
      const bool set = static_cast<const uint8_t *>(a.b)[row * a.b_rs + j] != 0;
      if constexpr (DT == kF32) {
        const uint32_t x = static_cast<const uint32_t *>(a.a)[row * a.a_rs + j];
        static_cast<uint32_t *>(a.out)[row * a.o_rs + j] = set ? fill_bits<DT>(a.value) : x;
      } else {
        const uint16_t x = static_cast<const uint16_t *>(a.a)[row * a.a_rs + j];
        static_cast<uint16_t *>(a.out)[row * a.o_rs + j] =
            set ? uint16_t(fill_bits<DT>(a.value)) : x;
      }
    } else {
      const float r = elt_value<OP>(E::ld(a.a, row * a.a_rs + j),
                                    OP == kOpAdd ? E::ld(a.b, row * a.b_rs + j) : 0.0f);
      E::st(a.out, row * a.o_rs + j, r);
    }
  }
}

// Embedding: workgroup b of nblk copies output rows b, b + nblk, ...; the
// row is table row ids[t] when it is in [0, n_rows), zeros otherwise.
template <int DT, bool VEC>
__device__ __forceinline__ void emb_rows(const EmbArgs &a, uint32_t nblk) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  for (int64_t t = blockIdx.x; t < a.T; t += nblk) {
    const int64_t id = a.ids64 ? static_cast<const int64_t *>(a.ids)[t]
                               : int64_t(static_cast<const int32_t *>(a.ids)[t]);
    const bool ok = id >= 0 && id < a.n_rows;
    const char *src = static_cast<const char *>(a.table) + (ok ? id : 0) * a.t_rs * E::ES;
    char *dst = static_cast<char *>(a.out) + t * a.o_rs * E::ES;
    if constexpr (VEC) {
      const int64_t nvr = a.H / V;
      for (int64_t vi = threadIdx.x; vi < nvr; vi += kThreads) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (ok) v = reinterpret_cast<const u32x4 *>(src)[vi];
        reinterpret_cast<u32x4 *>(dst)[vi] = v;
      }
    } else {
      for (int64_t j = threadIdx.x; j < a.H; j += kThreads) {
        if constexpr (DT == kF32)
          reinterpret_cast<uint32_t *>(dst)[j] = ok ? reinterpret_cast<const uint32_t *>(src)[j] : 0u;
        else
          reinterpret_cast<uint16_t *>(dst)[j] = ok ? reinterpret_cast<const uint16_t *>(src)[j] : 0;
      }
    }
  }
}

// ---- kernel bodies -----------------------------------------------------------------
// One body per kernel family, called by the precompiled kernels and by the
// runtime-compiled specializations; a specialization passes arguments whose
// shape fields are compile-time constants.
template <int DT, int NV, bool RES>
__device__ __forceinline__ void body_rn_wave(const RnArgs &a) {
  rn_wave_block<DT, NV, RES, false>(a, blockIdx.x);
}

template <int DT, int NB, bool RES>
__device__ __forceinline__ void body_rn_block(const RnArgs &a) {
  __shared__ float red[4];
  rn_row_regs<DT, NB, RES, 256, false>(a, blockIdx.x, threadIdx.x, red);
}

template <int DT, bool RES>
__device__ __forceinline__ void body_rn_loop(const RnArgs &a) {
  __shared__ double red[4];
  rn_loop_row<DT, RES>(a, blockIdx.x, red);
}

// Plain RMSNorm of a row held by a 1024-work-item workgroup, 8 vectors per
// lane: the row is kept packed across the reduction and the weights are
// requested only after it, in two halves, so a lane holds at most 8 + 4
// vectors and two workgroups fit on a CU (61 VGPRs, 8 waves per SIMD,
// against 122 with the weights requested with the row and the row kept
// unpacked: one workgroup per CU, whose loads then never overlap another
// row's stores). Same arithmetic in the same order as rn_row_regs.
template <int DT>
__device__ __forceinline__ void rn_row_wide_plain(const RnArgs &a, int64_t row, int lane,
                                                  float *red) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  constexpr int NV = 8, L = kWideLanes, HALF = NV / 2;
  const int nvec = a.H / V;
  // uniform row bases and 32-bit per-lane byte offsets, so that every
  // access is a scalar base plus one offset register
  const char *xb = static_cast<const char *>(a.x) + row * a.x_rs * E::ES;
  const char *wb = static_cast<const char *>(a.w);
  char *yb = static_cast<char *>(a.y) + row * a.y_rs * E::ES;
  const uint32_t off0 = uint32_t(lane) * 16u;
  // Loads past the row's end read its last vector instead (no branch, no
  // saved lane masks) and are zeroed.
  const uint32_t last = uint32_t(nvec - 1) * 16u;
  u32x4 xv[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const uint32_t off = off0 + uint32_t(k) * (L * 16u);
    const u32x4 v = *reinterpret_cast<const u32x4 *>(xb + (off < last ? off : last));
    xv[k] = off <= last ? v : u32x4{0, 0, 0, 0};
  }
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float f[V];
    E::unpack(xv[k], f);
#pragma unroll
    for (int e = 0; e < V; ++e) ss = __builtin_fmaf(f[e], f[e], ss);
  }
  // the unpacked floats are not kept for the output pass: it unpacks again
#pragma unroll
  for (int k = 0; k < NV; ++k) asm volatile("" : "+v"(xv[k]));
  // The 16 wavefront sums: each lane takes one of them (every one four
  // times over the wavefront), so the combine holds one value per lane
  // rather than all 16 next to the row; the wavefront total is exactly four
  // times the row's and is the same bits in every lane.
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  static_assert(L / 64 == 16, "one partial per lane of a 16-lane group");
  ss = wave_sum(red[threadIdx.x & 15]) * 0.25f;
  const float inv = rsqrtf(ss / float(a.H) + a.eps);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    u32x4 wv[HALF];
#pragma unroll
    for (int k = 0; k < HALF; ++k) {
      const uint32_t off = off0 + uint32_t(h * HALF + k) * (L * 16u);
      wv[k] = *reinterpret_cast<const u32x4 *>(wb + (off < last ? off : last));
    }
#pragma unroll
    for (int k = 0; k < HALF; ++k) {
      const int j = h * HALF + k;
      if (off0 + uint32_t(j) * (L * 16u) <= last) {
        // one 32-bit word at a time: few temporaries live at once
        u32x4 yv;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          if constexpr (DT == kBF16) {
            const float x0 = __uint_as_float(xv[j][d] << 16), x1 = __uint_as_float(xv[j][d] & 0xFFFF0000u);
            const float w0 = __uint_as_float(wv[k][d] << 16), w1 = __uint_as_float(wv[k][d] & 0xFFFF0000u);
            yv[d] = E::pack2((x0 * inv) * w0, (x1 * inv) * w1);
          } else {
            yv[d] = __float_as_uint((__uint_as_float(xv[j][d]) * inv) * __uint_as_float(wv[k][d]));
          }
        }
        *reinterpret_cast<u32x4 *>(yb + off0 + uint32_t(j) * (L * 16u)) = yv;
      }
    }
    // the second half's weights are requested after the first half's stores
    asm volatile("" ::: "memory");
  }
}

// Buffer access to one row: the row's uniform base with its byte length as
// the range. A load past the range returns zeros and a store past it is
// dropped, so a row of any length up to 8 * kWideLanes vectors needs no
// branch, and each access is the descriptor plus one per-lane offset.
// Descriptor word 3: data format 32 bits (nonzero, as untyped loads need),
// no swizzle, no index stride.
constexpr int kRowRsrcWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void *base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, kRowRsrcWord3);
}

__device__ __forceinline__ void wide_load(__amdgpu_buffer_rsrc_t r, uint32_t off0, u32x4 *xv) {
#pragma unroll
  for (int k = 0; k < 8; ++k)
    xv[k] = __builtin_amdgcn_raw_buffer_load_b128(r, off0 + uint32_t(k) * (kWideLanes * 16u), 0, 0);
}

// One row of the pipelined plain form, held packed in xv (zeros past the
// row's end); the lane's weight vectors are in wl. Same arithmetic in the
// same order as rn_row_wide_plain, so both give the same bits.
template <int DT>
__device__ __forceinline__ void wide_norm_store(const RnArgs &a, u32x4 *xv, const u32x4 *wl,
                                                __amdgpu_buffer_rsrc_t yr, uint32_t off0,
                                                float *red) {
  using E = Elt<DT>;
  constexpr int V = E::V;
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float f[V];
    E::unpack(xv[k], f);
#pragma unroll
    for (int e = 0; e < V; ++e) ss = __builtin_fmaf(f[e], f[e], ss);
  }
  // the output pass unpacks again: the floats are not kept
#pragma unroll
  for (int k = 0; k < 8; ++k) asm volatile("" : "+v"(xv[k]));
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = wave_sum(red[threadIdx.x & 15]) * 0.25f;
  const float inv = rsqrtf(ss / float(a.H) + a.eps);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const u32x4 w = wl[j * kWideLanes + threadIdx.x];
    u32x4 yv;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      if constexpr (DT == kBF16) {
        const float x0 = __uint_as_float(xv[j][d] << 16), x1 = __uint_as_float(xv[j][d] & 0xFFFF0000u);
        const float w0 = __uint_as_float(w[d] << 16), w1 = __uint_as_float(w[d] & 0xFFFF0000u);
        yv[d] = E::pack2((x0 * inv) * w0, (x1 * inv) * w1);
      } else {
        yv[d] = __float_as_uint((__uint_as_float(xv[j][d]) * inv) * __uint_as_float(w[d]));
      }
    }
    __builtin_amdgcn_raw_buffer_store_b128(yv, yr, off0 + uint32_t(j) * (kWideLanes * 16u), 0, 0);
  }
}

// Plain RMSNorm when a workgroup has several rows: workgroup b takes rows
// b, b + nblk, ... and requests each next row before the current row's
// reduction, so one row's loads overlap the previous row's stores on the
// same CU (one row per workgroup, the loads of every workgroup on the chip
// start together and then their stores, at bf16 rows of 57,344 measured
// 0.85 of a copy of the same bytes, against 0.90 with this loop). Two row
// buffers used in turn, so no register copy makes the next row's loads
// complete early; the weights wait in LDS (each lane reads back only the
// vectors it wrote: no barrier), which keeps the lane at 8 + 8 vectors
// (121 VGPRs; holding the weights in registers spills). The partial sums
// alternate between two LDS rows, so one barrier per row suffices.
template <int DT>
__device__ __forceinline__ void rn_rows_wide_plain(const RnArgs &a, uint32_t nblk, u32x4 *wl,
                                                   float (*red)[kWideLanes / 64]) {
  using E = Elt<DT>;
  const uint32_t off0 = uint32_t(threadIdx.x) * 16u;
  const int rowb = (a.H / E::V) * 16;
  const char *xbase = static_cast<const char *>(a.x);
  char *ybase = static_cast<char *>(a.y);
  const int64_t xs = a.x_rs * E::ES, ys = a.y_rs * E::ES;
  int64_t row = blockIdx.x;
  u32x4 ra[8], rb[8];
  wide_load(row_rsrc(a.w, rowb), off0, ra);
#pragma unroll
  for (int k = 0; k < 8; ++k) wl[k * kWideLanes + threadIdx.x] = ra[k];
  wide_load(row_rsrc(xbase + row * xs, rowb), off0, ra);
  for (;;) {
    if (row + nblk >= a.T) {
      wide_norm_store<DT>(a, ra, wl, row_rsrc(ybase + row * ys, rowb), off0, red[0]);
      return;
    }
    wide_load(row_rsrc(xbase + (row + nblk) * xs, rowb), off0, rb);
    wide_norm_store<DT>(a, ra, wl, row_rsrc(ybase + row * ys, rowb), off0, red[0]);
    row += nblk;
    if (row + nblk >= a.T) {
      wide_norm_store<DT>(a, rb, wl, row_rsrc(ybase + row * ys, rowb), off0, red[1]);
      return;
    }
    wide_load(row_rsrc(xbase + (row + nblk) * xs, rowb), off0, ra);
    wide_norm_store<DT>(a, rb, wl, row_rsrc(ybase + row * ys, rowb), off0, red[1]);
    row += nblk;
  }
}

// Rows of 4097..8192 vectors on 1024-work-item workgroups, up to 8 vectors
// per lane held in registers (all loads issued up front). The residual form
// takes one row per workgroup (grid T) and requests the weights with the
// row (measured 1 % faster for it; a loop over rows measured 4-35 % slower).
// The plain form is launched on at most kWideGrid workgroups: with one row
// each, rn_row_wide_plain; with more, rn_rows_wide_plain.
template <int DT, bool RES>
__device__ __forceinline__ void body_rn_wide(const RnArgs &a, uint32_t nblk = gridDim.x) {
  if constexpr (RES) {
    __shared__ float red[kWideLanes / 64];
    rn_row_regs<DT, 8, RES, kWideLanes, false>(a, blockIdx.x, threadIdx.x, red);
  } else {
    __shared__ float red[2][kWideLanes / 64];
    __shared__ u32x4 wl[8 * kWideLanes];
    if (a.T <= int64_t(nblk)) {
      if (int64_t(blockIdx.x) < a.T) rn_row_wide_plain<DT>(a, blockIdx.x, threadIdx.x, red[0]);
    } else {
      rn_rows_wide_plain<DT>(a, nblk, wl, red);
    }
  }
}

// Rows of more than 4096 vectors over several workgroups (rn_split_row).
template <int DT, bool RES>
__device__ __forceinline__ void body_rn_split(const RnSplitArgs &a) {
  rn_split_row<DT, RES>(a.rn, a.scratch);
}

template <int DT, bool RES>
__device__ __forceinline__ void body_rn_scalar(const RnArgs &a) {
  __shared__ double red[4];
  rn_scalar_row<DT, RES>(a, blockIdx.x, red);
}

// QKN: per-head RMSNorm of Q and K before the rotation; INTER: GPT-J pairs.
template <int DT, bool QKN, bool INTER>
__device__ __forceinline__ void body_rope_vec(const RopeArgs &a) {
  __shared__ float lds[2 * 256 * kRopeTokensMax];
  rope_vec_block<DT, false, 4, QKN, INTER>(a, blockIdx.x, lds);
}

template <int DT, bool QKN>
__device__ __forceinline__ void body_rope_scalar(const RopeArgs &a) {
  __shared__ float lds[(QKN ? 3 : 2) * 256];
  rope_scalar_block<DT, QKN>(a, blockIdx.x, lds);
}

// The bodies that stride over the grid take the launch's workgroup count:
// gridDim.x, or a resident block's count in a launch without kernel
// arguments (which must not read gridDim: that would give it implicit
// kernel arguments again).
template <int DT, int U, bool NT>
__device__ __forceinline__ void body_sw_flat(const SwArgs &a, uint32_t nblk = gridDim.x) {
  sw_flat_part<DT, U, NT>(a, blockIdx.x, nblk);
}

template <int DT>
__device__ __forceinline__ void body_sw_rows(const SwArgs &a, uint32_t nblk = gridDim.x) {
  sw_rows_part<DT>(a, blockIdx.x, nblk);
}

template <int DT>
__device__ __forceinline__ void body_sw_scalar(const SwArgs &a, uint32_t nblk = gridDim.x) {
  sw_scalar_part<DT>(a, blockIdx.x, nblk);
}

// U vectors per work-item, cached loads and stores.
template <int DT, int OP, int U>
__device__ __forceinline__ void body_elt_flat(const EltArgs &a, uint32_t nblk = gridDim.x) {
  elt_flat_part<DT, OP, false, U>(a, blockIdx.x, nblk);
}

template <int DT, int OP>
__device__ __forceinline__ void body_elt_rows(const EltArgs &a, uint32_t nblk = gridDim.x) {
  elt_rows_part<DT, OP>(a, blockIdx.x, nblk);
}

template <int DT, int OP>
__device__ __forceinline__ void body_elt_scalar(const EltArgs &a, uint32_t nblk = gridDim.x) {
  elt_scalar_part<DT, OP>(a, blockIdx.x, nblk);
}

template <int DT, bool VEC>
__device__ __forceinline__ void body_emb(const EmbArgs &a, uint32_t nblk = gridDim.x) {
  emb_rows<DT, VEC>(a, nblk);
}

// The fused decode chain: workgroups take the residual-RMSNorm, RoPE-QK and
// SwiGLU roles by blockIdx range. Norm role: one wavefront per row with N
// vectors per lane (WAVE) or one workgroup per row with N per work-item;
// RoPE role: one token, one head slice of a token, or up to four tokens per
// workgroup, as the argument block's mode says (QK norm first when QKN,
// GPT-J pairs when INTER); SwiGLU role: one vector per work-item,
// nontemporal when NT (calls that stream more than the last-level cache).
//
// Role order by blockIdx: norm rows, RoPE tokens, then SwiGLU. At decode
// sizes the norm and RoPE roles take about as long as SwiGLU but have far
// fewer workgroups, so dispatching them first shortens the critical path
// (2.75 vs 3.1 us device time at 1 token); at 8192 tokens this order with a
// one-vector nontemporal SwiGLU role measured 331.5 us, against 344-349 us
// for SwiGLU first or with two / four vectors per work-item.
//
// In the streaming form (NT: calls that move more than the last-level
// cache) the RoPE role also streams nontemporally and keeps one head item
// per work-item in flight instead of four: its 77 registers per lane
// (four items) capped the whole fused kernel at 6 wavefronts per SIMD where
// SwiGLU alone runs 8, and in alternating launches at 8192 tokens the
// lighter role took the chain from 357 to 346.5 us (the decode form keeps
// four items in flight, which its latency needs).
template <int DT, bool WAVE, int N>
__device__ __forceinline__ void chain_norm_role(const ChainArgs &a, uint32_t blk) {
  if constexpr (WAVE) {
    rn_wave_block<DT, N, true, false>(a.rn, blk);
  } else {
    __shared__ float red[4];
    rn_row_regs<DT, N, true, 256, false>(a.rn, blk, threadIdx.x, red);
  }
}

//
// `nblk` is the launch's workgroup count (gridDim.x, or the resident block's
// count in a launch without kernel arguments, which must not read gridDim:
// that would give the kernel implicit arguments again).
template <int DT, bool WAVE, int N, bool NT, bool QKN, bool INTER>
__device__ __forceinline__ void body_chain(const ChainArgs &a, uint32_t nblk) {
  __shared__ float lds[2 * 256 * kRopeTokensMax];
  const uint32_t b = blockIdx.x;
  const uint32_t R = a.rn_blocks, P = a.rope_blocks, S = nblk - R - P;
  if (b < R) {
    chain_norm_role<DT, WAVE, N>(a, b);
  } else if (b < R + P) {
    rope_vec_block<DT, NT, NT ? 1 : 4, QKN, INTER>(a.rope, b - R, lds);
  } else {
    sw_flat_part<DT, 1, NT>(a.sw, b - R - P, S);
  }
}

// The slot of a launch without kernel arguments. The workgroup's LDS
// allocation is readable in the LDS_ALLOC hardware register (bits 12..20,
// in 256-byte units; the hardware allocates whole kLdsGranule-byte
// granules): less the granules of the kernel's static LDS, it is the slot
// the host encoded as slot * kLdsGranule bytes of dynamic LDS. Reading a
// register costs no memory access, unlike the dispatch packet.
__device__ __forceinline__ uint32_t resident_slot() {
  const uint32_t units = __builtin_amdgcn_s_getreg((8 << 11) | (12 << 6) | 6);
  return units / (kLdsGranule / 256) -
         (__builtin_amdgcn_groupstaticsize() + kLdsGranule - 1) / kLdsGranule;
}

template <typename P>
__device__ __forceinline__ P *in_global(P *p) {
  typedef __attribute__((address_space(1))) P *gptr;
  gptr g;
  // an empty move the compiler cannot look through: the result is a
  // global-address-space pointer, so no cast pair folds back to flat
  asm("" : "=s"(g) : "0"((gptr)p));
  return (P *)g;
}

// Pointers read from memory could point anywhere; these are global memory,
// as kernel-argument pointers are taken to be (global, not flat, loads and
// stores).
__device__ __forceinline__ void to_global(RnArgs &a) {
  a.x = in_global(a.x);
  a.res = in_global(a.res);
  a.w = in_global(a.w);
  a.y = in_global(a.y);
  a.res_out = in_global(a.res_out);
}
__device__ __forceinline__ void to_global(RnSplitArgs &a) {
  to_global(a.rn);
  a.scratch = in_global(a.scratch);
}
__device__ __forceinline__ void to_global(RopeArgs &a) {
  a.q = in_global(a.q);
  a.k = in_global(a.k);
  a.pos = in_global(a.pos);
  a.inv_freq = in_global(a.inv_freq);
  a.qw = in_global(a.qw);
  a.kw = in_global(a.kw);
  a.cos_sin = in_global(a.cos_sin);
}
__device__ __forceinline__ void to_global(SwArgs &a) {
  a.gate = in_global(a.gate);
  a.up = in_global(a.up);
  a.out = in_global(a.out);
}
__device__ __forceinline__ void to_global(EltArgs &a) {
  a.a = in_global(a.a);
  a.b = in_global(a.b);
  a.out = in_global(a.out);
}
__device__ __forceinline__ void to_global(EmbArgs &a) {
  a.table = in_global(a.table);
  a.ids = in_global(a.ids);
  a.out = in_global(a.out);
}
__device__ __forceinline__ void to_global(ChainArgs &a) {
  to_global(a.rn);
  to_global(a.rope);
  to_global(a.sw);
}

// The argument block of a launch without kernel arguments: slot
// resident_slot() of `table` (this device's table of the kernel's family and
// dtype, read as constant memory: the host writes a slot only while no
// launch can read it). False for an index beyond the table or an unwritten
// slot: the launch then runs nothing.
template <class A>
__device__ __forceinline__ bool resident_args(const ResidentBlock *table, A &a, uint32_t &grid) {
  const uint32_t s = resident_slot();
  if (s >= kResidentSlots) return false;
  typedef __attribute__((address_space(4))) const uint32_t cu32;
  cu32 *w = (cu32 *)(table + s);
  if (w[__builtin_offsetof(ResidentBlock, tag) / 4] != kResidentTag + s) return false;
  uint32_t words[sizeof(A) / 4];
#pragma unroll
  for (uint32_t i = 0; i < sizeof(A) / 4; ++i) words[i] = w[i];
  __builtin_memcpy(&a, words, sizeof a);
  to_global(a);
  grid = w[__builtin_offsetof(ResidentBlock, grid) / 4];
  return true;
}

}  // namespace dev
}  // namespace tri

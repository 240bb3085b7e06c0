// Reference streaming copy for the benchmark: the practical HBM ceiling
// reported beside the path's kernels (a kernel that only moves bytes, with
// the same 16-byte vector access and 256-work-item workgroups).
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// U vectors per work-item per step, grid-stride; NT: nontemporal loads and
// stores. Every access is guarded by i < n.
template <int U, bool NT>
__global__ __launch_bounds__(256) void k_copy(const u32x4 *__restrict__ a, u32x4 *__restrict__ o,
                                              int64_t n) {
  const int64_t step = int64_t(gridDim.x) * 256 * U;
  for (int64_t base = int64_t(blockIdx.x) * 256 * U + threadIdx.x; base < n; base += step) {
    u32x4 v[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < n) v[k] = NT ? __builtin_nontemporal_load(a + i) : a[i];
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < n) {
        if (NT)
          __builtin_nontemporal_store(v[k], o + i);
        else
          o[i] = v[k];
      }
    }
  }
}

template <int U, bool NT>
int launch(const void *src, void *dst, int64_t n, hipStream_t s) {
  int64_t g = (n + 256 * U - 1) / (256 * U);
  if (g > (int64_t(1) << 20)) g = int64_t(1) << 20;
  k_copy<U, NT><<<dim3(uint32_t(g)), dim3(256), 0, s>>>(static_cast<const u32x4 *>(src),
                                                        static_cast<u32x4 *>(dst), n);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <bool NT>
__device__ inline u32x4 ld(const u32x4 *p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT>
__device__ inline void st(u32x4 *p, u32x4 v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// Vectors [v0, v1) of R input arrays streamed to W output arrays by one
// workgroup, U vectors per work-item in flight (all loads before any store).
// With INPLACE the W = R arrays are read and written back at the same
// addresses (RoPE's access). The stored value depends on every loaded one,
// so no load can be dropped (and an in-place store always changes the
// value, so it cannot be dropped either).
template <int R, int W, bool INPLACE, bool NT, int U>
__device__ inline void span(const u32x4 *const *in, u32x4 *const *out, int64_t v0, int64_t v1) {
  for (int64_t base = v0 + threadIdx.x; base < v1; base += 256 * U) {
    u32x4 v[U][R];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < v1) {
#pragma unroll
        for (int r = 0; r < R; ++r) v[k][r] = ld<NT>(in[r] + i);
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t i = base + int64_t(k) * 256;
      if (i < v1) {
        u32x4 x = v[k][0];
#pragma unroll
        for (int r = 1; r < R; ++r) x ^= v[k][r];
#pragma unroll
        for (int w = 0; w < W; ++w) {
          u32x4 *dst = INPLACE ? const_cast<u32x4 *>(in[w]) : out[w];
          st<NT>(dst + i, x + u32x4{uint32_t(w) + 1u, 0u, 0u, 0u});
        }
      }
    }
  }
}

struct Streams {
  const u32x4 *in[2];
  u32x4 *out[2];
  int64_t n;
};

// Grid-stride stream over n vectors per array, one vector per work-item.
template <int R, int W, bool INPLACE, bool NT>
__global__ __launch_bounds__(256) void k_mix(Streams a) {
  const int64_t step = int64_t(gridDim.x) * 256;
  for (int64_t b = int64_t(blockIdx.x) * 256; b < a.n; b += step)
    span<R, W, INPLACE, NT, 1>(a.in, a.out, b, b + 256 < a.n ? b + 256 : a.n);
}

// The decode chain's traffic with no arithmetic, in one launch with the
// chain's role layout: the first ga workgroups stream rows of the residual
// norm (two arrays read, two written, na vectors per workgroup), the next
// gb stream tokens of RoPE in place (nb0 vectors of q and nb1 of k per
// workgroup, nontemporal), the rest SwiGLU (two read, one written, grid
// stride over nc vectors, nontemporal).
struct ChainStreams {
  const u32x4 *a_in[2];
  u32x4 *a_out[2];
  const u32x4 *q;
  const u32x4 *k;
  const u32x4 *c_in[2];
  u32x4 *c_out[1];
  int64_t na, nb0, nb1, nc;
  uint32_t ga, gb;
};

__global__ __launch_bounds__(256) void k_chain_streams(ChainStreams a) {
  const uint32_t b = blockIdx.x;
  if (b < a.ga) {
    span<2, 2, false, false, 4>(a.a_in, a.a_out, int64_t(b) * a.na, int64_t(b + 1) * a.na);
  } else if (b < a.ga + a.gb) {
    const int64_t t = b - a.ga;
    span<1, 1, true, true, 4>(&a.q, nullptr, t * a.nb0, (t + 1) * a.nb0);
    if (a.nb1) span<1, 1, true, true, 4>(&a.k, nullptr, t * a.nb1, (t + 1) * a.nb1);
  } else {
    const int64_t nblk = int64_t(gridDim.x) - a.ga - a.gb;
    for (int64_t v = (int64_t(b) - a.ga - a.gb) * 256; v < a.nc; v += nblk * 256)
      span<2, 1, false, true, 1>(a.c_in, a.c_out, v, v + 256 < a.nc ? v + 256 : a.nc);
  }
}

template <int R, int W, bool INPLACE, bool NT>
int launch_mix(const Streams &a, hipStream_t s) {
  int64_t g = (a.n + 255) / 256;
  if (g > (int64_t(1) << 20)) g = int64_t(1) << 20;
  k_mix<R, W, INPLACE, NT><<<dim3(uint32_t(g)), dim3(256), 0, s>>>(a);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

bool a16(const void *p) { return (uintptr_t(p) & 15) == 0; }

}  // namespace

extern "C" {

// Reference streams of a fixed read:write mix over n16 16-byte vectors per
// array (all pointers 16-byte aligned and non-null where the kind uses
// them): kind 0 copy in0 -> out0; 1 in place (in0 read and written back);
// 2 two reads, one write (in0, in1 -> out0); 3 two reads, two writes. nt
// selects nontemporal loads and stores. Returns 0, or -1 for bad arguments
// or a failed launch.
int trib_mix(const void *in0, const void *in1, void *out0, void *out1, int64_t n16,
                int kind, int nt, void *stream) {
  const bool need1 = kind >= 2, needo = kind != 1, needo1 = kind == 3;
  if (n16 < 1 || !in0 || !a16(in0) || (need1 && (!in1 || !a16(in1))) ||
      (needo && (!out0 || !a16(out0))) || (needo1 && (!out1 || !a16(out1))))
    return -1;
  const Streams a{{static_cast<const u32x4 *>(in0), static_cast<const u32x4 *>(in1)},
                  {static_cast<u32x4 *>(out0), static_cast<u32x4 *>(out1)}, n16};
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (kind * 2 + (nt ? 1 : 0)) {
    case 0: return launch_mix<1, 1, false, false>(a, s);
    case 1: return launch_mix<1, 1, false, true>(a, s);
    case 2: return launch_mix<1, 1, true, false>(a, s);
    case 3: return launch_mix<1, 1, true, true>(a, s);
    case 4: return launch_mix<2, 1, false, false>(a, s);
    case 5: return launch_mix<2, 1, false, true>(a, s);
    case 6: return launch_mix<2, 2, false, false>(a, s);
    case 7: return launch_mix<2, 2, false, true>(a, s);
    default: return -1;
  }
}

// The decode chain's traffic without its arithmetic (k_chain_streams): T
// rows of H elements (x, res -> y, res_out), T tokens of qn and kn elements
// rotated in place (q, k), and T * I elements of SwiGLU (gate, up -> out),
// es bytes per element; every width a multiple of 16 bytes, every pointer
// 16-byte aligned. One launch of T + T + min(ceil(T * I * es / 4096), 2^20)
// workgroups. Returns 0 or -1.
int trib_chain_mix(const void *x, const void *res, void *y, void *res_out, void *q, void *k,
                      const void *gate, const void *up, void *out, int64_t T, int64_t H,
                      int64_t qn, int64_t kn, int64_t I, int es, void *stream) {
  if (T < 1 || T > (int64_t(1) << 22) || (es != 2 && es != 4) || (H * es) % 16 ||
      (qn * es) % 16 || (kn * es) % 16 || (I * es) % 16 || H < 1 || qn < 1 || kn < 0 || I < 1)
    return -1;
  const void *ptrs[] = {x, res, y, res_out, q, gate, up, out};
  for (const void *p : ptrs)
    if (!p || !a16(p)) return -1;
  if (kn > 0 && (!k || !a16(k))) return -1;
  ChainStreams a;
  a.a_in[0] = static_cast<const u32x4 *>(x);
  a.a_in[1] = static_cast<const u32x4 *>(res);
  a.a_out[0] = static_cast<u32x4 *>(y);
  a.a_out[1] = static_cast<u32x4 *>(res_out);
  a.q = static_cast<const u32x4 *>(q);
  a.k = kn > 0 ? static_cast<const u32x4 *>(k) : static_cast<const u32x4 *>(q);
  a.c_in[0] = static_cast<const u32x4 *>(gate);
  a.c_in[1] = static_cast<const u32x4 *>(up);
  a.c_out[0] = static_cast<u32x4 *>(out);
  a.na = H * es / 16;
  a.nb0 = qn * es / 16;
  a.nb1 = kn * es / 16;
  a.nc = T * I * es / 16;
  a.ga = uint32_t(T);
  a.gb = uint32_t(T);
  int64_t gc = (a.nc + 255) / 256;
  if (gc > (int64_t(1) << 20)) gc = int64_t(1) << 20;
  k_chain_streams<<<dim3(uint32_t(2 * T + gc)), dim3(256), 0,
                    static_cast<hipStream_t>(stream)>>>(a);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Copy n16 16-byte vectors from src to dst (both 16-byte aligned) on
// `stream`. form 0: one vector per work-item; 1: two; 2: four,
// nontemporal. Returns 0, or -1 for bad arguments or a failed launch.
int trib_copy(const void *src, void *dst, int64_t n16, int form, void *stream) {
  if (!src || !dst || n16 < 1 || (uintptr_t(src) | uintptr_t(dst)) % 16) return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (form) {
    case 0: return launch<1, false>(src, dst, n16, s);
    case 1: return launch<2, false>(src, dst, n16, s);
    case 2: return launch<4, true>(src, dst, n16, s);
    default: return -1;
  }
}

}  // extern "C"

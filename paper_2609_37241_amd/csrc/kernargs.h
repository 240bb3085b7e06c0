// Kernel argument blocks: one struct per kernel family, passed by value as
// the kernel's only parameter. Host code fills them on the hit path and hands
// a pointer to the launch; device code reads them from the kernarg segment.
// Plain fixed-width fields only, so host (x86-64) and device (amdgcn) lay
// them out identically; the static_asserts below pin the layout on both
// (with the compiler's own offsetof, as the runtime compiler ships no
// <stddef.h>).
#pragma once
#include <stdint.h>

namespace tri {

// RoPE variant bits: RopeArgs::mode, and key word 3 above the 16-bit rotary
// dim. Bits 8..15 of RopeArgs::mode: workgroups per token of the vector
// forms; bits 16..23: tokens per workgroup of the vector forms (0 or 1 in
// either: one; at most one of the two is above one).
constexpr uint32_t kRopeInterleaved = 1, kRopePos64 = 2, kRopeCache = 4;
constexpr uint32_t kRopeSliceShift = 8, kRopeTokensShift = 16;
constexpr int kRopeTokensMax = 4;

// Work-items of the wide norm workgroup (RN_WIDE): one row of up to
// 8 * kWideLanes 16-byte vectors per workgroup; every other kernel uses 256.
constexpr int kWideLanes = 1024;
// Most workgroups of a plain wide-row launch (one per compute unit of an
// MI355X); beyond that many rows each workgroup takes rows b, b + grid, ...
constexpr int kWideGrid = 256;

// Split norm rows (RN_SPLIT): a row of more than 16 * 256 vectors is held
// by S = ceil(vectors / kSplitSpan) workgroups of 256 work-items, kSplitVecs
// vectors per work-item, which exchange their partial sums of squares
// through a scratch buffer: 8 header words (word 0: a sticky failure flag),
// then T * S slots (row-major, one per workgroup), then T per-row counters.
constexpr int kSplitVecs = 8;
constexpr int kSplitSpan = 256 * kSplitVecs;   // vectors per workgroup
constexpr int kSplitMaxSlices = 64;            // workgroups per row, at most
constexpr int kSplitHeaderWords = 8;

// Residual add + RMSNorm and plain RMSNorm ([T, H] rows, element strides).
struct RnArgs {
  const void *x;
  const void *res;       // residual input (residual variants only)
  const void *w;         // [H]
  void *y;
  void *res_out;         // residual output (residual variants only)
  int64_t x_rs, res_rs, y_rs, ro_rs;
  int64_t T;
  int32_t H;
  float eps;
};

// A split norm launch: the row arguments and the scratch of the call
// (kSplitHeaderWords + T * (S + 1) 64-bit words, all zero when the call
// starts; the kernel leaves them zero).
struct RnSplitArgs {
  RnArgs rn;
  uint64_t *scratch;
};

// RoPE on Q [T, nq, hd] and K [T, nk, hd], in place, over the first rd
// elements of each head; with QK-RMSNorm the whole heads are normalised first
// (qw, kw: [hd] head-norm weights). Angles come from pos and inv_freq, or
// from the cos_sin cache [cs_len, rd] (mode bit kRopeCache).
struct RopeArgs {
  void *q;
  void *k;
  const void *pos;        // int32 [T], or int64 [T] with mode bit kRopePos64
  const float *inv_freq;  // [rd/2], the version's table (null with a cache)
  const void *qw;
  const void *kw;
  const float *cos_sin;
  int64_t q_ts, k_ts;
  int64_t T;
  int64_t cs_len;
  int32_t nq, nk, hd, rd;
  float eps;
  uint32_t mode;          // kRopeInterleaved | kRopePos64 | kRopeCache | slices << 8
};

// SwiGLU over [T, I].
struct SwArgs {
  const void *gate;
  const void *up;
  void *out;
  int64_t g_rs, u_rs, o_rs;
  int64_t T, I;
  int64_t nvec;           // flat variants: whole 16-byte vectors in T*I
  int64_t n;              // flat variants: T*I elements
};

// Element-wise ops over [T, W]: silu(a), a + b, or masked_fill(a, mask b,
// value). Flat variants use nvec whole 16-byte vectors of the contiguous
// T*W elements and n = T*W.
struct EltArgs {
  const void *a;
  const void *b;          // second operand, or the uint8 mask
  void *out;
  int64_t a_rs, b_rs, o_rs;
  int64_t T, W;
  int64_t nvec, n;
  float value;            // masked_fill: fill value (rounded to the dtype on the device)
  int32_t pad;
};

// Embedding: out[t, :] = table[ids[t], :], zeros for ids outside [0, n_rows).
struct EmbArgs {
  const void *table;
  const void *ids;        // int32 or int64 [T]
  void *out;
  int64_t t_rs, o_rs;
  int64_t T, H, n_rows;
  int32_t ids64;
  int32_t pad;
};

// The fused decode chain: rn_blocks workgroups run residual RMSNorm rows,
// rope_blocks run RoPE tokens, the remaining gridDim.x - rn_blocks -
// rope_blocks run SwiGLU (the kernel fixes the order of the three ranges).
struct ChainArgs {
  RnArgs rn;
  RopeArgs rope;
  SwArgs sw;
  uint32_t rn_blocks;
  uint32_t rope_blocks;
};

// An argument block held in device memory for launches without kernel
// arguments: the kernel's argument struct (zero beyond its size), the
// launch's workgroup count and a tag that marks the slot as written
// (kResidentTag + slot; zero until then). Each kernel family has a table of
// kResidentSlots blocks per device and dtype; slot k is found by a launch
// that requests k * kLdsGranule bytes of dynamic LDS (the kernel reads its
// own LDS allocation back). `size` is the host's bookkeeping.
constexpr uint32_t kResidentSlots = 40;        // per device, family and dtype
constexpr uint32_t kResidentTag = 0x52455300u;
constexpr uint32_t kLdsGranule = 1280;         // LDS allocation granule, bytes
constexpr uint32_t kResidentArgsMax = 288;     // the largest argument struct
enum ResidentFamily : uint32_t {
  kResChain = 0,   // the fused decode chain (ChainArgs)
  kResNorm,        // RMSNorm and residual RMSNorm rows (RnArgs, RnSplitArgs)
  kResRope,        // RoPE and QK-RMSNorm + RoPE (RopeArgs)
  kResSwiglu,      // SwiGLU (SwArgs)
  kResElt,         // silu, add, masked_fill (EltArgs)
  kResEmb,         // embedding rows (EmbArgs)
  kResFamilies
};
struct ResidentBlock {
  uint64_t args[kResidentArgsMax / 8];
  uint32_t grid;
  uint32_t tag;
  uint32_t size;
  uint32_t pad0;
  uint64_t pad[2];
};

static_assert(sizeof(RnArgs) == 88 && __builtin_offsetof(RnArgs, T) == 72 &&
                  __builtin_offsetof(RnArgs, eps) == 84,
              "RnArgs layout");
static_assert(sizeof(RnSplitArgs) == 96 && __builtin_offsetof(RnSplitArgs, scratch) == 88,
              "RnSplitArgs layout");
static_assert(sizeof(RopeArgs) == 112 && __builtin_offsetof(RopeArgs, nq) == 88 &&
                  __builtin_offsetof(RopeArgs, mode) == 108,
              "RopeArgs layout");
static_assert(sizeof(SwArgs) == 80 && __builtin_offsetof(SwArgs, n) == 72, "SwArgs layout");
static_assert(sizeof(EltArgs) == 88 && __builtin_offsetof(EltArgs, value) == 80, "EltArgs layout");
static_assert(sizeof(EmbArgs) == 72 && __builtin_offsetof(EmbArgs, ids64) == 64, "EmbArgs layout");
static_assert(sizeof(ChainArgs) == 288 && __builtin_offsetof(ChainArgs, rn_blocks) == 280,
              "ChainArgs layout");
static_assert(sizeof(ResidentBlock) == 320 && __builtin_offsetof(ResidentBlock, grid) == 288 &&
                  __builtin_offsetof(ResidentBlock, tag) == 292,
              "ResidentBlock layout");
static_assert(sizeof(ChainArgs) <= kResidentArgsMax && sizeof(RnSplitArgs) <= kResidentArgsMax,
              "argument structs fit a resident block");

}  // namespace tri

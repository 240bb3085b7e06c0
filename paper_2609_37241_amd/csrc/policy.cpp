// Install policy: which precompiled kernel variant serves a specialization
// key, and how many workgroups a call with T tokens launches.
//
// In the paper a miss captures and compiles a new specialization (Sec. 3.5);
// here every specialization a key can need is already compiled for gfx950,
// and installing a version means choosing among them. The choice is a pure
// function of the key (dtype, sizes, token bucket, alignment and contiguity
// flags, RoPE variant), so the same key always selects the same kernels.
#include <string.h>

#include <initializer_list>

#include "internal.h"

namespace tri {

namespace {

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline int64_t next_pow2(int64_t n) {
  int64_t p = 1;
  while (p < n) p <<= 1;
  return p;
}

inline int64_t vec_elems(uint32_t dtype) { return dtype == TRI_F32 ? 4 : 8; }

inline uint32_t clamp_grid(int64_t g) {
  if (g < 1) return 1;
  return g > int64_t(kGridCap) ? kGridCap : uint32_t(g);
}

int32_t pow2_index(int64_t n) {   // n in {1, 2, 4, 8, 16}
  int32_t i = 0;
  while ((int64_t(1) << i) < n) ++i;
  return i;
}

bool rope_vec_role(int32_t v) {
  return v == ROPE_VEC || v == ROPE_VEC_I || v == ROPE_QKN_VEC || v == ROPE_QKN_VEC_I;
}

}  // namespace

int32_t split_slices(uint32_t dtype, int64_t H) {
  return int32_t(cdiv(H / vec_elems(dtype), kSplitSpan));
}

bool split_fits(uint32_t dtype, int64_t H, uint32_t bucket) {
  const int32_t S = split_slices(dtype, H);
  return S <= kSplitMaxSlices && split_words(int64_t(1) << bucket, S) <= kSplitScratchWords;
}

// Rows of up to 128 16-byte vectors (2 KiB) take one wavefront each, four
// rows per workgroup, with no barrier. Longer rows take one 256-work-item
// workgroup per row, up to 16 vectors per work-item: the four wavefronts
// issue the row's loads and stores in parallel (measured 1.8 µs vs 3.4 µs
// device time for a single 4096-element bf16 row held by one wavefront) and
// hold fewer registers per lane when streaming. Rows beyond 4096 vectors
// are split over S = ceil(vectors / 2048) workgroups of 256 work-items, 8
// vectors per work-item, which exchange partial sums through the version's
// scratch (up to 64 workgroups per row, and a scratch of at most
// kSplitScratchWords for the top of the token bucket). Against the forms
// it replaces, at 256-512 MiB per operand (probe, 1 GiB read flush): bf16
// rows of 49,152 / 65,536 elements 94.9 / 94.5 us vs 97.2 / 101.1 us for a
// 1024-work-item workgroup per row holding the weights with the row
// (residual 176.1 / 177.9 vs 182.2 / 181.8), f32 rows of 32,768 a tie (93.0 / 176.0 us both); bf16 rows of
// 131,072 / 262,144 and f32 rows of 65,536 1.25-1.37x faster than two
// passes over memory. Beyond the split's limits a row of up to
// kWideRowVecs vectors takes the 1024-work-item workgroup and longer rows
// make two passes. Plain RMSNorm rows of 4097..kWidePlainVecs vectors take
// the 1024-work-item workgroups at every bucket, and longer plain rows of up
// to kWideRowVecs vectors from bucket kWidePlainBucket on (more than 256
// rows, where its workgroups each take several rows and overlap one row's
// loads with the previous row's stores): the plain form has no exchange to
// wait for, which the residual form's early residual_out stores hide in the
// split. Against the split at 8192 vectors (bf16 and f32, 256-4096 rows,
// after a 1 GiB read flush and back to back) it took 0.84-0.98 of the
// split's time, except bf16 rows at 2048 and 4096 back to back (1.02). An
// earlier sweep of both forms
// (bf16 and f32 rows of 4097, 5120, 6144, 7168 and 8192 vectors, 1-4096
// rows, back to back and after a 1 GiB read flush) put the split ahead
// only for rows of 8192 vectors (by up to 15 % at 1-64 rows, where four
// workgroups per row pull it from HBM in parallel). Unaligned or ragged
// rows take the scalar kernel.
Role rn_role(uint32_t dtype, int64_t H, unsigned flags, int64_t T, uint32_t bucket, bool res) {
  const int64_t v = vec_elems(dtype);
  if (!(flags & kAlign) || H % v) return {RN_SCALAR, uint32_t(T)};
  const int64_t nvec = H / v;
  if (nvec <= 128) return {nvec <= 64 ? RN_WAVE_1 : RN_WAVE_2, uint32_t(cdiv(T, 4))};
  const int64_t nb = next_pow2(cdiv(nvec, 256));
  if (nb <= 16) return {RN_BLOCK_1 + pow2_index(nb), uint32_t(T)};
  if (!res && nvec <= kWidePlainVecs) return {RN_WIDE, norm_grid(RN_WIDE, dtype, T, H, res)};
  if (!res && nvec <= kWideRowVecs && bucket >= kWidePlainBucket)
    return {RN_WIDE, norm_grid(RN_WIDE, dtype, T, H, res)};
  if (split_fits(dtype, H, bucket)) return {RN_SPLIT, uint32_t(T * split_slices(dtype, H))};
  if (nvec <= kWideRowVecs) return {RN_WIDE, norm_grid(RN_WIDE, dtype, T, H, res)};
  return {RN_LOOP, uint32_t(T)};
}

// Vector RoPE needs the rotated span of a head to split into a power-of-two
// number of 16-byte vectors per work-item group: rd/2 elements per half for
// rotate-half pairs (a work-item holds chunk c of both halves), rd elements
// for GPT-J pairs (a work-item holds one vector of whole pairs). One token per
// workgroup at every size (it also streamed best at 8192 tokens: more
// workgroups, one angle table each). With QK-RMSNorm the vector form needs
// the group to hold the whole head (rd == hd) in at most 64 lanes, since the
// norm's per-head reduction runs over the group's lanes; otherwise the scalar
// form reduces each head with a wavefront.
Role rope_role(uint32_t dtype, int32_t hd, int32_t rd, bool interleaved, unsigned flags, int64_t T,
               bool qk_norm) {
  const int64_t v = vec_elems(dtype);
  const int64_t span = interleaved ? rd : rd / 2;   // elements one group covers per half
  const int64_t cpb = span / v;
  bool vec = (flags & kAlign) && span % v == 0 && cpb > 0 && (cpb & (cpb - 1)) == 0;
  if (qk_norm) vec = vec && rd == hd && cpb <= 64;
  if (!vec) return {qk_norm ? ROPE_QKN_SCALAR : ROPE_SCALAR, uint32_t(T)};
  if (interleaved) return {qk_norm ? ROPE_QKN_VEC_I : ROPE_VEC_I, uint32_t(T)};
  return {qk_norm ? ROPE_QKN_VEC : ROPE_VEC, uint32_t(T)};
}

// At decode sizes a token's RoPE work is latency-bound: a work-item that
// holds two head items runs them back to back. Splitting the heads of a
// token round-robin over S = ceil(heads * cpb / 256) workgroups (at most 4)
// gives every work-item at most one item. Beyond decode sizes one workgroup
// per token already fills the machine.
int32_t rope_slices(uint32_t dtype, int32_t hd, int32_t rd, bool interleaved, int32_t n_heads,
                    uint32_t bucket, int32_t variant) {
  (void)hd;
  const bool vec = variant == ROPE_VEC || variant == ROPE_VEC_I || variant == ROPE_QKN_VEC ||
                   variant == ROPE_QKN_VEC_I;
  if (!vec || bucket > kDecodeBucketMax) return 1;
  const int64_t cpb = (interleaved ? rd : rd / 2) / vec_elems(dtype);
  const int64_t s = cdiv(int64_t(n_heads) * cpb, kBlock);
  return s < 1 ? 1 : (s > 4 ? 4 : int32_t(s));
}

// Beyond decode sizes a token whose heads fill fewer than 256 lanes
// (n_heads * cpb) leaves most of a workgroup idle; a workgroup then takes
// enough tokens to fill its lanes, rounded up to a power of two, at most 4
// (8192 tokens, 8 + 1 heads of 128 bf16: the fused chain 113.0 vs 122.6 us
// with one token per workgroup; with 72 heads one token stays fastest).
int32_t rope_tokens(uint32_t dtype, int32_t rd, bool interleaved, int32_t n_heads,
                    uint32_t bucket, int32_t variant) {
  if (!rope_vec_role(variant) || bucket <= kDecodeBucketMax) return 1;
  const int64_t lanes = int64_t(n_heads) * ((interleaved ? rd : rd / 2) / vec_elems(dtype));
  if (lanes >= int64_t(kBlock)) return 1;
  const int64_t t = next_pow2(cdiv(kBlock, lanes));
  return t > kRopeTokensMax ? kRopeTokensMax : int32_t(t);
}

// Bytes a call at the top of the key's token bucket moves (activations read
// once, outputs written once; weights, positions and tables left out):
// SwiGLU 3 T I elements, the chain 4 T H + 2 T (nq + nk) hd + 3 T I; else 0.
uint64_t call_bytes(const Key &k) {
  const uint64_t T = uint64_t(1) << key_bucket(k), es = key_dtype(k) == TRI_F32 ? 4 : 2;
  const uint32_t op = key_op(k);
  if (op == TRI_OP_SWIGLU) return 3 * T * key_I(k) * es;
  if (op == TRI_OP_CHAIN)
    return T * es *
           (4 * uint64_t(key_H(k)) + 2 * uint64_t(key_nq(k) + key_nk(k)) * key_hd(k) +
            3 * uint64_t(key_I(k)));
  return 0;
}

// Flat SwiGLU, one vector per work-item, standalone and as the fused
// chain's role, streams nontemporally when the call moves more than
// kStreamBytes: below that the operands stay in the 256 MiB last-level
// cache across back-to-back calls and cached loads win (1-7 % at 128-2048
// tokens of Llama-shaped chains, 263-277 MB), above it streaming wins (4-7 %
// at 336-554 MB; in the 8192-token chain 331.5 us against 344-349 us with
// two or four vectors per work-item or SwiGLU dispatched first).
Role sw_role(uint32_t dtype, int64_t I, unsigned flags, bool stream, int64_t T) {
  const int64_t v = vec_elems(dtype);
  if ((flags & kAlign) && (flags & kContig)) {
    const int64_t nvec = (T * I) / v;
    return {stream ? SW_FLAT_NT : SW_FLAT, clamp_grid(cdiv(nvec, kBlock))};
  }
  if ((flags & kAlign) && I % v == 0) {
    const int64_t cb = cdiv(I / v, kBlock);
    const int64_t g = T * cb;
    return {SW_ROWS, g > int64_t(kGridCap) ? kGridCap : uint32_t(g)};
  }
  const int64_t g = cdiv(T * I, kBlock);
  return {SW_SCALAR, g > int64_t(kGridCap) ? kGridCap : uint32_t(g)};
}

// Element-wise ops: flat vectors when aligned and contiguous (beyond decode
// sizes two vectors per work-item, cached: measured 80 / 82 / 79 % of HBM
// peak for add / masked_fill / silu at 8192 x 8192 bf16, against 74-75 %
// nontemporal and 1-4 % less with one or four vectors), vector rows when
// only the rows are aligned, element-wise otherwise.
Role elt_role(uint32_t dtype, int64_t W, unsigned flags, uint32_t bucket, int64_t T) {
  const int64_t v = vec_elems(dtype);
  if ((flags & kAlign) && (flags & kContig)) {
    if (bucket <= kDecodeBucketMax) return {ELT_FLAT, clamp_grid(cdiv((T * W) / v, kBlock))};
    return {ELT_FLAT_U2, clamp_grid(cdiv((T * W) / v, 2 * int64_t(kBlock)))};
  }
  if ((flags & kAlign) && W % v == 0) {
    const int64_t g = T * cdiv(W / v, kBlock);
    return {ELT_ROWS, g > int64_t(kGridCap) ? kGridCap : uint32_t(g)};
  }
  const int64_t g = cdiv(T * W, kBlock);
  return {ELT_SCALAR, g > int64_t(kGridCap) ? kGridCap : uint32_t(g)};
}

// Embedding: one workgroup per output row (grid-stride beyond the cap);
// 16-byte vectors when table and output rows are aligned and H is a whole
// number of vectors, elements otherwise.
Role emb_role(uint32_t dtype, int64_t H, unsigned flags, int64_t T) {
  const int64_t v = vec_elems(dtype);
  return {(flags & kAlign) && H % v == 0 ? EMB_VEC : EMB_SCALAR, clamp_grid(T)};
}

// Workgroups of a role variant for T tokens (I is the row width: the norm
// row H, the SwiGLU width, the row width of an element-wise op, or the
// embedding row width).
uint32_t role_grid(int32_t variant, uint32_t dtype, int64_t T, int64_t I, int32_t slices,
                   int32_t tokens) {
  if (variant == RN_WAVE_1 || variant == RN_WAVE_2) return uint32_t(cdiv(T, 4));
  if (variant == RN_SPLIT) return uint32_t(T * split_slices(dtype, I));
  switch (variant) {
    case RN_SCALAR: case RN_BLOCK_1: case RN_BLOCK_2: case RN_BLOCK_4: case RN_BLOCK_8:
    case RN_BLOCK_16: case RN_LOOP: case RN_WIDE: case ROPE_SCALAR: case ROPE_QKN_SCALAR:
      return uint32_t(T);
    case ROPE_VEC: case ROPE_VEC_I: case ROPE_QKN_VEC: case ROPE_QKN_VEC_I:
      return slices > 1 ? uint32_t(T * slices) : uint32_t(cdiv(T, tokens < 1 ? 1 : tokens));
    case SW_FLAT: case SW_FLAT_NT: case ELT_FLAT:
      return clamp_grid(cdiv((T * I) / vec_elems(dtype), kBlock));
    case ELT_FLAT_U2:
      return clamp_grid(cdiv((T * I) / vec_elems(dtype), 2 * int64_t(kBlock)));
    case EMB_VEC: case EMB_SCALAR:
      return clamp_grid(T);
    case SW_ROWS: case ELT_ROWS: {
      const int64_t g = T * cdiv(I / vec_elems(dtype), kBlock);
      return g > int64_t(kGridCap) ? kGridCap : uint32_t(g);
    }
    case SW_SCALAR: case ELT_SCALAR: {
      const int64_t g = cdiv(T * I, kBlock);
      return g > int64_t(kGridCap) ? kGridCap : uint32_t(g);
    }
    default:
      return 0;
  }
}

uint32_t norm_grid(int32_t variant, uint32_t dtype, int64_t T, int64_t H, bool res) {
  if (variant == RN_WIDE && !res && T > kWideGrid) return uint32_t(kWideGrid);
  return role_grid(variant, dtype, T, H);
}

int64_t launch_width(const Key &k, int32_t kv) {
  const uint32_t op = key_op(k);
  if (is_norm_variant(kv) || (op >= TRI_OP_SILU && op <= TRI_OP_EMBEDDING)) return key_H(k);
  return key_I(k);
}

namespace {

// Template index of the fused chain kernel (see Plan::ksub).
int32_t fused_sub(int32_t rn, int32_t rope, int32_t sw) {
  const bool inter = rope == ROPE_VEC_I || rope == ROPE_QKN_VEC_I;
  const bool qkn = rope == ROPE_QKN_VEC || rope == ROPE_QKN_VEC_I;
  return (rn - RN_WAVE_1) * 8 + (inter ? 4 : 0) + (qkn ? 2 : 0) + (sw == SW_FLAT_NT ? 1 : 0);
}

}  // namespace

// A key the entry points could have produced (used to check imported keys):
// the same limits as argument validation, unused fields zero.
bool key_valid(const Key &k) {
  const uint32_t op = key_op(k), dt = key_dtype(k), fl = key_flags(k);
  const bool short_op = op >= TRI_OP_SILU && op <= TRI_OP_EMBEDDING;
  if ((op < TRI_OP_RMSNORM || op > TRI_OP_QK_NORM_ROPE) && !short_op) return false;
  if (dt != TRI_F32 && dt != TRI_BF16) return false;
  if (key_bucket(k) > 22) return false;
  const bool chain = op == TRI_OP_CHAIN;
  if (fl > (chain ? 0x7Fu : 0x3u)) return false;
  if (short_op) {   // width in the H field; embedding: bit 16 of k3 = int64 ids
    const uint64_t W = key_H(k);
    if (W < 1 || int64_t(W) >= kILimit || key_I(k) != 0) return false;
    if (op == TRI_OP_EMBEDDING && (fl & kContig)) return false;
    const uint64_t k3_ok = op == TRI_OP_EMBEDDING ? (uint64_t(1) << 16) : 0;
    return (k.k0 >> 32) == 0 && k.k2 == 0 && (k.k3 & ~k3_ok) == 0 && k.k4 == 0 && k.k5 == 0;
  }
  const bool norm = op == TRI_OP_RMSNORM || op == TRI_OP_RES_RMSNORM || chain;
  const bool sw = op == TRI_OP_SWIGLU || chain;
  const bool rope = op == TRI_OP_ROPE_QK || op == TRI_OP_QK_NORM_ROPE || chain;
  const uint64_t H = key_H(k), I = key_I(k);
  if (norm ? (H < 1 || int64_t(H) >= kHLimit) : H != 0) return false;
  if (sw ? (I < 1 || int64_t(I) >= kILimit) : I != 0) return false;
  if (!rope) return k.k0 >> 32 == 0 && k.k2 == 0 && k.k3 == 0 && k.k4 == 0 && k.k5 == 0;
  const uint32_t hd = key_hd(k), nq = key_nq(k), nk = key_nk(k), rd = key_rd(k);
  if (k.k2 >> 48) return false;
  if (hd < 2 || (hd & 1) || int32_t(hd) > kHdMax) return false;
  if (nq < 1 || int32_t(nq) > kHeadsMax || int32_t(nk) > kHeadsMax) return false;
  if (rd < 2 || (rd & 1) || rd > hd) return false;
  const uint32_t bits = key_rope_bits(k), scaling = key_scaling(k);
  if (bits > 7) return false;
  if (bits & kRopeCache) return (k.k3 >> 24) == 0 && k.k0 >> 32 == 0 && k.k4 == 0 && k.k5 == 0;
  float base, f, lo, hi;
  const uint32_t bb = key_base_bits(k), fb = uint32_t(k.k4), lb = uint32_t(k.k4 >> 32),
                 hb = uint32_t(k.k5);
  memcpy(&base, &bb, 4);
  if (!(base > 1.0f && base <= 3.4028235e38f)) return false;   // finite, > 1 (NaN fails)
  if (scaling == TRI_ROPE_SCALING_NONE) return (k.k3 >> 24) == 0 && k.k4 == 0 && k.k5 == 0;
  if (scaling != TRI_ROPE_SCALING_LLAMA3 || k.k5 >> 32) return false;
  memcpy(&f, &fb, 4);
  memcpy(&lo, &lb, 4);
  memcpy(&hi, &hb, 4);
  const float fmax = 3.4028235e38f;
  if (!(f > 0.0f && f <= fmax) || !(lo > 0.0f && lo <= fmax) || !(hi > lo && hi <= fmax))
    return false;
  return int32_t(key_orig_max(k)) >= 1;
}

Plan plan_for_key(const Key &k) {
  const uint32_t op = key_op(k), dt = key_dtype(k), b = key_bucket(k), fl = key_flags(k);
  Plan p{};
  p.rope_slices = 1;
  p.rope_tokens = 1;
  // The grid does not affect the choice of variant; T = 1 stands in here.
  switch (op) {
    case TRI_OP_RMSNORM:
    case TRI_OP_RES_RMSNORM: {
      const Role r = rn_role(dt, key_H(k), fl, 1, b, op == TRI_OP_RES_RMSNORM);
      p.variant = r.variant;
      p.n_launches = 1;
      p.kvariant[0] = r.variant;
      p.ksub[0] = op == TRI_OP_RES_RMSNORM ? 1 : 0;
      return p;
    }
    case TRI_OP_ROPE_QK:
    case TRI_OP_QK_NORM_ROPE: {
      const bool inter = (key_rope_bits(k) & kRopeInterleaved) != 0;
      const Role r = rope_role(dt, int32_t(key_hd(k)), int32_t(key_rd(k)), inter, fl, 1,
                               op == TRI_OP_QK_NORM_ROPE);
      p.variant = r.variant;
      p.n_launches = 1;
      p.kvariant[0] = r.variant;
      p.rope_slices = rope_slices(dt, int32_t(key_hd(k)), int32_t(key_rd(k)), inter,
                                  int32_t(key_nq(k) + key_nk(k)), b, r.variant);
      p.rope_tokens = rope_tokens(dt, int32_t(key_rd(k)), inter, int32_t(key_nq(k) + key_nk(k)),
                                  b, r.variant);
      return p;
    }
    case TRI_OP_SILU:
    case TRI_OP_ADD:
    case TRI_OP_MASKED_FILL: {
      const Role r = elt_role(dt, key_H(k), fl, b, 1);
      p.variant = r.variant;
      p.n_launches = 1;
      p.kvariant[0] = r.variant;
      p.ksub[0] = int32_t(op);
      return p;
    }
    case TRI_OP_EMBEDDING: {
      const Role r = emb_role(dt, key_H(k), fl, 1);
      p.variant = r.variant;
      p.n_launches = 1;
      p.kvariant[0] = r.variant;
      p.ksub[0] = int32_t(key_rope_bits(k) & 1);   // int64 ids
      return p;
    }
    case TRI_OP_SWIGLU: {
      const Role r = sw_role(dt, key_I(k), fl, call_bytes(k) > kStreamBytes, 1);
      p.variant = r.variant;
      p.n_launches = 1;
      p.kvariant[0] = r.variant;
      return p;
    }
    default:
      break;
  }
  const Role rn = rn_role(dt, key_H(k), fl & 3u, 1, b, true);
  const bool inter = (key_rope_bits(k) & kRopeInterleaved) != 0;
  const Role ro = rope_role(dt, int32_t(key_hd(k)), int32_t(key_rd(k)), inter, (fl >> 2) & 3u, 1,
                            (fl & kChainQkNorm) != 0);
  p.rope_slices = rope_slices(dt, int32_t(key_hd(k)), int32_t(key_rd(k)), inter,
                              int32_t(key_nq(k) + key_nk(k)), b, ro.variant);
  p.rope_tokens = rope_tokens(dt, int32_t(key_rd(k)), inter, int32_t(key_nq(k) + key_nk(k)), b,
                              ro.variant);
  const Role sw = sw_role(dt, key_I(k), (fl >> 4) & 3u, call_bytes(k) > kStreamBytes, 1);
  p.roles[0] = rn.variant;
  p.roles[1] = ro.variant;
  p.roles[2] = sw.variant;
  const bool rn_regs = rn.variant >= RN_WAVE_1 && rn.variant <= RN_BLOCK_16;
  const bool ro_vec = rope_vec_role(ro.variant);
  const bool sw_flat = sw.variant == SW_FLAT || sw.variant == SW_FLAT_NT;
  if ((fl & 0x3Fu) == 0x3Fu && rn_regs && ro_vec && sw_flat) {
    p.variant = CH_FUSED;
    p.n_launches = 1;
    p.kvariant[0] = CH_FUSED;
    p.ksub[0] = fused_sub(rn.variant, ro.variant, sw.variant);
    return p;
  }
  p.variant = CH_SEQ;
  p.n_launches = 3;
  p.kvariant[0] = rn.variant;
  p.ksub[0] = 1;   // residual flavour
  p.kvariant[1] = ro.variant;
  p.kvariant[2] = sw.variant;
  return p;
}

// ---- generic guards ------------------------------------------------------------------
namespace {

Key with_bucket(const Key &k, uint32_t b) {
  Key x = k;
  x.k0 = (x.k0 & ~(uint64_t(0xFF) << 16)) | (uint64_t(b) << 16);
  return x;
}

// The row lengths served by the norm kernel rn_role picks for H at every
// bucket: unaligned rows take the scalar kernel at any length, aligned
// ragged ones at every length that is not a whole number of vectors; rows
// of whole vectors one wavefront (1-64, 65-128 vectors) or one workgroup
// (129-256, 257-512, ..., 2049-4096 vectors; plain rows also 4097-8192 in
// the 1024-lane workgroup). Longer rows: none (their kernel depends on the
// bucket through the split's scratch).
bool norm_h_range(uint32_t dt, uint32_t H, unsigned fl, bool res, Guard *g) {
  const int64_t v = vec_elems(dt);
  if (!(fl & kAlign) || H % v) {
    g->h_lo = 1;
    g->h_hi = uint32_t(kHLimit - 1);
    g->h_mod = (fl & kAlign) ? TRI_H_RAGGED : TRI_H_ANY;
    return true;
  }
  const int64_t n = int64_t(H) / v;
  int64_t lo, hi;
  if (n <= 64) {
    lo = 1, hi = 64;
  } else if (n <= 128) {
    lo = 65, hi = 128;
  } else if (n <= 4096) {
    const int64_t nb = next_pow2(cdiv(n, 256));
    lo = nb == 1 ? 129 : 128 * nb + 1;
    hi = 256 * nb;
  } else if (!res && n <= kWidePlainVecs) {
    lo = 4097, hi = kWidePlainVecs;
  } else {
    return false;
  }
  g->h_lo = uint32_t(lo * v);
  g->h_hi = uint32_t(hi * v);
  g->h_mod = TRI_H_MULTIPLE;
  return true;
}

}  // namespace

bool splits_rows(const Plan &p) {
  for (int i = 0; i < p.n_launches; ++i)
    if (p.kvariant[i] == RN_SPLIT) return true;
  return p.roles[0] == RN_SPLIT;
}

Guard generic_guard(const Key &k, const Plan &chosen) {
  const Plan P = plan_for_key(k);
  const uint32_t b = key_bucket(k);
  uint32_t lo = b, hi = b;
  while (lo > 0 && plan_for_key(with_bucket(k, lo - 1)) == P) --lo;
  while (hi < kBucketMax && plan_for_key(with_bucket(k, hi + 1)) == P) ++hi;
  // A split version's scratch is sized for the top of its run: keep only
  // the buckets whose scratch fits (the policy's own split stops there
  // already; a tuned split choice is clamped here).
  // It also matches only its own row length: the scratch is sized by the
  // row's slice count.
  const bool splits = splits_rows(chosen);
  if (splits)
    while (hi > b && !split_fits(key_dtype(k), key_H(k), hi)) --hi;
  Guard g = kExact;
  g.b_lo = int32_t(lo);
  g.b_hi = int32_t(hi);
  const uint32_t op = key_op(k);
  if ((op == TRI_OP_RMSNORM || op == TRI_OP_RES_RMSNORM) && !splits) {
    Guard h = g;
    if (norm_h_range(key_dtype(k), key_H(k), key_flags(k), op == TRI_OP_RES_RMSNORM, &h)) g = h;
  }
  return g;
}

bool guard_holds(const Key &vk, const Guard &g, const Key &k) {
  if (g.b_lo < 0) return vk == k;
  const uint64_t bucket_bits = uint64_t(0xFF) << 16;
  if ((vk.k0 & ~bucket_bits) != (k.k0 & ~bucket_bits)) return false;
  const int32_t b = int32_t(key_bucket(k));
  if (b < g.b_lo || b > g.b_hi) return false;
  if (g.h_lo) {   // word 1: H in the low half, I in the high half
    if ((vk.k1 >> 32) != (k.k1 >> 32)) return false;
    const uint32_t H = key_H(k);
    if (H < g.h_lo || H > g.h_hi) return false;
    const uint32_t v = key_dtype(vk) == TRI_F32 ? 4u : 8u;
    if ((g.h_mod == TRI_H_MULTIPLE && H % v) || (g.h_mod == TRI_H_RAGGED && H % v == 0))
      return false;
  } else if (vk.k1 != k.k1) {
    return false;
  }
  return vk.k2 == k.k2 && vk.k3 == k.k3 && vk.k4 == k.k4 && vk.k5 == k.k5;
}

// ---- candidate plans of install-time tuning ---------------------------------------
// Index 0 is the policy's plan. The others are the kernel variants whose
// requirements the key also meets: a norm row held by one wavefront can be
// held by one workgroup (one vector per lane), a row of more than 1024
// vectors held by a 256-lane workgroup can be held by a 1024-lane one (and,
// beyond 2048 vectors, split over workgroups), a split row of at most 8192
// vectors by a 1024-lane workgroup, and a row held in registers can take
// the two-pass kernel (standalone only); a vector RoPE role can
// take another geometry (at decode sizes 1, 2 or 4 workgroups per token;
// beyond them 1, 2 or 4 tokens per workgroup, or up to 8192 tokens 2 or 4
// workgroups per token) or the scalar kernel; flat SwiGLU and element-wise kernels have a cached
// and a streaming (SwiGLU: nontemporal; element-wise: two vectors per
// work-item) form and a row form when a row is whole vectors. The fused
// chain takes every combination of its roles' options (norm, then slices,
// then SwiGLU form, each starting with the policy's choice), then the
// three-launch sequence of the policy's roles.
namespace {

int rn_options(uint32_t dt, int64_t H, unsigned fl, uint32_t b, bool standalone, bool res,
               int32_t *out) {
  const int32_t P = rn_role(dt, H, fl, 1, b, res).variant;
  int n = 0;
  out[n++] = P;
  if (P == RN_SCALAR || P == RN_LOOP) return n;
  if (P == RN_WAVE_1 || P == RN_WAVE_2) out[n++] = RN_BLOCK_1;
  if (!standalone) return n;
  if (P == RN_BLOCK_8 || P == RN_BLOCK_16) {
    out[n++] = RN_WIDE;
    // a split row is at least two workgroups: rows beyond 2048 vectors
    if (P == RN_BLOCK_16 &&
        split_words(int64_t(1) << b, split_slices(dt, H)) <= kSplitScratchWords)
      out[n++] = RN_SPLIT;
  }
  if (P == RN_SPLIT && H / vec_elems(dt) <= kWideRowVecs) out[n++] = RN_WIDE;
  if (P == RN_WIDE && split_fits(dt, H, b)) out[n++] = RN_SPLIT;
  out[n++] = RN_LOOP;
  return n;
}

// (slices, tokens per workgroup) of a vector RoPE role, the policy's first:
// at decode sizes slice counts 1, 2, 4; beyond them 1, 2, 4 tokens per
// workgroup, then (up to bucket 13) 2 and 4 slices of one token.
struct Geometry {
  int32_t slices, tokens;
};

int geometry_options(int32_t S, int32_t P, uint32_t bucket, Geometry *out) {
  const int32_t choices[3] = {1, 2, 4};
  int n = 0;
  if (bucket <= kDecodeBucketMax) {
    out[n++] = {S, 1};
    for (int32_t c : choices)
      if (c != S) out[n++] = {c, 1};
    return n;
  }
  out[n++] = {1, P};
  for (int32_t c : choices)
    if (c != P) out[n++] = {1, c};
  if (bucket <= kSliceBucketMax) {
    out[n++] = {2, 1};
    out[n++] = {4, 1};
  }
  return n;
}

Plan single(int32_t variant, int32_t sub, Geometry g = {1, 1}) {
  Plan p{};
  p.variant = variant;
  p.n_launches = 1;
  p.kvariant[0] = variant;
  p.ksub[0] = sub;
  p.rope_slices = g.slices;
  p.rope_tokens = g.tokens;
  return p;
}

}  // namespace

int plan_candidates(const Key &k, Plan *out) {
  const Plan P = plan_for_key(k);
  const uint32_t op = key_op(k), dt = key_dtype(k), b = key_bucket(k), fl = key_flags(k);
  const int64_t v = vec_elems(dt);
  int n = 0;
  out[n++] = P;
  switch (op) {
    case TRI_OP_RMSNORM:
    case TRI_OP_RES_RMSNORM: {
      int32_t r[4];
      const int nr = rn_options(dt, key_H(k), fl, b, true, op == TRI_OP_RES_RMSNORM, r);
      for (int i = 1; i < nr; ++i) out[n++] = single(r[i], P.ksub[0]);
      return n;
    }
    case TRI_OP_ROPE_QK:
    case TRI_OP_QK_NORM_ROPE: {
      if (!rope_vec_role(P.variant)) return n;
      Geometry g[5];
      const int ng = geometry_options(P.rope_slices, P.rope_tokens, b, g);
      for (int i = 1; i < ng; ++i) out[n++] = single(P.variant, 0, g[i]);
      out[n++] = single(op == TRI_OP_QK_NORM_ROPE ? ROPE_QKN_SCALAR : ROPE_SCALAR, 0);
      return n;
    }
    case TRI_OP_SWIGLU:
      if (P.variant == SW_FLAT || P.variant == SW_FLAT_NT) {
        out[n++] = single(P.variant == SW_FLAT ? SW_FLAT_NT : SW_FLAT, 0);
        if (key_I(k) % v == 0) out[n++] = single(SW_ROWS, 0);
      }
      return n;
    case TRI_OP_SILU:
    case TRI_OP_ADD:
    case TRI_OP_MASKED_FILL:
      if (P.variant == ELT_FLAT || P.variant == ELT_FLAT_U2) {
        out[n++] = single(P.variant == ELT_FLAT ? ELT_FLAT_U2 : ELT_FLAT, int32_t(op));
        if (key_H(k) % v == 0) out[n++] = single(ELT_ROWS, int32_t(op));
      }
      return n;
    case TRI_OP_CHAIN:
      break;
    default:
      return n;
  }
  if (P.variant != CH_FUSED) return n;
  int32_t r[4];
  Geometry g[5];
  const int nr = rn_options(dt, key_H(k), fl & 3u, b, false, true, r);
  const int ng = geometry_options(P.rope_slices, P.rope_tokens, b, g);
  const int32_t sw0 = P.roles[2], sw1 = sw0 == SW_FLAT ? SW_FLAT_NT : SW_FLAT;
  n = 0;
  for (int i = 0; i < nr; ++i)
    for (int j = 0; j < ng; ++j)
      for (int32_t w : {sw0, sw1}) {
        Plan c{};
        c.variant = CH_FUSED;
        c.roles[0] = r[i];
        c.roles[1] = P.roles[1];
        c.roles[2] = w;
        c.n_launches = 1;
        c.kvariant[0] = CH_FUSED;
        c.ksub[0] = fused_sub(r[i], P.roles[1], w);
        c.rope_slices = g[j].slices;
        c.rope_tokens = g[j].tokens;
        out[n++] = c;
      }
  Plan q{};
  q.variant = CH_SEQ;
  q.roles[0] = P.roles[0];
  q.roles[1] = P.roles[1];
  q.roles[2] = P.roles[2];
  q.n_launches = 3;
  q.kvariant[0] = P.roles[0];
  q.ksub[0] = 1;
  q.kvariant[1] = P.roles[1];
  q.kvariant[2] = P.roles[2];
  q.rope_slices = P.rope_slices;
  q.rope_tokens = P.rope_tokens;
  out[n++] = q;
  return n;
}

}  // namespace tri

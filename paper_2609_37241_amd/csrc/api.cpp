// The op entry points: the cache-hit path.
//
// One call = validate arguments -> pack the guard key -> ordered lookup
// (Algorithm 1, Sec. 3.2) -> fill the kernel's argument block -> launch the
// version's resolved kernel on the caller's stream (Sec. 3.3: the launch
// preconditions are checked right before submission). Nothing on this path
// allocates, logs, or queries the runtime. A miss returns TRI_MISS with
// nothing launched; an error returns a negative status, tries no other
// version and installs nothing (Sec. 3.5).
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include "internal.h"
#include "kernargs.h"

using namespace tri;

namespace {

enum { kGo = 2 };   // validation passed, continue (distinct from every status)

inline uint64_t es_of(uint32_t dtype) { return dtype == TRI_F32 ? 4u : 2u; }
inline uint64_t addr(const void *p) { return uint64_t(uintptr_t(p)); }

// Status of a call that ended before lookup: T == 0 (OK) or an error.
tri_status finish_early(tri_cache *c, uint32_t op, int st) {
  if (st == TRI_OK)
    c->stats.empty++;
  else
    c->stats.errors++;
  tri_selection &r = c->last;
  memset(&r, 0, sizeof r);
  r.op = int32_t(op);
  r.status = st;
  r.version = -1;
  return tri_status(st);
}

inline int check_common(int32_t dtype, int64_t T) {
  if (dtype != TRI_F32 && dtype != TRI_BF16) return TRI_E_INVALID;
  if (T < 0) return TRI_E_INVALID;
  if (T == 0) return TRI_OK;
  if (T > kTMax) return TRI_E_UNSUPPORTED;
  return kGo;
}

// `rows` rows of `width` elements, `stride` elements apart (stride >= width
// >= 1, rows >= 1): their span ((rows - 1) * stride + width) * es must not
// exceed kSpanMax bytes. No memory that large exists, and within it every
// offset a kernel forms stays far from int64 overflow.
inline bool extent_ok(int64_t rows, int64_t stride, int64_t width, uint64_t es) {
  const uint64_t lim = kSpanMax / es;
  if (uint64_t(width) > lim) return false;
  return rows <= 1 || uint64_t(stride) <= (lim - uint64_t(width)) / uint64_t(rows - 1);
}

// Norm rows: H range, non-null and element-aligned pointers, strides >= H
// and within the extent limit over T rows, finite non-negative eps.
inline int check_norm(uint64_t es, int64_t T, int64_t H, const void *const *ptrs, int np,
                      const int64_t *strides, int ns, float eps) {
  if (H < 1) return TRI_E_INVALID;
  if (H >= kHLimit) return TRI_E_UNSUPPORTED;
  for (int i = 0; i < np; ++i)
    if (!ptrs[i]) return TRI_E_INVALID;
  for (int i = 0; i < np; ++i)
    if (addr(ptrs[i]) % es) return TRI_E_INVALID;
  for (int i = 0; i < ns; ++i)
    if (strides[i] < H || !extent_ok(T, strides[i], H, es)) return TRI_E_INVALID;
  if (!isfinite(eps) || eps < 0.0f) return TRI_E_INVALID;
  return kGo;
}

// The plain rotation: rotate-half over the whole head, int32 positions,
// computed angles without scaling.
const tri_rope_ext kRopePlain = {0, 0, 0, TRI_ROPE_SCALING_NONE, 0.0f, 0.0f, 0.0f, 0, nullptr, 0};

// RoPE arguments in the documented order: head_dim and head counts; the
// variant fields; pointers and their alignment; strides; the angle source.
inline int check_rope(uint64_t es, int64_t T, const void *q, int64_t q_ts, const void *k,
                      int64_t k_ts, const void *pos, int32_t nq, int32_t nk, int32_t hd,
                      float base, const tri_rope_ext &x) {
  if (hd < 2 || (hd & 1)) return TRI_E_INVALID;
  if (hd > kHdMax) return TRI_E_UNSUPPORTED;
  if (nq < 1 || nk < 0) return TRI_E_INVALID;
  if (nq > kHeadsMax || nk > kHeadsMax) return TRI_E_UNSUPPORTED;
  if (x.rotary_dim != 0 && (x.rotary_dim < 2 || (x.rotary_dim & 1) || x.rotary_dim > hd))
    return TRI_E_INVALID;
  if ((x.interleaved | 1) != 1 || (x.pos_int64 | 1) != 1) return TRI_E_INVALID;
  if (x.scaling != TRI_ROPE_SCALING_NONE && x.scaling != TRI_ROPE_SCALING_LLAMA3)
    return TRI_E_INVALID;
  if (!q || !pos || (nk > 0 && !k)) return TRI_E_INVALID;
  if (addr(pos) % (x.pos_int64 ? 8 : 4)) return TRI_E_INVALID;
  if (addr(q) % es || (nk > 0 && addr(k) % es)) return TRI_E_INVALID;
  if (q_ts < int64_t(nq) * hd || !extent_ok(T, q_ts, int64_t(nq) * hd, es))
    return TRI_E_INVALID;
  if (nk > 0 && (k_ts < int64_t(nk) * hd || !extent_ok(T, k_ts, int64_t(nk) * hd, es)))
    return TRI_E_INVALID;
  if (x.cos_sin) {
    const int64_t rd = x.rotary_dim ? x.rotary_dim : hd;
    if (addr(x.cos_sin) % 4 || x.cos_sin_len < 1 || !extent_ok(x.cos_sin_len, rd, rd, 4) ||
        x.scaling != TRI_ROPE_SCALING_NONE)
      return TRI_E_INVALID;
    return kGo;
  }
  if (!isfinite(base) || base <= 1.0f) return TRI_E_INVALID;
  if (x.scaling == TRI_ROPE_SCALING_LLAMA3) {
    if (!isfinite(x.factor) || x.factor <= 0.0f) return TRI_E_INVALID;
    if (!isfinite(x.low_freq_factor) || x.low_freq_factor <= 0.0f) return TRI_E_INVALID;
    if (!isfinite(x.high_freq_factor) || x.high_freq_factor <= x.low_freq_factor)
      return TRI_E_INVALID;
    if (x.original_max_pos < 1) return TRI_E_INVALID;
  }
  return kGo;
}

// Head-norm weights of QK-RMSNorm: q_w always, k_w when there are K heads;
// element-aligned; finite non-negative eps.
inline int check_qkn(uint64_t es, const void *q_w, const void *k_w, int32_t nk, float eps) {
  if (!q_w || (nk > 0 && !k_w)) return TRI_E_INVALID;
  if (addr(q_w) % es || (nk > 0 && addr(k_w) % es)) return TRI_E_INVALID;
  if (!isfinite(eps) || eps < 0.0f) return TRI_E_INVALID;
  return kGo;
}

inline int check_sw(uint64_t es, int64_t T, int64_t I, const void *g, int64_t g_rs,
                    const void *u, int64_t u_rs, const void *o, int64_t o_rs) {
  if (I < 1) return TRI_E_INVALID;
  if (I >= kILimit) return TRI_E_UNSUPPORTED;
  if (!g || !u || !o) return TRI_E_INVALID;
  if ((addr(g) | addr(u) | addr(o)) % es) return TRI_E_INVALID;
  if (g_rs < I || u_rs < I || o_rs < I) return TRI_E_INVALID;
  if (!extent_ok(T, g_rs, I, es) || !extent_ok(T, u_rs, I, es) || !extent_ok(T, o_rs, I, es))
    return TRI_E_INVALID;
  return kGo;
}

// ---- guard flags --------------------------------------------------------------
inline unsigned flags_of(uint64_t or_bits, bool contig) {
  return ((or_bits & 15u) == 0 ? kAlign : 0u) | (contig ? kContig : 0u);
}

inline unsigned rn_flags(uint64_t es, const void *x, int64_t x_rs, const void *w, const void *y,
                         int64_t y_rs, int64_t H) {
  const uint64_t o = addr(x) | addr(w) | addr(y) | uint64_t(x_rs) * es | uint64_t(y_rs) * es;
  return flags_of(o, x_rs == H && y_rs == H);
}

inline unsigned res_flags(uint64_t es, const void *x, int64_t x_rs, const void *r, int64_t r_rs,
                          const void *w, const void *y, int64_t y_rs, const void *ro,
                          int64_t ro_rs, int64_t H) {
  const uint64_t o = addr(x) | addr(r) | addr(w) | addr(y) | addr(ro) | uint64_t(x_rs) * es |
                     uint64_t(r_rs) * es | uint64_t(y_rs) * es | uint64_t(ro_rs) * es;
  return flags_of(o, x_rs == H && r_rs == H && y_rs == H && ro_rs == H);
}

// With QK-RMSNorm (q_w non-null) the head-norm weights join the alignment test.
inline unsigned rope_flags(uint64_t es, const void *q, int64_t q_ts, const void *k, int64_t k_ts,
                           int32_t nq, int32_t nk, int32_t hd, const void *q_w = nullptr,
                           const void *k_w = nullptr) {
  uint64_t o = addr(q) | uint64_t(q_ts) * es | addr(q_w);
  bool contig = q_ts == int64_t(nq) * hd;
  if (nk > 0) {
    o |= addr(k) | uint64_t(k_ts) * es;
    if (q_w) o |= addr(k_w);
    contig = contig && k_ts == int64_t(nk) * hd;
  }
  return flags_of(o, contig);
}

inline unsigned sw_flags(uint64_t es, const void *g, int64_t g_rs, const void *u, int64_t u_rs,
                         const void *o, int64_t o_rs, int64_t I) {
  const uint64_t b = addr(g) | addr(u) | addr(o) | uint64_t(g_rs) * es | uint64_t(u_rs) * es |
                     uint64_t(o_rs) * es;
  return flags_of(b, g_rs == I && u_rs == I && o_rs == I);
}

inline uint32_t f32_bits(float f) {
  uint32_t b;
  memcpy(&b, &f, sizeof b);
  return b;
}

inline Key make_key(uint32_t op, uint32_t dtype, int64_t T, unsigned flags, uint32_t base_bits,
                    uint64_t H, uint64_t I, uint64_t hd, uint64_t nq, uint64_t nk) {
  Key k;
  k.k0 = uint64_t(op) | (uint64_t(dtype) << 8) | (uint64_t(token_bucket(T)) << 16) |
         (uint64_t(flags) << 24) | (uint64_t(base_bits) << 32);
  k.k1 = H | (I << 32);
  k.k2 = hd | (nq << 16) | (nk << 32);
  k.k3 = k.k4 = k.k5 = 0;
  return k;
}

// The RoPE variant words of a key (k3..k5) and the base bits of k0. With a
// cos/sin cache the base and scaling fields are unused and stay zero.
inline void rope_key_words(Key &k, int32_t hd, float base, const tri_rope_ext &x) {
  const uint64_t rd = uint64_t(x.rotary_dim ? x.rotary_dim : hd);
  const uint64_t bits = (x.interleaved ? kRopeInterleaved : 0u) | (x.pos_int64 ? kRopePos64 : 0u) |
                        (x.cos_sin ? kRopeCache : 0u);
  k.k3 = rd | (bits << 16);
  if (x.cos_sin) return;
  k.k0 |= uint64_t(f32_bits(base)) << 32;
  if (x.scaling == TRI_ROPE_SCALING_LLAMA3) {
    k.k3 |= (uint64_t(TRI_ROPE_SCALING_LLAMA3) << 24) | (uint64_t(uint32_t(x.original_max_pos)) << 32);
    k.k4 = uint64_t(f32_bits(x.factor)) | (uint64_t(f32_bits(x.low_freq_factor)) << 32);
    k.k5 = uint64_t(f32_bits(x.high_freq_factor));
  }
}

// Kernel arguments of the RoPE role (q_w null: no head norm).
inline RopeArgs rope_args(const Version &v, void *q, int64_t q_ts, void *kp, int64_t k_ts,
                          const void *pos, int64_t T, int32_t nq, int32_t nk, int32_t hd,
                          const tri_rope_ext &x, const void *q_w, const void *k_w, float eps) {
  const uint32_t mode = (x.interleaved ? kRopeInterleaved : 0u) |
                        (x.pos_int64 ? kRopePos64 : 0u) | (x.cos_sin ? kRopeCache : 0u) |
                        rope_geometry_bits(v.plan.rope_slices, v.plan.rope_tokens);
  return RopeArgs{q, nk > 0 ? kp : nullptr, pos, v.d_consts, q_w, (q_w && nk > 0) ? k_w : nullptr,
                  x.cos_sin, q_ts, k_ts, T, x.cos_sin ? x.cos_sin_len : 0, nq, nk, hd,
                  x.rotary_dim ? x.rotary_dim : hd, q_w ? eps : 0.0f, mode};
}

// ---- lookup and launch bookkeeping -----------------------------------------------------
// Finds the version for `k`. On a miss records it and, with auto-install,
// installs and returns the new version (*auto_inst = true).
// The bookkeeping of a miss: counter, recorded key, selection record.
inline tri_selection &note_miss(tri_cache *c, uint32_t op, const Key &k, int64_t T) {
  c->stats.misses++;
  c->has_miss = true;
  c->miss_key = k;
  c->miss_T = T;
  tri_selection &r = c->last;
  memset(&r, 0, sizeof r);
  r.op = int32_t(op);
  r.version = -1;
  key_words(k, r.key);
  r.status = TRI_MISS;
  return r;
}

inline int lookup(tri_cache *c, uint32_t op, const Key &k, int64_t T, int32_t *vi,
                  bool *auto_inst) {
  int32_t i = find_version(c, op, k);
  if (i >= 0) {
    *vi = i;
    return TRI_OK;
  }
  tri_selection &r = note_miss(c, op, k, T);
  if (!(c->flags & TRI_CACHE_AUTO_INSTALL)) return TRI_MISS;
  const tri_status st = install_key(c, k, -1, (c->flags & TRI_CACHE_GENERIC) != 0);
  if (st != TRI_OK) {
    r.status = st;
    return st;
  }
  *vi = find_version(c, op, k);
  *auto_inst = true;
  return TRI_OK;
}

inline void record(tri_cache *c, uint32_t op, const Version &v, int32_t vi, const Key &k,
                   int n, const tri_launch_rec *l, int st) {
  tri_selection &r = c->last;
  r.op = int32_t(op);
  r.status = st;
  r.version = vi;
  r.variant = v.plan.variant;
  r.n_launches = n;
  r.roles[0] = v.plan.roles[0];
  r.roles[1] = v.plan.roles[1];
  r.roles[2] = v.plan.roles[2];
  for (int i = 0; i < 3; ++i) r.launch[i] = i < n ? l[i] : tri_launch_rec{0, 0, 0};
  key_words(k, r.key);
}

inline tri_status finish(tri_cache *c, Version &v, bool auto_inst, int rc) {
  if (rc != 0) {
    if (!auto_inst) c->stats.errors++;
    return TRI_E_LAUNCH;
  }
  if (!auto_inst) {
    c->stats.hits++;
    v.hits++;
  }
  return TRI_OK;
}

inline int64_t vec_elems(uint32_t dtype) { return dtype == TRI_F32 ? 4 : 8; }

// Validation and key of one decode-chain call: kGo with *out set, TRI_OK
// for T == 0, or an error. Order: common, norm, RoPE, QK norm, SwiGLU.
int chain_check(const tri_chain_args *p, Key *out) {
  if (!p) return TRI_E_INVALID;
  const int32_t dtype = p->dtype;
  const int64_t T = p->T, H = p->H, I = p->I;
  int st = check_common(dtype, T);
  if (st != kGo) return st;
  const uint64_t es = es_of(uint32_t(dtype));
  {
    const void *ptrs[5] = {p->x, p->res, p->w, p->y, p->res_out};
    const int64_t strides[4] = {p->x_rs, p->res_rs, p->y_rs, p->ro_rs};
    st = check_norm(es, T, H, ptrs, 5, strides, 4, p->eps);
    if (st != kGo) return st;
  }
  const tri_rope_ext &x = p->rope_ext ? *p->rope_ext : kRopePlain;
  st = check_rope(es, T, p->q, p->q_ts, p->k, p->k_ts, p->pos, p->nq, p->nk, p->hd, p->base, x);
  if (st != kGo) return st;
  const bool qkn = p->q_norm_w != nullptr;
  if (qkn) {
    st = check_qkn(es, p->q_norm_w, p->k_norm_w, p->nk, p->qk_eps);
    if (st != kGo) return st;
  }
  st = check_sw(es, T, I, p->gate, p->g_rs, p->up, p->u_rs, p->out, p->o_rs);
  if (st != kGo) return st;

  const unsigned fl =
      res_flags(es, p->x, p->x_rs, p->res, p->res_rs, p->w, p->y, p->y_rs, p->res_out, p->ro_rs,
                H) |
      (rope_flags(es, p->q, p->q_ts, p->k, p->k_ts, p->nq, p->nk, p->hd,
                  qkn ? p->q_norm_w : nullptr, qkn ? p->k_norm_w : nullptr) << 2) |
      (sw_flags(es, p->gate, p->g_rs, p->up, p->u_rs, p->out, p->o_rs, I) << 4) |
      (qkn ? kChainQkNorm : 0u);
  *out = make_key(TRI_OP_CHAIN, uint32_t(dtype), T, fl, 0, uint64_t(H), uint64_t(I),
                  uint64_t(p->hd), uint64_t(p->nq), uint64_t(p->nk));
  rope_key_words(*out, p->hd, p->base, x);
  return kGo;
}

// Launch i of version v of cache c with its argument block: from a
// resident block when the launch has an argument-free form and the cache
// holds (or can hold) the block in a slot the launch may take (any slot up
// to kResidentMaxGrid workgroups, else the first kResidentAnyGridSlots);
// otherwise with kernel arguments. 0 or the launch's failure code.
int launch(tri_cache *c, const Version &v, int i, uint32_t dtype, uint32_t grid, uint32_t block,
           const void *args, uint32_t size, void *stream) {
  if (v.fn_res[i]) {
    const uint32_t limit = grid <= kResidentMaxGrid ? kResidentSlots : kResidentAnyGridSlots;
    const int32_t slot = resident_slot(c, resident_family(v.plan.kvariant[i]), dtype, args,
                                       size, grid, stream, limit);
    if (slot >= 0) {
      const int rc = be_launch_resident(v.fn_res[i], grid, block, uint32_t(slot), stream);
      if (rc == 0) c->resident_launches++;
      return rc;
    }
  }
  return be_launch(v.fn[i], grid, block, args, size, stream);
}

// The launches of one chain call on version v of cache c: one fused launch,
// or the three role kernels in order (stopping at the first failure), each
// through launch(). l receives the launch records, *n their count. Returns
// 0 or the failing launch's code.
int chain_launch(tri_cache *c, const Version &v, const tri_chain_args &p, void *stream,
                 tri_launch_rec *l, int *n) {
  const uint32_t dtype = uint32_t(p.dtype);
  const int64_t T = p.T, I = p.I;
  const tri_rope_ext &x = p.rope_ext ? *p.rope_ext : kRopePlain;
  const bool qkn = p.q_norm_w != nullptr;
  const RnArgs rn{p.x, p.res, p.w, p.y, p.res_out, p.x_rs, p.res_rs, p.y_rs, p.ro_rs,
                  T, int32_t(p.H), p.eps};
  const RopeArgs ro = rope_args(v, p.q, p.q_ts, p.k, p.k_ts, p.pos, T, p.nq, p.nk, p.hd, x,
                                qkn ? p.q_norm_w : nullptr, p.k_norm_w, p.qk_eps);
  const SwArgs sw{p.gate, p.up, p.out, p.g_rs, p.u_rs, p.o_rs, T, I,
                  (T * I) / vec_elems(dtype), T * I};
  const uint32_t g0 = role_grid(v.plan.roles[0], dtype, T, p.H);
  const uint32_t g1 =
      role_grid(v.plan.roles[1], dtype, T, I, v.plan.rope_slices, v.plan.rope_tokens);
  const uint32_t g2 = role_grid(v.plan.roles[2], dtype, T, I);

  if (v.plan.variant == CH_FUSED) {
    const ChainArgs a{rn, ro, sw, g0, g1};
    const uint32_t grid = g0 + g1 + g2;
    l[0] = {CH_FUSED, grid, kBlock};
    *n = 1;
    return launch(c, v, 0, dtype, grid, kBlock, &a, sizeof a, stream);
  }
  // Three launches: the residual norm, RoPE and SwiGLU role kernels (a
  // split norm role takes the version's scratch with its rows).
  const RnSplitArgs rs{rn, v.d_scratch};
  const bool split = v.plan.kvariant[0] == RN_SPLIT;
  const void *args[3] = {split ? static_cast<const void *>(&rs) : &rn, &ro, &sw};
  const uint32_t sizes[3] = {split ? uint32_t(sizeof rs) : uint32_t(sizeof rn), sizeof ro,
                             sizeof sw};
  const uint32_t grids[3] = {g0, g1, g2};
  *n = 3;
  int rc = 0;
  for (int i = 0; i < 3; ++i) {
    l[i] = {v.plan.kvariant[i], grids[i], role_block(v.plan.kvariant[i])};
    if (rc == 0) rc = launch(c, v, i, dtype, grids[i], l[i].block_x, args[i], sizes[i], stream);
  }
  return rc;
}

// Element-wise ops: W range, non-null element-aligned operands (the mask is
// bytes), strides >= W and within the extent limit over T rows.
inline int check_elt(uint64_t es, int64_t T, int64_t W, const void *a, int64_t a_rs,
                     const void *b, int64_t b_rs, bool b_is_mask, const void *o, int64_t o_rs) {
  if (W < 1) return TRI_E_INVALID;
  if (W >= kILimit) return TRI_E_UNSUPPORTED;
  if (!a || !b || !o) return TRI_E_INVALID;
  if (addr(a) % es || addr(o) % es || (!b_is_mask && addr(b) % es)) return TRI_E_INVALID;
  if (a_rs < W || b_rs < W || o_rs < W) return TRI_E_INVALID;
  if (!extent_ok(T, a_rs, W, es) || !extent_ok(T, b_rs, W, b_is_mask ? 1 : es) ||
      !extent_ok(T, o_rs, W, es))
    return TRI_E_INVALID;
  return kGo;
}

// One launch of a single-kernel op (SwiGLU, the short ops): lookup (miss /
// auto-install), launch with the argument block, record, count. `width` is
// what role_grid takes as the row width (SwiGLU's I, a short op's W).
tri_status single_launch(tri_cache *c, uint32_t op, const Key &k, int64_t T, int64_t width,
                         const void *args, uint32_t args_size, void *stream) {
  int32_t vi;
  bool auto_inst = false;
  const int st = lookup(c, op, k, T, &vi, &auto_inst);
  if (st != TRI_OK) return tri_status(st);
  Version &v = c->versions[vi];
  const tri_launch_rec l{v.plan.kvariant[0],
                         role_grid(v.plan.kvariant[0], key_dtype(k), T, width),
                         role_block(v.plan.kvariant[0])};
  const int rc = launch(c, v, 0, key_dtype(k), l.grid_x, l.block_x, args, args_size, stream);
  record(c, op, v, vi, k, 1, &l, rc ? TRI_E_LAUNCH : TRI_OK);
  return finish(c, v, auto_inst, rc);
}

// One launch of a norm version: RnArgs, or with a split plan the rows and
// the version's scratch.
tri_status norm_launch(tri_cache *c, uint32_t op, const Key &k, const RnArgs &a, void *stream) {
  int32_t vi;
  bool auto_inst = false;
  const int st = lookup(c, op, k, a.T, &vi, &auto_inst);
  if (st != TRI_OK) return tri_status(st);
  Version &v = c->versions[vi];
  const int32_t kv = v.plan.kvariant[0];
  const tri_launch_rec l{kv, norm_grid(kv, key_dtype(k), a.T, a.H, op == TRI_OP_RES_RMSNORM),
                         role_block(kv)};
  int rc;
  if (kv == RN_SPLIT) {
    const RnSplitArgs sa{a, v.d_scratch};
    rc = launch(c, v, 0, key_dtype(k), l.grid_x, l.block_x, &sa, sizeof sa, stream);
  } else {
    rc = launch(c, v, 0, key_dtype(k), l.grid_x, l.block_x, &a, sizeof a, stream);
  }
  record(c, op, v, vi, k, 1, &l, rc ? TRI_E_LAUNCH : TRI_OK);
  return finish(c, v, auto_inst, rc);
}

// silu (b unused: pass a), add, masked_fill (b = mask).
tri_status elt_entry(tri_cache *c, uint32_t op, int32_t dtype, const void *a, int64_t a_rs,
                     const void *b, int64_t b_rs, void *out, int64_t o_rs, int64_t T, int64_t W,
                     float value, void *stream) {
  if (!c) return TRI_E_INVALID;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(uint32_t(dtype));
  const bool mask = op == TRI_OP_MASKED_FILL;
  st = check_elt(es, T, W, a, a_rs, b, b_rs, mask, out, o_rs);
  if (st != kGo) return finish_early(c, op, st);
  // alignment: data 16 B; the mask 16 / es bytes (one byte per element of a vector)
  const uint64_t v = 16 / es;
  uint64_t o16 = addr(a) | addr(out) | uint64_t(a_rs) * es | uint64_t(o_rs) * es;
  bool aligned;
  if (mask) {
    aligned = (o16 & 15u) == 0 && addr(b) % v == 0 && uint64_t(b_rs) % v == 0;
  } else {
    o16 |= addr(b) | uint64_t(b_rs) * es;
    aligned = (o16 & 15u) == 0;
  }
  const bool contig = a_rs == W && b_rs == W && o_rs == W;
  const unsigned fl = (aligned ? kAlign : 0u) | (contig ? kContig : 0u);
  const Key k = make_key(op, uint32_t(dtype), T, fl, 0, uint64_t(W), 0, 0, 0, 0);
  const EltArgs args{a, b, out, a_rs, b_rs, o_rs, T, W, (T * W) / vec_elems(uint32_t(dtype)),
                     T * W, value, 0};
  return single_launch(c, op, k, T, W, &args, sizeof args, stream);
}

// Several chains per call, split in two passes so that a graph capture can
// record the second one alone.
struct LayerPlan {
  int32_t vis[TRI_MAX_LAYERS];   // version per layer, -1 for an empty layer
  int32_t last;                  // last non-empty layer, -1 if none
  bool missed;
};

// Pass 1, in layer order: validate, pack the key, look the version up;
// then, under auto-install, install the missing versions. Nothing is
// installed or launched before every layer has passed. Returns kGo, or the
// call's final status (error, MISS, install error, or OK for an empty call)
// with the statistics and record already written.
int layers_prepare(tri_cache *c, const tri_chain_args *layers, uint32_t n_layers, LayerPlan *lp) {
  const uint32_t op = TRI_OP_CHAIN_LAYERS;
  c->stats.calls++;
  if (n_layers > uint32_t(TRI_MAX_LAYERS) || (n_layers > 0 && !layers))
    return finish_early(c, op, TRI_E_INVALID);
  int32_t first_miss = -1;
  lp->last = -1;
  for (uint32_t i = 0; i < n_layers; ++i) {
    Key k;
    const int st = chain_check(&layers[i], &k);
    if (st == TRI_OK) {            // T == 0: this layer is a no-op
      lp->vis[i] = -1;
      continue;
    }
    if (st != kGo) return finish_early(c, op, st);
    lp->vis[i] = find_version(c, TRI_OP_CHAIN, k);
    if (lp->vis[i] < 0 && first_miss < 0) first_miss = int32_t(i);
    lp->last = int32_t(i);
  }
  if (lp->last < 0) return finish_early(c, op, TRI_OK);
  // Misses: one per entry call; the first missed layer's key is recorded.
  // With auto-install every missing version is installed, in layer order.
  lp->missed = first_miss >= 0;
  if (lp->missed) {
    c->stats.misses++;
    Key k;
    chain_check(&layers[first_miss], &k);
    c->has_miss = true;
    c->miss_key = k;
    c->miss_T = layers[first_miss].T;
    tri_selection &r = c->last;
    memset(&r, 0, sizeof r);
    r.op = int32_t(op);
    r.version = -1;
    key_words(k, r.key);
    if (!(c->flags & TRI_CACHE_AUTO_INSTALL)) {
      r.status = TRI_MISS;
      return TRI_MISS;
    }
    for (uint32_t i = uint32_t(first_miss); i <= uint32_t(lp->last); ++i) {
      if (lp->vis[i] >= 0 || layers[i].T == 0) continue;
      chain_check(&layers[i], &k);
      // an earlier layer's generic install may already cover this key
      const tri_status ist = install_key(c, k, -1, (c->flags & TRI_CACHE_GENERIC) != 0);
      if (ist != TRI_OK) {
        r.status = ist;
        return ist;
      }
      lp->vis[i] = find_version(c, TRI_OP_CHAIN, k);
    }
  }
  return kGo;
}

// Pass 2: the launches, in layer order on `stream`; record and count.
tri_status layers_launch(tri_cache *c, const tri_chain_args *layers, uint32_t n_layers,
                         const LayerPlan &lp, void *stream, uint32_t *n_launched) {
  const uint32_t op = TRI_OP_CHAIN_LAYERS;
  int total = 0;
  for (uint32_t i = 0; i < n_layers; ++i) {
    if (lp.vis[i] < 0) continue;
    Version &v = c->versions[lp.vis[i]];
    tri_launch_rec l[3];
    int n = 0;
    const int rc = chain_launch(c, v, layers[i], stream, l, &n);
    total += n;
    if (rc != 0 || int32_t(i) == lp.last) {
      Key k;
      chain_check(&layers[i], &k);
      record(c, op, v, lp.vis[i], k, n, l, rc ? TRI_E_LAUNCH : TRI_OK);
      c->last.n_launches = total;
    }
    if (rc != 0) {
      if (!lp.missed) c->stats.errors++;
      return TRI_E_LAUNCH;
    }
  }
  if (n_launched) *n_launched = uint32_t(total);
  if (!lp.missed) {
    c->stats.hits++;
    for (uint32_t i = 0; i < n_layers; ++i)
      if (lp.vis[i] >= 0) c->versions[lp.vis[i]].hits++;
  }
  return TRI_OK;
}

// RoPE (op 3) or QK-RMSNorm + RoPE (op 6; the head-norm weights are then
// required) with an optional variant.
tri_status rope_entry(tri_cache *c, uint32_t op, int32_t dtype, void *q, int64_t q_ts, void *kp,
                      int64_t k_ts, const void *pos, int64_t T, int32_t nq, int32_t nk,
                      int32_t hd, float base, const tri_rope_ext *ext, const void *q_w,
                      const void *k_w, float eps, void *stream) {
  if (!c) return TRI_E_INVALID;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(uint32_t(dtype));
  const tri_rope_ext &x = ext ? *ext : kRopePlain;
  st = check_rope(es, T, q, q_ts, kp, k_ts, pos, nq, nk, hd, base, x);
  if (st != kGo) return finish_early(c, op, st);
  const bool qkn = op == TRI_OP_QK_NORM_ROPE;
  if (qkn) {
    st = check_qkn(es, q_w, k_w, nk, eps);
    if (st != kGo) return finish_early(c, op, st);
  }

  Key k = make_key(op, uint32_t(dtype), T,
                   rope_flags(es, q, q_ts, kp, k_ts, nq, nk, hd, qkn ? q_w : nullptr, k_w), 0, 0,
                   0, uint64_t(hd), uint64_t(nq), uint64_t(nk));
  rope_key_words(k, hd, base, x);
  int32_t vi;
  bool auto_inst = false;
  st = lookup(c, op, k, T, &vi, &auto_inst);
  if (st != TRI_OK) return tri_status(st);
  Version &v = c->versions[vi];

  const RopeArgs a =
      rope_args(v, q, q_ts, kp, k_ts, pos, T, nq, nk, hd, x, qkn ? q_w : nullptr, k_w, eps);
  const tri_launch_rec l{v.plan.kvariant[0],
                         role_grid(v.plan.kvariant[0], uint32_t(dtype), T, 0, v.plan.rope_slices,
                                   v.plan.rope_tokens),
                         kBlock};
  const int rc = launch(c, v, 0, uint32_t(dtype), l.grid_x, kBlock, &a, sizeof a, stream);
  record(c, op, v, vi, k, 1, &l, rc ? TRI_E_LAUNCH : TRI_OK);
  return finish(c, v, auto_inst, rc);
}

}  // namespace

extern "C" {

tri_status tri_rmsnorm(tri_cache *c, tri_dtype dtype, const void *x, int64_t x_rs,
                       const void *w, void *y, int64_t y_rs, int64_t T, int64_t H, float eps,
                       void *stream) {
  if (!c) return TRI_E_INVALID;
  const uint32_t op = TRI_OP_RMSNORM;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(dtype);
  const void *ptrs[3] = {x, w, y};
  const int64_t strides[2] = {x_rs, y_rs};
  st = check_norm(es, T, H, ptrs, 3, strides, 2, eps);
  if (st != kGo) return finish_early(c, op, st);

  const Key k = make_key(op, dtype, T, rn_flags(es, x, x_rs, w, y, y_rs, H), 0, uint64_t(H), 0,
                         0, 0, 0);
  const RnArgs a{x, nullptr, w, y, nullptr, x_rs, 0, y_rs, 0, T, int32_t(H), eps};
  return norm_launch(c, op, k, a, stream);
}

tri_status tri_residual_rmsnorm(tri_cache *c, tri_dtype dtype, const void *x, int64_t x_rs,
                                const void *res, int64_t res_rs, const void *w, void *y,
                                int64_t y_rs, void *res_out, int64_t ro_rs, int64_t T, int64_t H,
                                float eps, void *stream) {
  if (!c) return TRI_E_INVALID;
  const uint32_t op = TRI_OP_RES_RMSNORM;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(dtype);
  const void *ptrs[5] = {x, res, w, y, res_out};
  const int64_t strides[4] = {x_rs, res_rs, y_rs, ro_rs};
  st = check_norm(es, T, H, ptrs, 5, strides, 4, eps);
  if (st != kGo) return finish_early(c, op, st);

  const Key k = make_key(op, dtype, T,
                         res_flags(es, x, x_rs, res, res_rs, w, y, y_rs, res_out, ro_rs, H), 0,
                         uint64_t(H), 0, 0, 0, 0);
  const RnArgs a{x, res, w, y, res_out, x_rs, res_rs, y_rs, ro_rs, T, int32_t(H), eps};
  return norm_launch(c, op, k, a, stream);
}

tri_status tri_residual_rmsnorm_noalloc(tri_cache *c, tri_dtype dtype, const void *x,
                                        int64_t x_rs, const void *res, int64_t res_rs,
                                        const void *w, void *y, int64_t y_rs, void *res_out,
                                        int64_t ro_rs, int64_t T, int64_t H, float eps,
                                        void *stream) {
  if (!c) return TRI_E_INVALID;
  const uint32_t op = TRI_OP_RES_RMSNORM;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(dtype);
  const void *ptrs[5] = {x, res, w, y, res_out};
  const int64_t strides[4] = {x_rs, res_rs, y_rs, ro_rs};
  st = check_norm(es, T, H, ptrs, 5, strides, 4, eps);
  if (st != kGo) return finish_early(c, op, st);

  const Key k = make_key(op, dtype, T,
                         res_flags(es, x, x_rs, res, res_rs, w, y, y_rs, res_out, ro_rs, H), 0,
                         uint64_t(H), 0, 0, 0, 0);
  // Lookup only: an install may allocate, so a miss is returned as is.
  const int32_t vi = find_version(c, op, k);
  if (vi < 0) {
    note_miss(c, op, k, T);
    return TRI_MISS;
  }
  Version &v = c->versions[vi];
  const int32_t kv = v.plan.kvariant[0];
  const RnArgs a{x, res, w, y, res_out, x_rs, res_rs, y_rs, ro_rs, T, int32_t(H), eps};
  const tri_launch_rec l{kv, norm_grid(kv, uint32_t(dtype), T, H, true), role_block(kv)};
  // Always with kernel arguments: a resident block's first use copies it
  // to the device, which this entry point does not do.
  int rc;
  if (kv == RN_SPLIT) {
    // the GPU's fixed scratch in place of the version's own
    if (!c->noalloc_scratch) return finish_early(c, op, TRI_E_RUNTIME);
    if (split_words(T, split_slices(uint32_t(dtype), H)) > kNoAllocScratchWords)
      return finish_early(c, op, TRI_E_UNSUPPORTED);
    const RnSplitArgs sa{a, static_cast<uint64_t *>(c->noalloc_scratch)};
    rc = be_launch(v.fn[0], l.grid_x, l.block_x, &sa, sizeof sa, stream);
  } else {
    rc = be_launch(v.fn[0], l.grid_x, l.block_x, &a, sizeof a, stream);
  }
  record(c, op, v, vi, k, 1, &l, rc ? TRI_E_LAUNCH : TRI_OK);
  return finish(c, v, false, rc);
}

tri_status tri_rope_qk_ext(tri_cache *c, tri_dtype dtype, void *q, int64_t q_ts, void *kp,
                           int64_t k_ts, const void *pos, int64_t T, int32_t nq, int32_t nk,
                           int32_t hd, float base, const tri_rope_ext *ext, const void *q_w,
                           const void *k_w, float eps, void *stream) {
  return rope_entry(c, q_w ? TRI_OP_QK_NORM_ROPE : TRI_OP_ROPE_QK, dtype, q, q_ts, kp, k_ts, pos,
                    T, nq, nk, hd, base, ext, q_w, k_w, eps, stream);
}

tri_status tri_rope_qk(tri_cache *c, tri_dtype dtype, void *q, int64_t q_ts, void *kp,
                       int64_t k_ts, const int32_t *pos, int64_t T, int32_t nq, int32_t nk,
                       int32_t hd, float base, void *stream) {
  return rope_entry(c, TRI_OP_ROPE_QK, dtype, q, q_ts, kp, k_ts, pos, T, nq, nk, hd, base,
                    nullptr, nullptr, nullptr, 0.0f, stream);
}

tri_status tri_qk_norm_rope(tri_cache *c, tri_dtype dtype, void *q, int64_t q_ts, void *kp,
                            int64_t k_ts, const int32_t *pos, int64_t T, int32_t nq, int32_t nk,
                            int32_t hd, float base, const void *q_w, const void *k_w, float eps,
                            void *stream) {
  return rope_entry(c, TRI_OP_QK_NORM_ROPE, dtype, q, q_ts, kp, k_ts, pos, T, nq, nk, hd, base,
                    nullptr, q_w, k_w, eps, stream);
}

tri_status tri_swiglu(tri_cache *c, tri_dtype dtype, const void *gate, int64_t g_rs,
                      const void *up, int64_t u_rs, void *out, int64_t o_rs, int64_t T, int64_t I,
                      void *stream) {
  if (!c) return TRI_E_INVALID;
  const uint32_t op = TRI_OP_SWIGLU;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(dtype);
  st = check_sw(es, T, I, gate, g_rs, up, u_rs, out, o_rs);
  if (st != kGo) return finish_early(c, op, st);

  const Key k = make_key(op, dtype, T, sw_flags(es, gate, g_rs, up, u_rs, out, o_rs, I), 0, 0,
                         uint64_t(I), 0, 0, 0);
  const SwArgs a{gate, up, out, g_rs, u_rs, o_rs, T, I, (T * I) / vec_elems(dtype), T * I};
  return single_launch(c, op, k, T, I, &a, sizeof a, stream);
}

tri_status tri_silu(tri_cache *c, tri_dtype dtype, const void *x, int64_t x_rs, void *out,
                    int64_t o_rs, int64_t T, int64_t W, void *stream) {
  return elt_entry(c, TRI_OP_SILU, dtype, x, x_rs, x, x_rs, out, o_rs, T, W, 0.0f, stream);
}

tri_status tri_add(tri_cache *c, tri_dtype dtype, const void *a, int64_t a_rs, const void *b,
                   int64_t b_rs, void *out, int64_t o_rs, int64_t T, int64_t W, void *stream) {
  return elt_entry(c, TRI_OP_ADD, dtype, a, a_rs, b, b_rs, out, o_rs, T, W, 0.0f, stream);
}

tri_status tri_masked_fill(tri_cache *c, tri_dtype dtype, const void *x, int64_t x_rs,
                           const uint8_t *mask, int64_t m_rs, float value, void *out,
                           int64_t o_rs, int64_t T, int64_t W, void *stream) {
  return elt_entry(c, TRI_OP_MASKED_FILL, dtype, x, x_rs, mask, m_rs, out, o_rs, T, W, value,
                   stream);
}

tri_status tri_embedding(tri_cache *c, tri_dtype dtype, const void *table, int64_t t_rs,
                         int64_t n_rows, const void *ids, int32_t ids_int64, void *out,
                         int64_t o_rs, int64_t T, int64_t H, void *stream) {
  if (!c) return TRI_E_INVALID;
  const uint32_t op = TRI_OP_EMBEDDING;
  c->stats.calls++;
  int st = check_common(dtype, T);
  if (st != kGo) return finish_early(c, op, st);
  const uint64_t es = es_of(uint32_t(dtype));
  if (H < 1 || n_rows < 1 || (ids_int64 | 1) != 1) return finish_early(c, op, TRI_E_INVALID);
  if (H >= kILimit) return finish_early(c, op, TRI_E_UNSUPPORTED);
  if (!table || !ids || !out) return finish_early(c, op, TRI_E_INVALID);
  if (addr(table) % es || addr(out) % es || addr(ids) % (ids_int64 ? 8 : 4))
    return finish_early(c, op, TRI_E_INVALID);
  if (t_rs < H || o_rs < H || !extent_ok(n_rows, t_rs, H, es) || !extent_ok(T, o_rs, H, es))
    return finish_early(c, op, TRI_E_INVALID);
  const bool aligned =
      ((addr(table) | addr(out) | uint64_t(t_rs) * es | uint64_t(o_rs) * es) & 15u) == 0;
  Key k = make_key(op, uint32_t(dtype), T, aligned ? kAlign : 0u, 0, uint64_t(H), 0, 0, 0, 0);
  k.k3 = uint64_t(ids_int64) << 16;
  const EmbArgs args{table, ids, out, t_rs, o_rs, T, H, n_rows, ids_int64, 0};
  return single_launch(c, op, k, T, H, &args, sizeof args, stream);
}

tri_status tri_decode_chain(tri_cache *c, const tri_chain_args *p, void *stream) {
  if (!c) return TRI_E_INVALID;
  const uint32_t op = TRI_OP_CHAIN;
  c->stats.calls++;
  Key k;
  int st = chain_check(p, &k);
  if (st != kGo) return finish_early(c, op, st);
  int32_t vi;
  bool auto_inst = false;
  st = lookup(c, op, k, p->T, &vi, &auto_inst);
  if (st != TRI_OK) return tri_status(st);
  Version &v = c->versions[vi];
  tri_launch_rec l[3];
  int n = 0;
  const int rc = chain_launch(c, v, *p, stream, l, &n);
  record(c, op, v, vi, k, n, l, rc ? TRI_E_LAUNCH : TRI_OK);
  return finish(c, v, auto_inst, rc);
}

tri_status tri_decode_chain_layers(tri_cache *c, const tri_chain_args *layers, uint32_t n_layers,
                                   void *stream) {
  if (!c) return TRI_E_INVALID;
  LayerPlan lp;
  const int st = layers_prepare(c, layers, n_layers, &lp);
  if (st != kGo) return tri_status(st);
  return layers_launch(c, layers, n_layers, lp, stream, nullptr);
}

tri_status tri_graph_build_layers(tri_cache *c, const tri_chain_args *layers, uint32_t n_layers,
                                  tri_graph **out) {
  if (!c || !out) return TRI_E_INVALID;
  *out = nullptr;
  // Validation, lookup and installs happen outside the capture (installs
  // allocate and may compile); only the launches are recorded.
  LayerPlan lp;
  int st = layers_prepare(c, layers, n_layers, &lp);
  if (st != kGo) return tri_status(st);
  tri_graph *g = static_cast<tri_graph *>(calloc(1, sizeof(tri_graph)));
  if (!g) return TRI_E_NOMEM;
  void *cap = nullptr;
  st = be_capture_begin(&cap);
  if (st != 0) {
    free(g);
    return tri_status(st);
  }
  uint32_t launched = 0;
  const tri_status ls = layers_launch(c, layers, n_layers, lp, cap, &launched);
  void *exec = nullptr;
  const int es = be_capture_end(cap, &exec);
  if (ls != TRI_OK || es != 0) {
    if (exec) be_graph_destroy(exec);
    free(g);
    return ls != TRI_OK ? ls : tri_status(es);
  }
  g->exec = exec;
  g->n_launches = launched;
  *out = g;
  return TRI_OK;
}

tri_status tri_graph_launch(tri_graph *g, void *stream) {
  if (!g) return TRI_E_INVALID;
  return be_graph_launch(g->exec, stream) == 0 ? TRI_OK : TRI_E_RUNTIME;
}

uint32_t tri_graph_launch_count(const tri_graph *g) { return g ? g->n_launches : 0; }

void tri_graph_destroy(tri_graph *g) {
  if (!g) return;
  if (g->exec) be_graph_destroy(g->exec);
  free(g);
}

}  // extern "C"

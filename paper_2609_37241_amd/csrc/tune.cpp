// Install-time tuning: the benchmark-and-keep scheme of Triton's autotuner
// that the paper describes (Sec. 2), applied to a key's candidate plans.
//
// Each candidate serves a tuning call of the key's shapes through the same
// entry point as a user call, on zero-filled device memory of its own and a
// private stream. The call's arguments are built from the key alone, and a
// private one-version cache holding the candidate must hit on them, which
// checks that the tuning call is a call of this key. Candidates are timed
// in turn (two warm-up rounds, five timed rounds) with HIP events around
// each call; the fastest median is kept when it beats candidate 0's median
// by more than the margin.
#include <stdlib.h>
#include <string.h>

#include <algorithm>

#include "internal.h"

namespace tri {

namespace {

// The operands of a tuning call. Norm, RoPE and SwiGLU fields live in a
// chain argument block (the single-op calls read the fields they need);
// the element-wise ops use their own fields.
struct TuneCall {
  uint32_t op;
  tri_chain_args a;
  tri_rope_ext ext;
  const void *ea, *eb;
  void *eo;
  int64_t ea_rs, eb_rs, eo_rs, W;
};

float f32_of(uint32_t bits) {
  float f;
  memcpy(&f, &bits, sizeof f);
  return f;
}

// Carves 256-byte aligned buffers out of one block starting at `base`
// (a stand-in address while sizing); `shift` displaces a buffer of an
// unaligned role by one element. Each buffer keeps 16 bytes of slack.
struct Carver {
  uintptr_t base;
  uint64_t off;
  void *take(uint64_t bytes, uint64_t shift) {
    off = (off + 255) & ~uint64_t(255);
    void *p = reinterpret_cast<void *>(base + off + shift);
    off += bytes + 16;
    return p;
  }
};

// Row stride of an operand of width `w` under a role's guard flags: the
// width when contiguous, else the next multiple of a vector above it when
// aligned, else one element more.
int64_t tune_stride(int64_t w, unsigned fl, int64_t v) {
  if (fl & kContig) return w;
  return (fl & kAlign) ? (w + 1 + v - 1) / v * v : w + 1;
}

// Fills `tc` for key k with buffers carved from `base`; returns the bytes
// of the block and, in *operands, the operand bytes (the size limit's
// measure).
uint64_t build_call(const Key &k, uintptr_t base, TuneCall *tc, uint64_t *operands) {
  memset(tc, 0, sizeof *tc);
  const uint32_t op = key_op(k), dt = key_dtype(k), fl = key_flags(k);
  const uint64_t es = dt == TRI_F32 ? 4 : 2;
  const int64_t v = int64_t(16 / es);
  const int64_t T = int64_t(1) << key_bucket(k);
  const int64_t H = key_H(k), I = key_I(k);
  tri_chain_args &a = tc->a;
  Carver cv{base, 0};
  uint64_t ops = 0;
  auto take = [&](uint64_t bytes, uint64_t shift) {
    ops += bytes;
    return cv.take(bytes, shift);
  };
  tc->op = op;
  a.dtype = int32_t(dt);
  a.T = T;
  a.eps = 1e-6f;

  auto norm = [&](unsigned f2, bool res) {
    const int64_t s = tune_stride(H, f2, v);
    const uint64_t sh = (f2 & kAlign) ? 0 : es, rows = uint64_t(T) * uint64_t(s) * es;
    a.H = H;
    a.x = take(rows, sh);
    a.x_rs = s;
    a.w = take(uint64_t(H) * es, sh);
    a.y = take(rows, sh);
    a.y_rs = s;
    if (res) {
      a.res = take(rows, sh);
      a.res_rs = s;
      a.res_out = take(rows, sh);
      a.ro_rs = s;
    }
  };
  auto rope = [&](unsigned f2, bool qkn) {
    const int32_t hd = int32_t(key_hd(k)), nq = int32_t(key_nq(k)), nk = int32_t(key_nk(k));
    const uint32_t bits = key_rope_bits(k);
    const uint64_t sh = (f2 & kAlign) ? 0 : es;
    a.hd = hd;
    a.nq = nq;
    a.nk = nk;
    a.q_ts = tune_stride(int64_t(nq) * hd, f2, v);
    a.q = take(uint64_t(T) * uint64_t(a.q_ts) * es, sh);
    if (nk > 0) {
      a.k_ts = tune_stride(int64_t(nk) * hd, f2, v);
      a.k = take(uint64_t(T) * uint64_t(a.k_ts) * es, sh);
    }
    a.pos = take(uint64_t(T) * ((bits & kRopePos64) ? 8 : 4), 0);
    if (qkn) {
      a.q_norm_w = take(uint64_t(hd) * es, sh);
      if (nk > 0) a.k_norm_w = take(uint64_t(hd) * es, sh);
      a.qk_eps = 1e-6f;
    }
    tri_rope_ext &x = tc->ext;
    x.rotary_dim = int32_t(key_rd(k));
    x.interleaved = (bits & kRopeInterleaved) ? 1 : 0;
    x.pos_int64 = (bits & kRopePos64) ? 1 : 0;
    if (bits & kRopeCache) {
      x.cos_sin = static_cast<const float *>(take(uint64_t(key_rd(k)) * 4, 0));
      x.cos_sin_len = 1;
    } else {
      a.base = f32_of(key_base_bits(k));
      x.scaling = int32_t(key_scaling(k));
      if (x.scaling == TRI_ROPE_SCALING_LLAMA3) {
        x.factor = f32_of(uint32_t(k.k4));
        x.low_freq_factor = f32_of(uint32_t(k.k4 >> 32));
        x.high_freq_factor = f32_of(uint32_t(k.k5));
        x.original_max_pos = int32_t(key_orig_max(k));
      }
    }
    a.rope_ext = &tc->ext;
  };
  auto swiglu = [&](unsigned f2) {
    const int64_t s = tune_stride(I, f2, v);
    const uint64_t sh = (f2 & kAlign) ? 0 : es, rows = uint64_t(T) * uint64_t(s) * es;
    a.I = I;
    a.gate = take(rows, sh);
    a.g_rs = s;
    a.up = take(rows, sh);
    a.u_rs = s;
    a.out = take(rows, sh);
    a.o_rs = s;
  };

  switch (op) {
    case TRI_OP_RMSNORM: norm(fl, false); break;
    case TRI_OP_RES_RMSNORM: norm(fl, true); break;
    case TRI_OP_ROPE_QK: rope(fl, false); break;
    case TRI_OP_QK_NORM_ROPE: rope(fl, true); break;
    case TRI_OP_SWIGLU: swiglu(fl); break;
    case TRI_OP_SILU:
    case TRI_OP_ADD:
    case TRI_OP_MASKED_FILL: {
      const int64_t s = tune_stride(H, fl, v);
      const uint64_t sh = (fl & kAlign) ? 0 : es, rows = uint64_t(T) * uint64_t(s) * es;
      tc->W = H;
      tc->ea = take(rows, sh);
      tc->ea_rs = tc->eb_rs = tc->eo_rs = s;
      tc->eo = take(rows, sh);
      if (op == TRI_OP_ADD)
        tc->eb = take(rows, sh);
      else if (op == TRI_OP_MASKED_FILL)
        tc->eb = take(uint64_t(T) * uint64_t(s), 0);
      else
        tc->eb = tc->ea;
      break;
    }
    case TRI_OP_CHAIN:
      norm(fl & 3u, true);
      rope((fl >> 2) & 3u, (fl & kChainQkNorm) != 0);
      swiglu((fl >> 4) & 3u);
      break;
    default:
      break;
  }
  *operands = ops;
  return cv.off;
}

// One tuning call through the entry point of the key's op.
tri_status issue(tri_cache *c, const TuneCall &tc, void *stream) {
  const tri_chain_args &a = tc.a;
  const tri_dtype dt = tri_dtype(a.dtype);
  switch (tc.op) {
    case TRI_OP_RMSNORM:
      return tri_rmsnorm(c, dt, a.x, a.x_rs, a.w, a.y, a.y_rs, a.T, a.H, a.eps, stream);
    case TRI_OP_RES_RMSNORM:
      return tri_residual_rmsnorm(c, dt, a.x, a.x_rs, a.res, a.res_rs, a.w, a.y, a.y_rs,
                                  a.res_out, a.ro_rs, a.T, a.H, a.eps, stream);
    case TRI_OP_ROPE_QK:
    case TRI_OP_QK_NORM_ROPE:
      return tri_rope_qk_ext(c, dt, a.q, a.q_ts, a.k, a.k_ts, a.pos, a.T, a.nq, a.nk, a.hd,
                             a.base, a.rope_ext, a.q_norm_w, a.k_norm_w, a.qk_eps, stream);
    case TRI_OP_SWIGLU:
      return tri_swiglu(c, dt, a.gate, a.g_rs, a.up, a.u_rs, a.out, a.o_rs, a.T, a.I, stream);
    case TRI_OP_SILU:
      return tri_silu(c, dt, tc.ea, tc.ea_rs, tc.eo, tc.eo_rs, a.T, tc.W, stream);
    case TRI_OP_ADD:
      return tri_add(c, dt, tc.ea, tc.ea_rs, tc.eb, tc.eb_rs, tc.eo, tc.eo_rs, a.T, tc.W, stream);
    case TRI_OP_MASKED_FILL:
      return tri_masked_fill(c, dt, tc.ea, tc.ea_rs, static_cast<const uint8_t *>(tc.eb),
                             tc.eb_rs, 0.0f, tc.eo, tc.eo_rs, a.T, tc.W, stream);
    case TRI_OP_CHAIN:
      return tri_decode_chain(c, &a, stream);
    default:
      return TRI_E_INVALID;
  }
}

// Times candidate j's calls through private one-version caches (one per
// candidate, so each call hits its own version); returns false on any
// failure (resolve, timer, memory, a call that does not hit, a timing).
bool time_candidates(tri_cache *c, const Key &k, const Plan *cands, int n, const Version &v,
                     TuneCall &tc, uint64_t bytes, Version *vs, tri_cache *pc, float *med) {
  for (int j = 0; j < n; ++j) {
    vs[j] = v;
    vs[j].plan = cands[j];
    for (int i = 0; i < 3; ++i) vs[j].fn[i] = vs[j].module[i] = nullptr;
    for (int i = 0; i < 3; ++i) vs[j].fn_res[i] = nullptr;   // tuning launches carry arguments
    for (int i = 0; i < cands[j].n_launches; ++i)
      if (be_resolve(cands[j].kvariant[i], key_dtype(k), cands[j].ksub[i], &vs[j].fn[i]) != 0)
        return false;
    memset(&pc[j], 0, sizeof pc[j]);
    pc[j].capacity = 1;
    pc[j].n_versions = 1;
    pc[j].versions = &vs[j];
    pc[j].device = c->device;
    for (int i = 0; i < kOps; ++i) pc[j].last_hit[i] = -1;
    pc[j].last.version = -1;
  }

  const uint32_t n_ev = uint32_t(2 * n * kTuneRounds);
  void *timer = nullptr, *stream = nullptr, *mem = nullptr;
  if (be_timer_create(n_ev, &timer, &stream) != 0) return false;
  uint64_t operands = 0;
  bool ok = be_scratch(bytes, stream, &mem) == 0;
  if (ok) build_call(k, reinterpret_cast<uintptr_t>(mem), &tc, &operands);
  for (int r = 0; ok && r < kTuneWarmup + kTuneRounds; ++r) {
    for (int j = 0; ok && j < n; ++j) {
      const bool timed = r >= kTuneWarmup;
      const uint32_t e = uint32_t(2 * ((r - kTuneWarmup) * n + j));
      if (timed) ok = be_timer_record(timer, e) == 0;
      // a miss here means the tuning call is not a call of this key
      ok = ok && issue(&pc[j], tc, stream) == TRI_OK;
      if (timed) ok = ok && be_timer_record(timer, e + 1) == 0;
    }
  }
  for (int j = 0; ok && j < n; ++j) {
    float t[kTuneRounds];
    for (int r = 0; ok && r < kTuneRounds; ++r) {
      const uint32_t e = uint32_t(2 * (r * n + j));
      ok = be_timer_elapsed(timer, e, e + 1, &t[r]) == 0;
    }
    std::sort(t, t + kTuneRounds);
    med[j] = t[kTuneRounds / 2];
  }
  be_timer_destroy(timer);   // waits for the stream's work first
  if (mem) be_scratch_free(mem);
  return ok;
}

}  // namespace

void tune_key(tri_cache *c, const Key &k, const Plan *cands, int n, const Version &v,
              int32_t *choice, int32_t *how) {
  *choice = 0;
  *how = TRI_TUNE_SKIPPED;
  TuneCall tc;
  uint64_t operands = 0;
  const uint64_t bytes = build_call(k, 256, &tc, &operands);
  if (n < 2 || n > kMaxCandidates || operands > kTuneScratchMax) return;
  // The private caches are large; they live on the heap, not the stack of
  // whatever thread installs.
  struct Private {
    Version vs[kMaxCandidates];
    tri_cache pc[kMaxCandidates];
    float med[kMaxCandidates];
  };
  Private *p = static_cast<Private *>(calloc(1, sizeof(Private)));
  if (!p) return;
  if (time_candidates(c, k, cands, n, v, tc, bytes, p->vs, p->pc, p->med)) {
    int best = 0;
    for (int j = 1; j < n; ++j)
      if (p->med[j] < p->med[best]) best = j;
    *choice = p->med[best] < kTuneMargin * p->med[0] ? best : 0;
    *how = TRI_TUNE_MEASURED;
  }
  free(p);
}

}  // namespace tri

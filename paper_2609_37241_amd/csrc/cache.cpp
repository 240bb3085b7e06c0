// The specialization cache: ordered versions, lookup, install on miss,
// counters and introspection.
//
// Versions are kept in creation order and looked up with the first-match
// rule of the paper's ordered dispatch (Algorithm 1, Sec. 3.2): the first
// version whose guard holds. Exact guards are equality on the packed key;
// generic guards accept ranges of token buckets (and of norm row lengths),
// so versions may overlap. Every guard is a function of the key alone and
// versions are only ever appended, so the first match of a key never
// changes once found: the op's last lookup key and a direct-mapped memo of
// keys return exactly the version the scan would, without scanning.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <chrono>
#include <initializer_list>

#include "internal.h"

namespace tri {

int32_t scan_versions(const tri_cache *c, const Key &k) {
  const uint32_t n = c->n_versions;
  for (uint32_t i = 0; i < n; ++i)
    if (guard_holds(c->versions[i].key, c->versions[i].guard, k)) return int32_t(i);
  return -1;
}

namespace {
inline uint32_t memo_slot(const Key &k) {
  uint64_t h = k.k0 * 0x9E3779B97F4A7C15ull;
  for (uint64_t w : {k.k1, k.k2, k.k3, k.k4, k.k5})
    h = (h ^ (w + 0x632BE59BD9B4E019ull + (h << 6) + (h >> 2))) * 0xBF58476D1CE4E5B9ull;
  return uint32_t(h ^ (h >> 29)) & (kMemoSlots - 1);
}
}  // namespace

int32_t find_version(tri_cache *c, uint32_t op, const Key &k) {
  const int32_t h = c->last_hit[op];
  if (h >= 0 && c->last_key[op] == k) return h;
  MemoSlot *m = c->memo ? &c->memo[memo_slot(k)] : nullptr;
  int32_t i;
  if (m && m->version >= 0 && m->key == k) {
    i = m->version;
  } else {
    i = scan_versions(c, k);
    if (i < 0) return -1;   // a miss is not remembered: an install may follow
    if (m) {
      m->key = k;
      m->version = i;
    }
  }
  c->last_hit[op] = i;
  c->last_key[op] = k;
  return i;
}

namespace {

float f32_of_bits(uint32_t bits) {
  float f;
  memcpy(&f, &bits, sizeof f);
  return f;
}

// inv_i = the float32 nearest to base^(-2i/rd), i < rd/2. The power is taken
// in x87 extended precision (64-bit significand) and rounded once to
// float32. With Llama-3 scaling the rule is applied to the extended value
// before that one rounding: wavelength w = 2 pi / inv; w < L / high keeps
// inv, w > L / low divides it by factor, and in between
// s = (L / w - low) / (high - low) blends inv / factor and inv as
// (1 - s) inv / factor + s inv (L = original context length).
void rope_inverse_frequencies(const Key &k, float *out) {
  const long double b = (long double)f32_of_bits(key_base_bits(k));
  const uint32_t rd = key_rd(k);
  const bool llama3 = key_scaling(k) == TRI_ROPE_SCALING_LLAMA3;
  const long double factor = f32_of_bits(uint32_t(k.k4 & 0xFFFFFFFFu));
  const long double low = f32_of_bits(uint32_t(k.k4 >> 32));
  const long double high = f32_of_bits(uint32_t(k.k5 & 0xFFFFFFFFu));
  const long double L = (long double)key_orig_max(k);
  const long double two_pi = 6.283185307179586476925286766559005768L;
  for (uint32_t i = 0; i < rd / 2; ++i) {
    const long double e = -2.0L * (long double)i / (long double)rd;
    long double inv = powl(b, e);
    if (llama3) {
      const long double w = two_pi / inv;
      if (w > L / low) {
        inv = inv / factor;
      } else if (w >= L / high) {
        const long double sm = (L / w - low) / (high - low);
        inv = (1.0L - sm) * inv / factor + sm * inv;
      }
    }
    out[i] = (float)inv;
  }
}

void release_modules(Version &v) {
  for (int i = 0; i < 3; ++i) {
    if (v.module[i]) be_unload(v.module[i]);
    v.module[i] = nullptr;
    v.fn[i] = nullptr;
  }
}

}  // namespace

namespace {

// Path of the stored tuning result of key k: named by a hash of the key,
// the device architecture and the candidate list, so a change of any of
// them names another file.
bool tune_path(const tri_cache *c, const Key &k, const Plan *cands, int n, char *path,
               size_t cap) {
  if (!c->code_dir[0]) return false;
  char arch[64] = {0};
  be_arch(arch, sizeof arch);
  uint64_t w[TRI_KEY_WORDS];
  key_words(k, w);
  uint64_t h = fnv1a64("tri-tune-1", 10);
  h = fnv1a64(arch, strlen(arch), h);
  h = fnv1a64(w, sizeof w, h);
  h = fnv1a64(cands, sizeof(Plan) * size_t(n), h);
  return snprintf(path, cap, "%s/tri-tune-%016llx.txt", c->code_dir, (unsigned long long)h) <
         int(cap);
}

// A stored choice: one decimal index below n.
bool read_choice(const char *path, int n, int32_t *choice) {
  void *data = nullptr;
  uint64_t len = 0;
  if (!read_file(path, &data, &len)) return false;
  char buf[16] = {0};
  memcpy(buf, data, len < 15 ? size_t(len) : 15);
  free(data);
  char *end = nullptr;
  const long v = strtol(buf, &end, 10);
  if (end == buf || (*end != '\n' && *end != '\0') || v < 0 || v >= n) return false;
  *choice = int32_t(v);
  return true;
}

// Releases what a partly built version holds.
void drop_version(Version &v) {
  release_modules(v);
  if (v.d_consts) be_free(v.d_consts);
  if (v.d_scratch) be_free(v.d_scratch);
  free(v.h_consts);
  v.d_consts = nullptr;
  v.h_consts = nullptr;
  v.d_scratch = nullptr;
}


}  // namespace

tri_status install_key(tri_cache *c, const Key &k, int32_t candidate, bool generic) {
  // A key that a version already matches adds nothing: a version appended
  // behind that one could never be selected.
  if (scan_versions(c, k) >= 0) return TRI_OK;
  Plan cands[kMaxCandidates];
  const int nc = plan_candidates(k, cands);
  if (candidate < -1 || candidate >= nc) return TRI_E_INVALID;
  if (c->n_versions >= c->capacity) return TRI_E_FULL;

  Version v;
  memset(&v, 0, sizeof v);
  v.key = k;
  v.guard = kExact;   // the generic guard follows the plan's choice below
  v.n_candidates = nc;
  v.candidate = candidate < 0 ? 0 : candidate;
  const uint32_t dt = key_dtype(k);
  const uint32_t op = key_op(k);
  const bool rope = op == TRI_OP_ROPE_QK || op == TRI_OP_QK_NORM_ROPE || op == TRI_OP_CHAIN;
  if (rope && !(key_rope_bits(k) & kRopeCache)) {
    v.n_consts = key_rd(k) / 2;
    v.h_consts = static_cast<float *>(malloc(sizeof(float) * v.n_consts));
    if (!v.h_consts) return TRI_E_NOMEM;
    rope_inverse_frequencies(k, v.h_consts);
    void *dev = nullptr;
    const int st = be_upload(v.h_consts, sizeof(float) * v.n_consts, &dev);
    if (st != 0) {
      drop_version(v);
      return tri_status(st);
    }
    v.d_consts = static_cast<float *>(dev);
  }

  // Split norm rows exchange partial sums through a scratch of the version,
  // zeroed here and left zero by every call, sized for the top token bucket
  // the version serves (the key's; for a generic version the top of its run
  // as a split version, whose guard keeps only buckets where this fits):
  // allocated when the plan splits, or before tuning when any candidate does
  // (the tuning calls share it, one after another on one stream), and kept
  // only if the chosen plan splits.
  const bool tuning = candidate < 0 && (c->flags & TRI_CACHE_AUTOTUNE) && nc > 1;
  int split_cand = splits_rows(cands[v.candidate]) ? v.candidate : -1;
  for (int i = 0; tuning && split_cand < 0 && i < nc; ++i)
    if (splits_rows(cands[i])) split_cand = i;
  if (split_cand >= 0) {
    const uint32_t top =
        generic ? uint32_t(generic_guard(k, cands[split_cand]).b_hi) : key_bucket(k);
    v.scratch_words = split_words(int64_t(1) << top, split_slices(dt, key_H(k)));
    void *dev = nullptr;
    const int st = be_alloc_zeroed(v.scratch_words * 8, &dev);
    if (st != 0) {
      drop_version(v);
      return tri_status(st);
    }
    v.d_scratch = static_cast<uint64_t *>(dev);
  }

  if (tuning) {
    // Benchmark-and-keep (Sec. 2): a stored choice, else a timed one.
    const auto t0 = std::chrono::steady_clock::now();
    char path[1100];
    const bool dir = tune_path(c, k, cands, nc, path, sizeof path);
    if (dir && read_choice(path, nc, &v.candidate)) {
      v.tuned = TRI_TUNE_STORED;
    } else {
      tune_key(c, k, cands, nc, v, &v.candidate, &v.tuned);
      if (dir && v.tuned == TRI_TUNE_MEASURED) {
        char buf[16];
        const int m = snprintf(buf, sizeof buf, "%d\n", v.candidate);
        write_file(path, buf, uint64_t(m));
      }
    }
    v.tune_ms = float(std::chrono::duration<double, std::milli>(
                          std::chrono::steady_clock::now() - t0).count());
  }
  v.plan = cands[v.candidate];
  v.guard = generic ? generic_guard(k, v.plan) : kExact;
  if (v.d_scratch && !splits_rows(v.plan)) {
    be_free(v.d_scratch);
    v.d_scratch = nullptr;
    v.scratch_words = 0;
  }

  // A compiled specialization fixes the key's shape fields, so a version
  // with a range of row lengths runs the precompiled kernels.
  if ((c->flags & TRI_CACHE_JIT) && v.guard.h_lo == 0) {
    // Compile one specialization per launch of the plan (Sec. 3.5 growth),
    // or load it from the code directory.
    v.jit = 2;
    for (int i = 0; i < v.plan.n_launches; ++i) {
      uint64_t len = 0;
      char *src = jit_source(k, v.plan, i, &len);
      if (!src) {
        drop_version(v);
        return TRI_E_NOMEM;
      }
      float ms = 0.0f;
      bool from_dir = false;
      const int st = jit_build(c, src, len, &v.fn[i], &v.module[i], &ms, &from_dir);
      free(src);
      v.build_ms += ms;
      if (!from_dir) v.jit = 1;
      if (st != 0) {
        drop_version(v);
        return tri_status(st);
      }
    }
  } else {
    for (int i = 0; i < v.plan.n_launches; ++i) {
      const int st = be_resolve(v.plan.kvariant[i], dt, v.plan.ksub[i], &v.fn[i]);
      if (st != 0) {
        drop_version(v);
        return tri_status(st);
      }
    }
    // the argument-free form of each launch's kernel, for resident argument
    // blocks (without it that launch carries its kernel arguments)
    for (int i = 0; dt <= 1 && i < v.plan.n_launches; ++i) {
      const uint32_t fam = resident_family(v.plan.kvariant[i]);
      if (fam < kResFamilies && c->rtable[fam][dt] &&
          be_resolve_resident(v.plan.kvariant[i], dt, v.plan.ksub[i], &v.fn_res[i]) != 0)
        v.fn_res[i] = nullptr;
    }
  }
  c->versions[c->n_versions++] = v;
  c->stats.installs++;
  c->stats.n_versions = c->n_versions;
  return TRI_OK;
}

void fill_selection(const Version &v, int32_t index, int64_t T, tri_selection *out,
                    const Key *call_key) {
  const Key &k = v.key;
  const uint32_t dt = key_dtype(k);
  memset(out, 0, sizeof *out);
  out->op = int32_t(key_op(k));
  out->status = TRI_OK;
  out->version = index;
  out->variant = v.plan.variant;
  out->n_launches = v.plan.n_launches;
  for (int i = 0; i < 3; ++i) out->roles[i] = v.plan.roles[i];
  if (v.plan.variant == CH_FUSED) {
    const uint32_t g = role_grid(v.plan.roles[0], dt, T, key_H(k)) +
                       role_grid(v.plan.roles[1], dt, T, key_I(k), v.plan.rope_slices,
                                 v.plan.rope_tokens) +
                       role_grid(v.plan.roles[2], dt, T, key_I(k));
    out->launch[0] = {CH_FUSED, g, kBlock};
  } else {
    for (int i = 0; i < v.plan.n_launches; ++i) {
      const int32_t kv = v.plan.kvariant[i];
      out->launch[i] = {kv,
                        is_norm_variant(kv)
                            ? norm_grid(kv, dt, T, launch_width(k, kv), key_op(k) != TRI_OP_RMSNORM)
                            : role_grid(kv, dt, T, launch_width(k, kv), v.plan.rope_slices,
                                        v.plan.rope_tokens),
                        role_block(kv)};
    }
  }
  key_words(call_key ? *call_key : k, out->key);
}

}  // namespace tri

using namespace tri;

extern "C" {

tri_status tri_spec_cache_create(tri_cache **out, uint32_t capacity, uint32_t flags) {
  if (!out) return TRI_E_INVALID;
  *out = nullptr;
  if (capacity > kMaxCapacity ||
      (flags & ~uint32_t(TRI_CACHE_AUTO_INSTALL | TRI_CACHE_JIT | TRI_CACHE_AUTOTUNE |
                         TRI_CACHE_GENERIC | TRI_CACHE_RESIDENT_ARGS)))
    return TRI_E_INVALID;
  if (capacity == 0) capacity = kDefaultCapacity;
  int device = 0;
  int st = be_init(&device);
  if (st != 0) return tri_status(st);
  tri_cache *c = static_cast<tri_cache *>(calloc(1, sizeof(tri_cache)));
  if (!c) return TRI_E_NOMEM;
  c->versions = static_cast<Version *>(calloc(capacity, sizeof(Version)));
  c->memo = static_cast<MemoSlot *>(calloc(kMemoSlots, sizeof(MemoSlot)));
  if (!c->versions || !c->memo) {
    free(c->versions);
    free(c->memo);
    free(c);
    return TRI_E_NOMEM;
  }
  for (uint32_t i = 0; i < kMemoSlots; ++i) c->memo[i].version = -1;
  st = be_resolve(EMPTY, 0, 0, &c->empty_fn);
  if (st != 0) {
    free(c->versions);
    free(c->memo);
    free(c);
    return tri_status(st);
  }
  // the allocation-free entry point's fixed scratch on this device (a
  // failed lookup only disables the split rows of that entry point)
  if (be_noalloc_scratch(device, &c->noalloc_scratch) != 0) c->noalloc_scratch = nullptr;
  // resident argument blocks: the device's tables (a failed lookup or
  // check leaves the flag without effect)
  if (flags & TRI_CACHE_RESIDENT_ARGS) {
    c->held = static_cast<ResidentBlock *>(
        calloc(size_t(kResFamilies) * 2 * kResidentSlots, sizeof(ResidentBlock)));
    if (!c->held) {
      free(c->versions);
      free(c->memo);
      free(c);
      return TRI_E_NOMEM;
    }
    for (uint32_t fam = 0; fam < kResFamilies; ++fam)
      for (uint32_t dt : {uint32_t(TRI_F32), uint32_t(TRI_BF16)})
        if (be_resident_table(device, fam, dt, &c->rtable[fam][dt]) != 0)
          c->rtable[fam][dt] = nullptr;
  }
  c->capacity = capacity;
  c->flags = flags;
  c->device = device;
  for (int i = 0; i < kOps; ++i) c->last_hit[i] = -1;
  c->stats.capacity = capacity;
  c->last.version = -1;
  *out = c;
  return TRI_OK;
}

void tri_spec_cache_destroy(tri_cache *c) {
  if (!c) return;
  resident_release_all(c);
  free(c->held);
  for (uint32_t i = 0; i < c->n_versions; ++i) {
    if (c->versions[i].d_consts) be_free(c->versions[i].d_consts);
    if (c->versions[i].d_scratch) be_free(c->versions[i].d_scratch);
    free(c->versions[i].h_consts);
    release_modules(c->versions[i]);
  }
  free(c->versions);
  free(c->memo);
  free(c);
}

tri_status tri_spec_install_last_miss(tri_cache *c, tri_selection *out) {
  if (!c || !c->has_miss) return TRI_E_INVALID;
  const tri_status st = install_key(c, c->miss_key, -1, (c->flags & TRI_CACHE_GENERIC) != 0);
  if (st != TRI_OK) return st;
  if (out) {
    const int32_t i = scan_versions(c, c->miss_key);
    if (i >= 0) fill_selection(c->versions[i], i, c->miss_T, out, &c->miss_key);
  }
  return TRI_OK;
}

tri_status tri_spec_last_selection(const tri_cache *c, tri_selection *out) {
  if (!c || !out) return TRI_E_INVALID;
  *out = c->last;
  return TRI_OK;
}

tri_status tri_spec_stats(const tri_cache *c, tri_stats *out) {
  if (!c || !out) return TRI_E_INVALID;
  *out = c->stats;
  return TRI_OK;
}

tri_status tri_spec_resident_info(const tri_cache *c, tri_resident_info *out) {
  if (!c || !out) return TRI_E_INVALID;
  memset(out, 0, sizeof *out);
  for (uint32_t fam = 0; fam < kResFamilies; ++fam) {
    for (uint32_t dt = 0; dt < 2; ++dt) {
      if (c->rtable[fam][dt]) out->enabled = 1;
      out->held += c->n_held[fam][dt];
    }
  }
  out->launches = c->resident_launches;
  return TRI_OK;
}

tri_status tri_spec_version_info(const tri_cache *c, uint32_t index, tri_version_info *out) {
  if (!c || !out || index >= c->n_versions) return TRI_E_INVALID;
  const Version &v = c->versions[index];
  key_words(v.key, out->key);
  out->variant = v.plan.variant;
  for (int i = 0; i < 3; ++i) out->roles[i] = v.plan.roles[i];
  out->hits = v.hits;
  out->jit = v.jit;
  out->build_ms = v.build_ms;
  out->n_launches = v.plan.n_launches;
  for (int i = 0; i < 3; ++i) out->kernels[i] = i < v.plan.n_launches ? v.plan.kvariant[i] : 0;
  out->rope_slices = v.plan.rope_slices;
  out->candidate = v.candidate;
  out->n_candidates = v.n_candidates;
  out->tuned = v.tuned;
  out->tune_ms = v.tune_ms;
  out->rope_tokens = v.plan.rope_tokens;
  out->b_lo = v.guard.b_lo;
  out->b_hi = v.guard.b_hi;
  out->h_lo = v.guard.h_lo;
  out->h_hi = v.guard.h_hi;
  out->h_mod = v.guard.h_mod;
  return TRI_OK;
}

tri_status tri_spec_set_code_dir(tri_cache *c, const char *dir) {
  if (!c) return TRI_E_INVALID;
  if (!dir) {
    c->code_dir[0] = '\0';
    return TRI_OK;
  }
  const size_t n = strlen(dir);
  if (n >= sizeof c->code_dir) return TRI_E_INVALID;
  memcpy(c->code_dir, dir, n + 1);
  return TRI_OK;
}

tri_status tri_spec_export_keys(const tri_cache *c, uint64_t *keys, uint32_t cap, uint32_t *n) {
  if (!c || !n || (cap && !keys)) return TRI_E_INVALID;
  *n = c->n_versions;
  for (uint32_t i = 0; i < c->n_versions && i < cap; ++i)
    key_words(c->versions[i].key, keys + size_t(i) * TRI_KEY_WORDS);
  return TRI_OK;
}

tri_status tri_spec_import_keys(tri_cache *c, const uint64_t *keys, uint32_t n, uint32_t *done) {
  if (!c || (n && !keys)) return TRI_E_INVALID;
  uint32_t i = 0;
  tri_status st = TRI_OK;
  for (; i < n; ++i) {
    const uint64_t *w = keys + size_t(i) * TRI_KEY_WORDS;
    const Key k{w[0], w[1], w[2], w[3], w[4], w[5]};
    if (!key_valid(k)) {
      st = TRI_E_INVALID;
      break;
    }
    st = install_key(c, k);
    if (st != TRI_OK) break;
  }
  if (done) *done = i;
  return st;
}

tri_status tri_spec_install_key(tri_cache *c, const uint64_t *key, int32_t candidate) {
  if (!c || !key) return TRI_E_INVALID;
  const Key k{key[0], key[1], key[2], key[3], key[4], key[5]};
  if (!key_valid(k)) return TRI_E_INVALID;
  return install_key(c, k, candidate);
}

tri_status tri_spec_version_constants(const tri_cache *c, uint32_t index, float *out,
                                      uint32_t cap, uint32_t *n) {
  if (!c || !n || index >= c->n_versions) return TRI_E_INVALID;
  const Version &v = c->versions[index];
  *n = v.n_consts;
  if (v.n_consts && !out) return TRI_E_INVALID;
  for (uint32_t i = 0; i < v.n_consts && i < cap; ++i) out[i] = v.h_consts[i];
  return TRI_OK;
}

tri_status tri_launch_empty(tri_cache *c, void *stream) {
  if (!c) return TRI_E_INVALID;
  return be_launch(c->empty_fn, 1, 64, nullptr, 0, stream) == 0 ? TRI_OK : TRI_E_LAUNCH;
}

const char *tri_status_str(int status) {
  switch (status) {
    case TRI_OK: return "TRI_OK";
    case TRI_MISS: return "TRI_MISS";
    case TRI_E_INVALID: return "TRI_E_INVALID";
    case TRI_E_UNSUPPORTED: return "TRI_E_UNSUPPORTED";
    case TRI_E_FULL: return "TRI_E_FULL";
    case TRI_E_NOMEM: return "TRI_E_NOMEM";
    case TRI_E_LAUNCH: return "TRI_E_LAUNCH";
    case TRI_E_RUNTIME: return "TRI_E_RUNTIME";
    default: return "TRI_UNKNOWN";
  }
}

}  // extern "C"

// Internals of the specialization cache: key, versions, the install policy
// and the launch backend interface. Host-only C++; no HIP headers, so the
// cache core also builds with a plain host compiler against a recording
// backend for CPU tests.
#pragma once
#include <stdint.h>

#include "kernargs.h"
#include "tri.h"

namespace tri {

// ---- variant ids (the install policy table) ------------------------------------
enum Variant : int32_t {
  RN_SCALAR = 10,
  RN_WAVE_1 = 11, RN_WAVE_2 = 12,
  RN_BLOCK_1 = 13, RN_BLOCK_2 = 14, RN_BLOCK_4 = 15, RN_BLOCK_8 = 16, RN_BLOCK_16 = 17,
  RN_LOOP = 18, RN_WIDE = 19, RN_SPLIT = 20,
  ROPE_SCALAR = 30, ROPE_VEC = 31, ROPE_VEC_I = 32, ROPE_QKN_SCALAR = 33, ROPE_QKN_VEC = 34,
  ROPE_QKN_VEC_I = 35,
  SW_SCALAR = 40, SW_FLAT = 41, SW_FLAT_NT = 42, SW_ROWS = 43,
  CH_FUSED = 50, CH_SEQ = 51,
  ELT_SCALAR = 60, ELT_FLAT = 61, ELT_FLAT_U2 = 62, ELT_ROWS = 63,
  EMB_SCALAR = 70, EMB_VEC = 71,
  EMPTY = 99,
};

// Token buckets up to this one are "decode sized": RoPE head slices, one
// token per RoPE workgroup, one vector per element-wise work-item.
constexpr uint32_t kDecodeBucketMax = 6;

constexpr uint32_t kBlock = 256;
constexpr uint32_t kGridCap = 1u << 20;
constexpr int64_t kTMax = int64_t(1) << 22;
constexpr int64_t kHLimit = int64_t(1) << 24;
constexpr int64_t kILimit = int64_t(1) << 31;
constexpr uint64_t kSpanMax = uint64_t(1) << 47;   // bytes an operand's rows may span
constexpr int64_t kWideRowVecs = 8 * int64_t(kWideLanes);   // longest RN_WIDE row (vectors)
constexpr int64_t kWidePlainVecs = 7 * int64_t(kWideLanes);  // plain rows up to here: RN_WIDE
constexpr uint32_t kWidePlainBucket = 9;  // longer plain rows (up to kWideRowVecs): RN_WIDE from here
// RN_SPLIT: rows beyond 16 * 256 vectors, at most kSplitMaxSlices workgroups
// per row; a version's scratch (kSplitHeaderWords + 2^bucket * (S + 1)
// words) may take at most kSplitScratchWords (32 MiB), else the longer
// forms serve the key.
constexpr uint64_t kSplitScratchWords = uint64_t(1) << 22;
constexpr int32_t kHdMax = 512;
constexpr int32_t kHeadsMax = 4096;
constexpr uint32_t kDefaultCapacity = 256;
constexpr uint32_t kMaxCapacity = 4096;
constexpr unsigned kAlign = 1, kContig = 2;   // per-role guard flag bits
constexpr unsigned kChainQkNorm = 0x40;        // chain key flag: QK-RMSNorm before RoPE

// ---- key --------------------------------------------------------------------------
// k0: op | dtype << 8 | bucket << 16 | flags << 24 | RoPE base bits << 32
// k1: H | I << 32
// k2: hd | nq << 16 | nk << 32
// k3: rotary dim | variant bits << 16 | scaling << 24 | original_max_pos << 32
// k4: factor bits | low_freq_factor bits << 32;  k5: high_freq_factor bits
// Fields an op does not use are zero.
struct Key {
  uint64_t k0, k1, k2, k3, k4, k5;
};
inline bool operator==(const Key &a, const Key &b) {
  return a.k0 == b.k0 && a.k1 == b.k1 && a.k2 == b.k2 && a.k3 == b.k3 && a.k4 == b.k4 &&
         a.k5 == b.k5;
}
inline uint32_t key_op(const Key &k) { return uint32_t(k.k0 & 0xFF); }
inline uint32_t key_dtype(const Key &k) { return uint32_t((k.k0 >> 8) & 0xFF); }
inline uint32_t key_bucket(const Key &k) { return uint32_t((k.k0 >> 16) & 0xFF); }
inline uint32_t key_flags(const Key &k) { return uint32_t((k.k0 >> 24) & 0xFF); }
inline uint32_t key_base_bits(const Key &k) { return uint32_t(k.k0 >> 32); }
inline uint32_t key_H(const Key &k) { return uint32_t(k.k1 & 0xFFFFFFFFu); }
inline uint32_t key_I(const Key &k) { return uint32_t(k.k1 >> 32); }
inline uint32_t key_hd(const Key &k) { return uint32_t(k.k2 & 0xFFFF); }
inline uint32_t key_nq(const Key &k) { return uint32_t((k.k2 >> 16) & 0xFFFF); }
inline uint32_t key_nk(const Key &k) { return uint32_t((k.k2 >> 32) & 0xFFFF); }
inline uint32_t key_rd(const Key &k) { return uint32_t(k.k3 & 0xFFFF); }
inline uint32_t key_rope_bits(const Key &k) { return uint32_t((k.k3 >> 16) & 0xFF); }
inline uint32_t key_scaling(const Key &k) { return uint32_t((k.k3 >> 24) & 0xFF); }
inline uint32_t key_orig_max(const Key &k) { return uint32_t(k.k3 >> 32); }
inline void key_words(const Key &k, uint64_t *w) {
  w[0] = k.k0;
  w[1] = k.k1;
  w[2] = k.k2;
  w[3] = k.k3;
  w[4] = k.k4;
  w[5] = k.k5;
}

// ceil(log2 T) for 1 <= T <= 2^22.
inline uint32_t token_bucket(int64_t T) {
  return T <= 1 ? 0u : uint32_t(64 - __builtin_clzll(uint64_t(T - 1)));
}

// ---- policy -------------------------------------------------------------------------
// Role choice: variant + workgroups for T tokens. Pure functions of the key
// fields they take; the per-call grid only depends on T and the sizes.
struct Role {
  int32_t variant;
  uint32_t grid;
};
// res: residual RMSNorm rows (and the chain's norm role); plain RMSNorm rows
// of 4097..kWidePlainVecs vectors take the 1024-lane workgroup at any bucket.
Role rn_role(uint32_t dtype, int64_t H, unsigned flags, int64_t T, uint32_t bucket, bool res);
// Workgroups per row of RN_SPLIT, and the scratch words a call of T rows
// of that split needs.
int32_t split_slices(uint32_t dtype, int64_t H);
// Whether rows of H split at most kSplitMaxSlices ways with a scratch for
// the top of `bucket` of at most kSplitScratchWords.
bool split_fits(uint32_t dtype, int64_t H, uint32_t bucket);
inline uint64_t split_words(int64_t T, int32_t S) {
  return uint64_t(kSplitHeaderWords) + uint64_t(T) * uint64_t(S + 1);
}
Role rope_role(uint32_t dtype, int32_t hd, int32_t rd, bool interleaved, unsigned flags, int64_t T,
               bool qk_norm);
Role sw_role(uint32_t dtype, int64_t I, unsigned flags, bool stream, int64_t T);
// Bytes a call at the top of the key's token bucket moves (SwiGLU and the
// chain; 0 for other ops); SwiGLU streams nontemporally above kStreamBytes.
uint64_t call_bytes(const Key &k);
constexpr uint64_t kStreamBytes = uint64_t(320) << 20;
// Workgroups of a role variant for T tokens; `width` is the row width of
// the launch's op (H for the norms, I for SwiGLU, W for the short ops); a
// vector RoPE role takes T * slices workgroups with head slices, else
// ceil(T / tokens).
uint32_t role_grid(int32_t variant, uint32_t dtype, int64_t T, int64_t width,
                   int32_t slices = 1, int32_t tokens = 1);
// Workgroups of a norm launch: role_grid's, except the plain (not residual)
// wide-row form, which takes at most kWideGrid workgroups.
uint32_t norm_grid(int32_t variant, uint32_t dtype, int64_t T, int64_t H, bool res);
// The row width role_grid takes for launch variant `kv` of a version with key k.
int64_t launch_width(const Key &k, int32_t kv);
inline bool is_norm_variant(int32_t v) { return v >= RN_SCALAR && v <= RN_SPLIT; }
// Work-items per workgroup of a launch of `variant`.
inline uint32_t role_block(int32_t variant) {
  return variant == RN_WIDE ? uint32_t(kWideLanes) : kBlock;
}
// RoPE vector roles at decode sizes split a token's heads over this many
// workgroups (1 otherwise).
int32_t rope_slices(uint32_t dtype, int32_t hd, int32_t rd, bool interleaved, int32_t n_heads,
                    uint32_t bucket, int32_t variant);
// RoPE vector roles beyond decode sizes take this many tokens per workgroup
// (1 at decode sizes).
int32_t rope_tokens(uint32_t dtype, int32_t rd, bool interleaved, int32_t n_heads,
                    uint32_t bucket, int32_t variant);
// The slice count's and tokens per workgroup's bits in RopeArgs::mode
// (none for one).
inline uint32_t rope_geometry_bits(int32_t slices, int32_t tokens) {
  return (slices > 1 ? uint32_t(slices) << kRopeSliceShift : 0u) |
         (tokens > 1 ? uint32_t(tokens) << kRopeTokensShift : 0u);
}
// Element-wise ops (silu, add, masked_fill) over [T, W] and embedding rows.
Role elt_role(uint32_t dtype, int64_t W, unsigned flags, uint32_t bucket, int64_t T);
Role emb_role(uint32_t dtype, int64_t H, unsigned flags, int64_t T);

// A version's plan: which kernels it launches, fixed at install.
struct Plan {
  int32_t variant;        // op variant or CH_FUSED / CH_SEQ
  int32_t roles[3];       // chain only
  int32_t n_launches;
  int32_t kvariant[3];    // kernel variant per launch
  int32_t rope_slices;    // workgroups per token of the RoPE role (vector forms)
  int32_t ksub[3];        // kernel sub-selector (residual flag / fused template index)
                          // fused: (role norm variant - RN_WAVE_1) * 8
                          //        + (GPT-J pairs) * 4
                          //        + (QK-RMSNorm before RoPE) * 2
                          //        + (SwiGLU role is SW_FLAT_NT)
  int32_t rope_tokens;    // tokens per workgroup of the RoPE role (vector forms)
};
Plan plan_for_key(const Key &k);

inline bool operator==(const Plan &a, const Plan &b) {
  if (a.variant != b.variant || a.n_launches != b.n_launches ||
      a.rope_slices != b.rope_slices || a.rope_tokens != b.rope_tokens)
    return false;
  for (int i = 0; i < 3; ++i)
    if (a.roles[i] != b.roles[i] || a.kvariant[i] != b.kvariant[i] || a.ksub[i] != b.ksub[i])
      return false;
  return true;
}

// ---- guards ----------------------------------------------------------------------------
// What a version matches (Algorithm 1 scans versions in creation order and
// takes the first whose guard holds). Exact (b_lo < 0): its key. Generic:
// every key equal to its own except that the token bucket may lie in
// [b_lo, b_hi] and, with h_lo > 0, H in [h_lo, h_hi] of divisibility class
// h_mod (TRI_H_*).
struct Guard {
  int32_t b_lo, b_hi;
  uint32_t h_lo, h_hi;
  int32_t h_mod;
};
constexpr Guard kExact = {-1, -1, 0, 0, TRI_H_ANY};
constexpr uint32_t kBucketMax = 22;
// The guard of the generic version a miss on k installs, running `chosen`:
// the widest run of buckets around k's with plan_for_key's plan, and for
// norm rows served by one bucket-independent kernel the row lengths it
// serves. When `chosen` splits norm rows the run keeps only the buckets
// whose split scratch fits (the version's scratch is sized for its top).
Guard generic_guard(const Key &k, const Plan &chosen);
bool splits_rows(const Plan &p);
bool guard_holds(const Key &vk, const Guard &g, const Key &k);

// Install-time tuning: the key's candidate plans, index 0 = plan_for_key.
constexpr int kMaxCandidates = 24;
int plan_candidates(const Key &k, Plan *out);   // returns the count (>= 1)
constexpr uint32_t kSliceBucketMax = 13;        // head-slice alternatives up to 8192 tokens
constexpr float kTuneMargin = 0.97f;
constexpr uint64_t kTuneScratchMax = uint64_t(4) << 30;
constexpr int kTuneWarmup = 2, kTuneRounds = 5;

// ---- backend --------------------------------------------------------------------------
// The launch backend. The HIP build resolves kernel handles with the runtime
// and launches with hipModuleLaunchKernel; the CPU test build records calls.
int be_init(int *device);                                         // 0 or tri_status
int be_resolve(int32_t kvariant, uint32_t dtype, int32_t ksub, void **fn);
// `args` is the kernel's single argument struct of `args_size` bytes (or null).
int be_launch(void *fn, uint32_t grid, uint32_t block, const void *args, uint32_t args_size,
              void *stream);
int be_upload(const void *host, uint64_t bytes, void **dev);      // per-version constants
int be_alloc_zeroed(uint64_t bytes, void **dev);                  // per-version scratch
void be_free(void *dev);
// Compile `src` (len bytes, NUL-terminated) for the device into a code
// object (*code malloc'd, caller frees) / load a code object: the kernel
// `tri_jit_kernel` becomes *fn, the loaded object *module. 0 or tri_status.
int be_compile(const char *src, uint64_t len, void **code, uint64_t *code_len);
int be_load_code(const void *code, uint64_t code_len, void **fn, void **module);
void be_unload(void *module);
// Graph capture: a private stream in capture mode; ending the capture
// instantiates the recorded launches. 0 or tri_status.
int be_capture_begin(void **stream);
int be_capture_end(void *stream, void **exec);   // also releases the stream
int be_graph_launch(void *exec, void *stream);
void be_graph_destroy(void *exec);
// Tuning: zero-filled device memory (released with be_scratch_free), and a
// timer = a private stream of default priority with n_events event slots.
int be_scratch(uint64_t bytes, void *stream, void **dev);
void be_scratch_free(void *dev);
int be_timer_create(uint32_t n_events, void **timer, void **stream);
int be_timer_record(void *timer, uint32_t i);                 // event i on the timer's stream
int be_timer_elapsed(void *timer, uint32_t i, uint32_t j, float *ms);   // waits for event j
void be_timer_destroy(void *timer);
void be_arch(char *out, uint32_t cap);                         // device architecture name
// The fixed scratch of the allocation-free entry point: the device address
// of this device's copy of the library's static array (looked up once per
// device, with that device current). 0 or tri_status.
constexpr uint64_t kNoAllocScratchWords = uint64_t(TRI_NOALLOC_SCRATCH_BYTES) / 8;
int be_noalloc_scratch(int device, void **ptr);

// Resident argument blocks (TRI_CACHE_RESIDENT_ARGS). be_resident_table: the
// device address of this device's table for a kernel family and dtype,
// looked up -- and the LDS channel checked -- once per device with it
// current. be_resolve_resident: the argument-free form of the kernel
// be_resolve gives for the same (kvariant, dtype, ksub). be_resident_write:
// a synchronous copy into `device`'s table.
// be_launch_resident: launch `fn` on slot `slot` (slot * kLdsGranule bytes
// of dynamic LDS, no kernel arguments). be_stream_capturing: 1 when the
// stream is being captured (or the query fails), else 0. be_device_sync:
// wait until `device` is idle (the current device is kept). 0 or tri_status.
int be_resident_table(int device, uint32_t family, uint32_t dtype, void **table);
int be_resolve_resident(int32_t kvariant, uint32_t dtype, int32_t ksub, void **fn);
int be_resident_write(int device, void *dst, const void *src, uint32_t bytes);
int be_launch_resident(void *fn, uint32_t grid, uint32_t block, uint32_t slot, void *stream);
int be_stream_capturing(void *stream);
void be_device_sync(int device);
static_assert(kResidentSlots == uint32_t(TRI_RESIDENT_SLOTS), "resident slots");
// Launches of more than kResidentMaxGrid workgroups take only slots below
// kResidentAnyGridSlots: slot k adds k * kLdsGranule bytes of LDS per
// workgroup, and up to slot 9 eight 256-lane workgroups (a compute unit's
// most) with at most 7 granules of static LDS still fit its 160 KB.
constexpr uint32_t kResidentMaxGrid = TRI_RESIDENT_MAX_GRID;
constexpr uint32_t kResidentAnyGridSlots = TRI_RESIDENT_ANY_GRID_SLOTS;
static_assert(8 * (kResidentAnyGridSlots - 1 + 7) * kLdsGranule <= 160 * 1024,
              "any-grid slots keep eight workgroups per compute unit");
// The resident family of a kernel variant (kResFamilies: none).
inline uint32_t resident_family(int32_t kvariant) {
  if (kvariant == CH_FUSED) return kResChain;
  if (kvariant >= RN_SCALAR && kvariant <= RN_SPLIT) return kResNorm;
  if (kvariant >= ROPE_SCALAR && kvariant <= ROPE_QKN_VEC_I) return kResRope;
  if (kvariant >= SW_SCALAR && kvariant <= SW_ROWS) return kResSwiglu;
  if (kvariant >= ELT_SCALAR && kvariant <= ELT_ROWS) return kResElt;
  if (kvariant == EMB_SCALAR || kvariant == EMB_VEC) return kResEmb;
  return kResFamilies;
}

// ---- versions and the cache ------------------------------------------------------------
struct Version {
  Key key;                // the key the version was made for
  Guard guard;
  Plan plan;
  void *fn[3];
  void *module[3];        // runtime-compiled code objects, or null
  int32_t jit;
  float build_ms;
  int32_t candidate, n_candidates, tuned;
  float tune_ms;
  float *d_consts;        // device copy of the RoPE inverse frequencies, or null
  float *h_consts;        // host copy (rotary_dim/2 floats), or null
  void *fn_res[3];        // the argument-free form of each launch's kernel, or null
  uint32_t n_consts;
  uint64_t *d_scratch;    // split norm rows: the exchange scratch, or null
  uint64_t scratch_words;
  uint64_t hits;
};

constexpr int kOps = 12;   // op ids 1..11

// Memo of first matches: a direct-mapped table of keys and the version
// Algorithm 1's scan selected for them. First match depends only on the key
// and versions are only ever appended, so an entry stays right for good.
constexpr uint32_t kMemoSlots = 1024;
struct MemoSlot {
  Key key;
  int32_t version;   // -1: empty
};

}  // namespace tri

struct tri_cache {
  uint32_t capacity;
  uint32_t flags;
  int device;
  uint32_t n_versions;
  tri::Version *versions;
  int32_t last_hit[tri::kOps];   // per op: version of the op's last lookup key, -1 none
  tri::Key last_key[tri::kOps];  // per op: that key
  tri::MemoSlot *memo;           // kMemoSlots entries, or null (no memo)
  bool has_miss;
  tri::Key miss_key;
  int64_t miss_T;
  tri_stats stats;
  tri_selection last;
  void *empty_fn;
  void *noalloc_scratch;         // this device's static scratch, or null
  char code_dir[1024];           // compiled code objects; empty: none
  // TRI_CACHE_RESIDENT_ARGS: per kernel family and dtype (TRI_F32, TRI_BF16)
  // the device table (null: not in use), the blocks held (host copies with
  // tag and size set) and the index of the block the last resident launch
  // matched.
  void *rtable[tri::kResFamilies][2];
  tri::ResidentBlock *held;      // [kResFamilies][2][kResidentSlots], or null
  uint32_t n_held[tri::kResFamilies][2];
  uint32_t last_held[tri::kResFamilies][2];
  uint64_t resident_launches;
};

namespace tri {
// The slot of a held block of the family and dtype equal to the `size`
// bytes at `args` and `grid`, holding a new one in a free slot below
// `limit` when the cache and the device's pool have room and `stream` is
// not being captured; -1: launch with kernel arguments (resident.cpp).
int32_t resident_slot(tri_cache *c, uint32_t family, uint32_t dtype, const void *args,
                      uint32_t size, uint32_t grid, void *stream, uint32_t limit);
// Return the cache's slots to the device's pool (after the device is idle).
void resident_release_all(tri_cache *c);
}  // namespace tri

// A captured decode step (api.cpp).
struct tri_graph {
  void *exec;              // the backend's instantiated graph
  uint32_t n_launches;
};

namespace tri {
// Cache core (cache.cpp). install_key: candidate -1 = the cache's rule.
int32_t find_version(tri_cache *c, uint32_t op, const Key &k);
// Algorithm 1 without the memos: the first version whose guard holds.
int32_t scan_versions(const tri_cache *c, const Key &k);
// candidate -1 = the cache's rule; generic: a generic version (miss installs
// under TRI_CACHE_GENERIC), else exact.
tri_status install_key(tri_cache *c, const Key &k, int32_t candidate = -1, bool generic = false);
// The selection record a call with T tokens and key *call_key (null: the
// version's own key) makes on version v.
void fill_selection(const Version &v, int32_t index, int64_t T, tri_selection *out,
                    const Key *call_key = nullptr);
// Runtime-compiled specializations (jit.cpp).
bool key_valid(const Key &k);
// Source of the specialization of launch `i` of a version (key k, plan p):
// the device prelude and one kernel; returns a malloc'd NUL-terminated text
// (caller frees) and its length, or null.
char *jit_source(const Key &k, const Plan &p, int i, uint64_t *len);
// Kernel of `src` for this cache: loaded from the cache's code directory
// when a code object of the same source is there, else compiled (and
// stored there). *from_dir tells which; *ms the time taken.
int jit_build(const tri_cache *c, const char *src, uint64_t len, void **fn, void **module,
              float *ms, bool *from_dir);
// Code-directory files (jit.cpp).
uint64_t fnv1a64(const void *p, uint64_t n, uint64_t h = 0xcbf29ce484222325ull);
bool read_file(const char *path, void **data, uint64_t *n);
void write_file(const char *path, const void *data, uint64_t n);
// Install-time tuning (tune.cpp): times the n candidates of `k` on a call
// of the key's shapes and returns the index to keep in *choice and
// TRI_TUNE_MEASURED or TRI_TUNE_SKIPPED in *how. `v` holds the version under
// construction (its device constants serve every candidate). Never fails:
// problems keep candidate 0.
void tune_key(tri_cache *c, const Key &k, const Plan *cands, int n, const Version &v,
              int32_t *choice, int32_t *how);
}  // namespace tri

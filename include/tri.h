/*
 * tri.h -- C ABI of libtri: guarded dispatch of short LLM decode kernels on
 * AMD MI355X (gfx950).
 *
 * What the library is
 * -------------------
 * A native specialization cache in the sense of the paper's Specialization
 * Cache Module (Sec. 3.1): one entry call per op invocation evaluates the
 * guards of every installed version in C, selects the first version whose
 * guards hold (ordered dispatch, Algorithm 1 in Sec. 3.2), prepares the
 * kernel arguments and launches the version's precompiled gfx950 kernel on
 * the caller's stream. No version matching is a MISS, reported with a status
 * distinct from every error (Sec. 3.4 keeps miss and error in distinct
 * result tags; Sec. 3.5 gives the three paths): nothing is launched and the
 * caller installs a version (tri_spec_install_last_miss) and calls again.
 * An error never installs anything and never tries another version.
 *
 * Guards (the key): op, dtype, hidden size H, intermediate size I, head_dim,
 * Q and K head counts, token-count bucket ceil(log2 T), 16-byte alignment of
 * every activation / weight pointer and row stride, contiguity of every row
 * stride, the RoPE base and the RoPE variant (rotary dim, pairing, position
 * width, angle source, frequency scaling and its parameters), packed into
 * one key. An exact version tests equality on the key, so at most one exact
 * version matches; a generic version (TRI_CACHE_GENERIC) holds over a range
 * of token buckets (and of row lengths), so versions may overlap and the
 * first in creation order runs.
 *
 * Conventions (all entry points)
 * ------------------------------
 * - Pointers are DEVICE pointers of the cache's device, owned by the caller,
 *   and must be aligned to their element size. Outputs are preallocated by
 *   the caller; no entry point allocates on the hit path.
 * - Strides are in ELEMENTS. `*_rs` is a row stride, `*_ts` a token stride;
 *   the innermost stride is always 1. A stride must be at least the logical
 *   width of its row, and the rows of one operand must span at most 2^47
 *   bytes: ((rows - 1) * stride + width) * element size, with rows = T (the
 *   embedding table: n_rows; a cos/sin cache: cos_sin_len rows of rd
 *   floats). No device memory is that large, and the bound keeps every
 *   offset the kernels form far from int64 overflow; beyond it the call is
 *   INVALID.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream). Work
 *   is enqueued asynchronously; the call returns before it completes.
 * - dtype: weights share the activations' dtype. Arithmetic is float32 with
 *   one rounding to the output dtype.
 * - T == 0 is a valid no-op: TRI_OK, nothing launched, no other argument
 *   inspected.
 * - Validation happens before any launch; a failed check returns a negative
 *   status and leaves the cache unchanged except its counters.
 * - One thread per cache. A cache is bound to the device current when it is
 *   created.
 * - Residual RMSNorm rows of more than 4096 16-byte vectors, and plain
 *   RMSNorm rows of more than 7168, may be split over several
 *   workgroups of one launch that exchange partial sums through scratch the
 *   version owns (allocated zeroed at install, left zeroed by every launch).
 *   Launches of one such version must not overlap in time: issue its calls
 *   on one stream (or order the streams), or use one cache per stream.
 *   The exchange waits a bounded time; a row whose partial sums do not all
 *   arrive is written as NaN and marks the scratch failed, after which
 *   every launch on it writes NaN rows (destroy the cache to recover). A
 *   failure is loud, never a silently wrong value.
 */
#ifndef TRI_H
#define TRI_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tri_cache tri_cache;
typedef struct tri_graph tri_graph;

typedef enum tri_dtype { TRI_F32 = 0, TRI_BF16 = 1 } tri_dtype;

/* TRI_MISS is positive and distinct from the negative errors (Sec. 3.4). */
typedef enum tri_status {
  TRI_OK = 0,
  TRI_MISS = 1,            /* no version matched; nothing launched         */
  TRI_E_INVALID = -1,      /* bad argument                                  */
  TRI_E_UNSUPPORTED = -2,  /* valid but beyond the library's limits         */
  TRI_E_FULL = -3,         /* install: cache at capacity                    */
  TRI_E_NOMEM = -4,        /* install: device or host allocation failed     */
  TRI_E_LAUNCH = -5,       /* the selected version's launch failed          */
  TRI_E_RUNTIME = -6       /* HIP runtime failure outside a launch          */
} tri_status;

typedef enum tri_op {
  TRI_OP_RMSNORM = 1, TRI_OP_RES_RMSNORM = 2, TRI_OP_ROPE_QK = 3,
  TRI_OP_SWIGLU = 4, TRI_OP_CHAIN = 5, TRI_OP_QK_NORM_ROPE = 6,
  TRI_OP_CHAIN_LAYERS = 7,  /* selection records of tri_decode_chain_layers */
  TRI_OP_SILU = 8, TRI_OP_ADD = 9, TRI_OP_MASKED_FILL = 10, TRI_OP_EMBEDDING = 11
} tri_op;

enum { TRI_MAX_LAYERS = 1024 };   /* layers per tri_decode_chain_layers call */

enum {
  TRI_CACHE_AUTO_INSTALL = 1u,   /* on a miss: install, then launch */
  TRI_CACHE_JIT = 2u,            /* install compiles a key-specialized kernel */
  TRI_CACHE_AUTOTUNE = 4u,       /* install times the key's candidate plans */
  TRI_CACHE_GENERIC = 8u,        /* a miss installs a generic (range) version */
  TRI_CACHE_RESIDENT_ARGS = 16u  /* argument blocks held in device memory */
};

/* Resident argument blocks (TRI_CACHE_RESIDENT_ARGS): blocks per device,
 * kernel family and dtype; the largest launch (workgroups) that may take
 * any of them; the first blocks, which launches of any size may take. */
enum { TRI_RESIDENT_SLOTS = 40, TRI_RESIDENT_MAX_GRID = 512, TRI_RESIDENT_ANY_GRID_SLOTS = 10 };

/* Divisibility class of a generic version's hidden-size range
 * (tri_version_info.h_mod). */
enum { TRI_H_ANY = 0, TRI_H_MULTIPLE = 1, TRI_H_RAGGED = 2 };

/* How a version's plan was chosen (tri_version_info.tuned). */
enum {
  TRI_TUNE_NONE = 0,       /* the install policy's plan, or a pinned candidate */
  TRI_TUNE_MEASURED = 1,   /* the fastest candidate of a timed tuning call     */
  TRI_TUNE_STORED = 2,     /* a tuning result read from the code directory      */
  TRI_TUNE_SKIPPED = 3     /* tuning call too large or not possible: policy plan */
};

/* One kernel launch of a selection. */
typedef struct tri_launch_rec {
  int32_t variant;     /* kernel variant id (the install policy table)       */
  uint32_t grid_x;     /* workgroups                                          */
  uint32_t block_x;    /* work-items per workgroup (256; 1024 for variant 19) */
} tri_launch_rec;

/* Words of the packed guard key. */
enum { TRI_KEY_WORDS = 6 };

/* The selection record of the last entry call (or of an install). */
typedef struct tri_selection {
  int32_t op;          /* tri_op                                              */
  int32_t status;      /* tri_status the call returned                        */
  int32_t version;     /* index in creation order, -1 when none ran           */
  int32_t variant;     /* op variant (chain: 50 fused / 51 three launches)    */
  int32_t n_launches;  /* launches issued (0 on miss / error / T == 0)        */
  int32_t roles[3];    /* chain only: norm, RoPE, SwiGLU role variants        */
  tri_launch_rec launch[3];
  uint64_t key[TRI_KEY_WORDS];  /* packed guard key, zero when not computed   */
} tri_selection;

typedef struct tri_stats {
  uint64_t calls;      /* entry calls with a non-NULL cache                   */
  uint64_t hits;       /* a version matched and its launches succeeded        */
  uint64_t misses;     /* no version matched (auto-installed ones included)   */
  uint64_t errors;     /* negative status (validation or launch)              */
  uint64_t empty;      /* T == 0 no-ops                                       */
  uint64_t installs;   /* versions created                                    */
  uint32_t n_versions;
  uint32_t capacity;
} tri_stats;

typedef struct tri_version_info {
  uint64_t key[TRI_KEY_WORDS];
  int32_t variant;
  int32_t roles[3];
  uint64_t hits;
  int32_t jit;         /* 1: kernels compiled at install for this key;
                          2: loaded from the code directory                  */
  float build_ms;      /* install time spent compiling (0 when precompiled)  */
  int32_t n_launches;  /* launches per call                                  */
  int32_t kernels[3];  /* kernel variant of each launch (fused chain: 50)    */
  int32_t rope_slices; /* workgroups per token of the RoPE role (1: none)    */
  int32_t candidate;   /* index of the plan among the key's candidates       */
  int32_t n_candidates;
  int32_t tuned;       /* TRI_TUNE_*                                          */
  float tune_ms;       /* install time spent tuning                          */
  int32_t rope_tokens; /* tokens per workgroup of the RoPE role (1: one)     */
  /* Guards (Sec. 3.2): an exact version (b_lo < 0) matches its key only; a
   * generic one matches every key equal to its own except that the token
   * bucket may lie in [b_lo, b_hi] and, when h_lo > 0, the hidden size H in
   * [h_lo, h_hi] within class h_mod (TRI_H_*: any; a whole number of 16-byte
   * vectors; not one). */
  int32_t b_lo, b_hi;
  uint32_t h_lo, h_hi;
  int32_t h_mod;
} tri_version_info;

/* RoPE variants. A zeroed struct (or a NULL pointer where one is taken) is
 * the plain rotation of tri_rope_qk. None of these is defined in the paper;
 * they are the common forms of the op in Llama-family and GPT-J / NeoX
 * models, each a guard field of the key (a new shape of the op grows the
 * cache, Sec. 3.5).
 *  rotary_dim   rd: rotate the first rd elements of each head, pass the rest
 *               through (0 means hd); even, 2..hd. inv_i = RN_f32(base^(-2i/rd)).
 *  interleaved  0: pairs (i, i + rd/2) (rotate-half); 1: pairs (2i, 2i + 1)
 *               (GPT-J).
 *  pos_int64    0: pos is int32 [T] (4-byte aligned); 1: int64 [T] (8-byte
 *               aligned). A position becomes float32 by round-to-nearest-even.
 *  scaling      TRI_ROPE_SCALING_LLAMA3: the inverse frequencies are
 *               rescaled at install by the Llama-3 rule with factor,
 *               low_freq_factor, high_freq_factor and original_max_pos
 *               (wavelength 2 pi / inv_i below original_max_pos /
 *               high_freq_factor: kept; above original_max_pos /
 *               low_freq_factor: divided by factor; in between: linear in
 *               original_max_pos / wavelength), evaluated in extended
 *               precision and rounded once. factor, low_freq_factor finite
 *               and > 0, high_freq_factor finite and > low_freq_factor,
 *               original_max_pos >= 1.
 *  cos_sin      optional float32 cache [cos_sin_len, rd] (4-byte aligned):
 *               row p holds cos_0 .. cos_{rd/2-1} then sin_0 .. sin_{rd/2-1}
 *               for position p; positions are clamped to [0, cos_sin_len -
 *               1]. With a cache, base is not used (nor checked) and scaling
 *               must be NONE; cos_sin_len >= 1. */
typedef enum tri_rope_scaling {
  TRI_ROPE_SCALING_NONE = 0,
  TRI_ROPE_SCALING_LLAMA3 = 1
} tri_rope_scaling;

typedef struct tri_rope_ext {
  int32_t rotary_dim;
  int32_t interleaved;
  int32_t pos_int64;
  int32_t scaling;               /* tri_rope_scaling */
  float factor;
  float low_freq_factor;
  float high_freq_factor;
  int32_t original_max_pos;
  const float *cos_sin;
  int64_t cos_sin_len;
} tri_rope_ext;

/* Arguments of tri_decode_chain: the three ops on disjoint operands. */
typedef struct tri_chain_args {
  int32_t dtype;       /* tri_dtype for every tensor                          */
  int32_t nq, nk, hd;  /* RoPE: Q heads, K heads, head_dim                    */
  int64_t T, H, I;     /* tokens, hidden size, intermediate size              */
  float eps;           /* RMSNorm epsilon                                      */
  float base;          /* RoPE base                                            */
  /* residual add + RMSNorm over [T, H] */
  const void *x;   int64_t x_rs;
  const void *res; int64_t res_rs;
  const void *w;                       /* [H]                                 */
  void *y;         int64_t y_rs;
  void *res_out;   int64_t ro_rs;
  /* RoPE, in place: q [T, nq, hd], k [T, nk, hd], head stride hd */
  void *q;         int64_t q_ts;
  void *k;         int64_t k_ts;
  const void *pos;                     /* [T] int32 (int64 if rope_ext says)  */
  /* SwiGLU over [T, I] */
  const void *gate; int64_t g_rs;
  const void *up;   int64_t u_rs;
  void *out;        int64_t o_rs;
  /* optional per-head RMSNorm of Q and K before RoPE (Qwen3-style): NULL
   * q_norm_w disables it; otherwise q_norm_w [hd] and (when nk > 0)
   * k_norm_w [hd] are the head-norm weights and qk_eps their epsilon. */
  const void *q_norm_w;
  const void *k_norm_w;
  float qk_eps;
  int32_t reserved;    /* padding; ignored */
  /* optional RoPE variant (NULL: plain rotate-half over hd, int32 positions) */
  const tri_rope_ext *rope_ext;
} tri_chain_args;

/* ---- cache ---------------------------------------------------------------- */

/* Create an empty cache on the current device. capacity 0 selects 256
 * (at most 4096); flags: TRI_CACHE_AUTO_INSTALL, TRI_CACHE_JIT,
 * TRI_CACHE_AUTOTUNE, TRI_CACHE_GENERIC and TRI_CACHE_RESIDENT_ARGS in any
 * combination. The
 * cache owns every version, its kernel handles (and, with TRI_CACHE_JIT,
 * its loaded code objects) and its device constants; release it with
 * tri_spec_cache_destroy. Errors: INVALID (NULL out, capacity or flags out
 * of range), RUNTIME (no usable device), NOMEM.
 *
 * TRI_CACHE_JIT is the paper's growth path (Sec. 3.5: a miss captures,
 * compiles and installs a new specialization): installing a key compiles,
 * with hipRTC for gfx950, a kernel for each of the version's launches whose
 * shape fields (hidden size, intermediate size, head_dim, rotary dim, head
 * counts, RoPE variant bits) are compile-time constants of that key, around
 * the same device bodies as the precompiled variants; the install policy,
 * the launch geometry and the selection records are those of the
 * precompiled path. A failed compilation fails the install with RUNTIME. */
/* TRI_CACHE_AUTOTUNE is the benchmark-and-keep scheme of Triton's
 * autotuner that the paper describes (Sec. 2): every key has an ordered
 * list of candidate plans -- index 0 the install policy's plan, then the
 * other kernel variants whose preconditions the key guarantees (another
 * register layout or the two-pass kernel for norm rows, 1 / 2 / 4
 * workgroups per token or the scalar kernel for vector RoPE, the other flat
 * form or the row kernel for SwiGLU and the element-wise ops, every
 * combination of those for the fused chain and then its three-launch
 * sequence). Installing a key with more than one candidate makes a tuning
 * call of the key's shapes (tokens = the top of its bucket, row strides =
 * the width when contiguous, else the next multiple of 16 bytes above it,
 * or one element more when unaligned) on zero-filled device memory of its
 * own, on a private stream, through the same entry points: two warm-up
 * rounds and five timed rounds over the candidates in turn, each call
 * timed with HIP events. The fastest median is kept when it beats
 * candidate 0's by more than 3 %; otherwise candidate 0 stays. Keys whose
 * tuning call needs more than 4 GiB of operands keep candidate 0
 * (TRI_TUNE_SKIPPED), as do keys whose memory cannot be allocated. With a
 * code directory the choice is stored there (named by a hash of the key,
 * the device's architecture and the candidate list) and later installs
 * read it instead of timing. With TRI_CACHE_JIT the chosen plan is then
 * compiled. Installs (and so misses under auto-install) allocate, create a
 * stream and synchronize: do them before capturing a graph. */
/* TRI_CACHE_GENERIC: the paper's guards can hold across many concrete
 * inputs (Sec. 3.2: a rank check and a shape bound such as
 * weight.numel() <= 4096), so versions may overlap and the first one in
 * creation order whose guards hold runs (Algorithm 1). With this flag an
 * install made for a miss (auto-install, tri_spec_install_last_miss)
 * creates a generic version: it matches the missed key with any token
 * bucket in the widest run of buckets around the key's over which the
 * install policy picks the same plan, and -- for RMSNorm and residual
 * RMSNorm rows held by one wavefront or one workgroup, or by the scalar
 * kernel -- any hidden size that kernel serves (rows of 1-64, 65-128,
 * 129-256, ..., 2049-4096 16-byte vectors, plain RMSNorm rows also
 * 4097-7168, every length of the scalar kernel's class). A version whose
 * plan (the policy's or a tuned one) splits norm rows over workgroups keeps
 * only the buckets of that run whose split scratch fits (at most 32 MiB,
 * allocated for the top bucket at install), and matches its exact hidden
 * size. tri_spec_install_key and tri_spec_import_keys always create
 * exact versions, so exact versions installed first take precedence over
 * later generic ones that overlap them, and a key that an installed
 * version already matches installs nothing (a version behind it could
 * never run). With TRI_CACHE_JIT, a version with a hidden-size range runs
 * the precompiled kernels (a compiled specialization fixes H). */
/* TRI_CACHE_RESIDENT_ARGS (not in the paper; it removes part of the
 * per-call launch cost the paper measures in Sec. 2.3): the runtime places
 * a launch's kernel arguments in device memory on every launch, which costs
 * about as much host and end-to-end time as the 1-token chain's whole
 * kernel. With this flag a launch by a precompiled version takes its
 * argument block from a table in device memory instead -- every op's
 * launches, the fused chain's and the three of a three-launch chain. The first call with a given block (every
 * pointer, stride, size, eps and the launch geometry equal) copies it into
 * a free slot of the device's table for the kernel's family (the chain,
 * norms, RoPE, SwiGLU, element-wise ops, embedding) and dtype
 * (TRI_RESIDENT_SLOTS each per device, shared by the process's caches),
 * synchronously on a private stream; every later call with an equal block
 * launches a form of the same kernel that takes no kernel arguments and
 * finds its slot through its own LDS allocation (the call requests slot x
 * 1280 bytes of dynamic LDS, which the kernel reads back from a hardware
 * register). Pointers are held, not the data behind them: positions,
 * activations and weights are read on every call. Outputs equal the
 * ordinary launch's bit for bit, and the selection records are the same. A
 * held block is never rewritten while the cache lives; slots return to the
 * device's pool when the cache is destroyed (after the device has finished
 * its work). Slot k costs k x 1280 bytes of LDS per workgroup: a launch of
 * more than TRI_RESIDENT_MAX_GRID workgroups only takes one of the first
 * TRI_RESIDENT_ANY_GRID_SLOTS slots, at which the most workgroups a compute
 * unit runs at once (eight of 256 work-items) still fit its 160 KB of LDS
 * beside the kernels' own, so a large launch never runs fewer workgroups at
 * once. Calls launch as without the flag (kernel arguments) when the cache
 * holds TRI_RESIDENT_SLOTS blocks of the family and dtype or the pool has
 * no slot free that the launch may take, when the block is new while the
 * caller's stream is being captured, for compiled specializations
 * (TRI_CACHE_JIT), tri_residual_rmsnorm_noalloc and plain RMSNorm rows
 * of 4097..8192 16-byte vectors (that kernel holds its weights in 128 KiB
 * of LDS, which leaves too little for the slot), and on a device that
 * fails the check made at creation (launches at several LDS sizes whose slot the kernel must
 * read back exactly). tri_spec_resident_info tells how many launches used a
 * held block. A first call with a new block synchronizes a private stream:
 * make it before another thread starts a global-mode stream capture. A
 * graph that captured resident launches (tri_graph_build_layers, or the
 * caller's own capture) reads the cache's slots when replayed: destroy it
 * before the cache. */
tri_status tri_spec_cache_create(tri_cache **out, uint32_t capacity, uint32_t flags);
/* Release a cache and everything it owns (versions, kernel handles, loaded
 * code objects, device constants and scratch). Not in the paper (its module
 * lives as long as the Python callable); NULL is ignored. Graphs built from
 * the cache must be destroyed first. */
void tri_spec_cache_destroy(tri_cache *cache);

/* ---- ops (the hit path) ------------------------------------------------------ */

/* RMSNorm of each row of x [T, H]: y = w * x / sqrt(mean(x^2) + eps).
 * The paper's motivating kernel (`rms_norm`, Sec. 2.3 and Fig. 1); the
 * formula is the standard Llama form, float32 accumulation. y may alias x
 * exactly. Returns OK, MISS or an error. */
tri_status tri_rmsnorm(tri_cache *cache, tri_dtype dtype,
                       const void *x, int64_t x_rs, const void *w,
                       void *y, int64_t y_rs,
                       int64_t T, int64_t H, float eps, void *stream);

/* Fused residual add + RMSNorm: h = RN_dtype(x + res), res_out = h,
 * y = RMSNorm(h) (the norm of the rounded sum). `add` and `rms_norm` are in
 * the paper's kernel suite (Sec. 4.1). res_out may alias res and y may alias
 * x exactly. */
tri_status tri_residual_rmsnorm(tri_cache *cache, tri_dtype dtype,
                                const void *x, int64_t x_rs,
                                const void *res, int64_t res_rs,
                                const void *w,
                                void *y, int64_t y_rs,
                                void *res_out, int64_t ro_rs,
                                int64_t T, int64_t H, float eps, void *stream);

/* Rotary position embedding on Q [T, nq, hd] and K [T, nk, hd], in place,
 * rotate-half pairs (i, i + hd/2): theta = float32(pos[t]) * inv_i with
 * inv_i = RN_f32(base^(-2i/hd)); the same angles for every Q and K head of
 * a token. Not defined in the paper (a standard Llama-family op). hd even,
 * 2..512; nq 1..4096; nk 0..4096 (k may be NULL when nk == 0); pos int32 [T],
 * 4-byte aligned; base finite and > 1. The per-version table of inv_i is
 * computed and uploaded at install. */
tri_status tri_rope_qk(tri_cache *cache, tri_dtype dtype,
                       void *q, int64_t q_ts, void *k, int64_t k_ts,
                       const int32_t *pos, int64_t T,
                       int32_t nq, int32_t nk, int32_t hd, float base,
                       void *stream);

/* Per-head RMSNorm of Q and K followed by RoPE, in place (the head layout of
 * Qwen3, one of the two model families the paper evaluates, Sec. 4.1): each
 * head vector v is normalised to n = q_w * v / sqrt(mean(v^2) + eps) (k_w
 * for K heads; mean over the hd elements, float32 on the device), n is
 * rotated with the angles of tri_rope_qk, and the result is rounded to the
 * dtype once (n is not rounded). q_w [hd] is required, k_w [hd] when
 * nk > 0; both element-aligned; eps finite and >= 0. Other arguments and
 * errors as tri_rope_qk. */
tri_status tri_qk_norm_rope(tri_cache *cache, tri_dtype dtype,
                            void *q, int64_t q_ts, void *k, int64_t k_ts,
                            const int32_t *pos, int64_t T,
                            int32_t nq, int32_t nk, int32_t hd, float base,
                            const void *q_w, const void *k_w, float eps, void *stream);

/* RoPE with the variants of tri_rope_ext (ext may be NULL), optionally
 * after the per-head QK-RMSNorm of tri_qk_norm_rope (q_w non-NULL; the norm
 * covers all hd elements of a head, including those past rotary_dim). With
 * ext == NULL and q_w == NULL this is tri_rope_qk; with ext == NULL and q_w
 * set it is tri_qk_norm_rope (same keys, same versions). pos points to int32
 * or int64 positions as ext->pos_int64 says. Validation order: head_dim and
 * head counts; the ext fields; pointers and their alignment; strides; the
 * angle source (cache, or base and scaling parameters); the head-norm
 * weights and eps. */
tri_status tri_rope_qk_ext(tri_cache *cache, tri_dtype dtype,
                           void *q, int64_t q_ts, void *k, int64_t k_ts,
                           const void *pos, int64_t T,
                           int32_t nq, int32_t nk, int32_t hd, float base,
                           const tri_rope_ext *ext,
                           const void *q_w, const void *k_w, float eps, void *stream);

/* SwiGLU: out = g / (1 + exp(-g)) * u over [T, I] (`silu` is in the paper's
 * kernel suite, Sec. 4.1). out may alias gate or up exactly. */
tri_status tri_swiglu(tri_cache *cache, tri_dtype dtype,
                      const void *gate, int64_t g_rs, const void *up, int64_t u_rs,
                      void *out, int64_t o_rs, int64_t T, int64_t I, void *stream);

/* ---- short ops of the paper's operator suite (Sec. 4.1 lists silu, add,
 * masked_fill and embedding among its kernels); same cache, same guards
 * (dtype, row width, token bucket, 16-byte alignment, contiguity). ----- */

/* out = x / (1 + exp(-x)) over [T, W] (a signed zero where exp overflows).
 * out may alias x exactly. */
tri_status tri_silu(tri_cache *cache, tri_dtype dtype, const void *x, int64_t x_rs,
                    void *out, int64_t o_rs, int64_t T, int64_t W, void *stream);

/* out = RN_dtype(a + b) over [T, W]. out may alias a or b exactly. */
tri_status tri_add(tri_cache *cache, tri_dtype dtype, const void *a, int64_t a_rs,
                   const void *b, int64_t b_rs, void *out, int64_t o_rs,
                   int64_t T, int64_t W, void *stream);

/* out = mask ? RN_dtype(value) : x over [T, W]; mask is uint8 [T, W] with
 * row stride m_rs (nonzero = fill). Unmasked elements are copied bit for
 * bit. out may alias x exactly. value may be any float (inf included). */
tri_status tri_masked_fill(tri_cache *cache, tri_dtype dtype, const void *x, int64_t x_rs,
                           const uint8_t *mask, int64_t m_rs, float value,
                           void *out, int64_t o_rs, int64_t T, int64_t W, void *stream);

/* out[t, :] = table[ids[t], :] for t < T: table [n_rows, H] with row stride
 * t_rs, ids int32 [T] (int64 when ids_int64 is 1; 4- / 8-byte aligned).
 * An id outside [0, n_rows) yields a row of zeros (ids are device data; the
 * host never reads them). n_rows >= 1; out must not overlap the table. */
tri_status tri_embedding(tri_cache *cache, tri_dtype dtype, const void *table, int64_t t_rs,
                         int64_t n_rows, const void *ids, int32_t ids_int64,
                         void *out, int64_t o_rs, int64_t T, int64_t H, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * tri_residual_rmsnorm that allocates nothing on any path. Same arguments,
 * validation, guards, version lookup, kernels and selection records as
 * tri_residual_rmsnorm, with two differences:
 *  - it never installs: a miss returns TRI_MISS (key recorded for
 *    tri_spec_install_last_miss) even under TRI_CACHE_AUTO_INSTALL, since
 *    an install may allocate; install the version beforehand (an ordinary
 *    call, tri_spec_install_key or tri_spec_import_keys);
 *  - a version that splits its rows over several workgroups (rows of more
 *    than 4096 16-byte vectors) exchanges its partial sums through the
 *    library's fixed per-GPU array of TRI_NOALLOC_SCRATCH_BYTES (held from
 *    the first cache created on that GPU until the process ends) instead of
 *    the version's own scratch. A call needs 8 * (8 + T * (S + 1)) bytes of
 *    it, S = ceil(H / (8 * 2048)) for bf16 (H / (4 * 2048) for f32); a
 *    larger call returns TRI_E_UNSUPPORTED with nothing launched. Every
 *    call on a GPU shares that GPU's array and leaves it zeroed for the
 *    next: calls whose kernels overlap on one GPU (other streams, other
 *    caches) race.
 * TRI_E_RUNTIME if the array could not be located on the cache's device. */
enum { TRI_NOALLOC_SCRATCH_BYTES = 1 << 20 };
tri_status tri_residual_rmsnorm_noalloc(tri_cache *cache, tri_dtype dtype,
                                        const void *x, int64_t x_rs,
                                        const void *res, int64_t res_rs,
                                        const void *w,
                                        void *y, int64_t y_rs,
                                        void *res_out, int64_t ro_rs,
                                        int64_t T, int64_t H, float eps, void *stream);

/* The decode chain: residual+RMSNorm, RoPE-QK (or QK-RMSNorm + RoPE when
 * q_norm_w is set; with the variant of rope_ext when set) and SwiGLU of one
 * decode step, on disjoint operands
 * (overlap between the three ops is undefined). Not an operation of the
 * paper, which keeps one launch per kernel (its Sec. 5 contrasts the SCM
 * with mega-kernels); it is this path's one native entry (Sec. 3.1) for the
 * three short ops of a decode step, with the guards of all three in one key
 * (validation order: norm, RoPE, QK norm, SwiGLU). When
 * every tensor is 16-byte aligned and contiguous this is ONE launch of a
 * fused kernel whose workgroups take the three roles by blockIdx range;
 * otherwise three launches. If a later launch of the three fails, earlier
 * ones may already be enqueued; E_LAUNCH is returned and no other version is
 * tried. */
tri_status tri_decode_chain(tri_cache *cache, const tri_chain_args *args, void *stream);

/* Several decode chains in one entry call, e.g. the chains of every layer of
 * one decode step: layers[0 .. n_layers) run in array order on `stream`, so
 * a layer may consume an earlier layer's outputs. Pass 1 validates each
 * layer, packs its key and looks its version up (installing it under
 * TRI_CACHE_AUTO_INSTALL), in layer order; the first layer that fails
 * validation returns its error, and without auto-install the first layer
 * that misses returns MISS with its key recorded for
 * tri_spec_install_last_miss. In both cases NOTHING is launched. Pass 2
 * launches every layer (layers with T == 0 are skipped); a launch failure
 * returns E_LAUNCH with the earlier launches already enqueued.
 * n_layers 0..TRI_MAX_LAYERS (0, or all layers empty: OK, an empty call).
 * One entry call counts once in the statistics; a hit counts one hit on
 * each layer's version. The selection record has op TRI_OP_CHAIN_LAYERS,
 * the version, variant, roles, launches and key of the last launched layer,
 * and n_launches = the launches of all layers. Not in the paper: it
 * amortises the single native entry over a whole decode step. */
tri_status tri_decode_chain_layers(tri_cache *cache, const tri_chain_args *layers,
                                   uint32_t n_layers, void *stream);

/* A decode step as a HIP graph: the launches that tri_decode_chain_layers
 * would issue for `layers` (validated, looked up and -- under
 * TRI_CACHE_AUTO_INSTALL -- installed exactly as that call does; MISS and
 * errors as there, with no graph made) are captured once, in layer order,
 * into an instantiated graph that tri_graph_launch replays with one
 * submission. The graph fixes every pointer, size and kernel: a replay
 * evaluates no guard, so it is only valid while the caller's arguments stay
 * exactly those of the build (the data behind the pointers may change).
 * This is the CUDA-Graph trade-off the paper compares against (Sec. 4):
 * no per-call host work, no per-call checks. The graph uses the cache's
 * kernels and constants: destroy graphs before their cache. Capture uses a
 * private stream of default priority. Not counted in the cache's
 * statistics beyond the one build call. */
tri_status tri_graph_build_layers(tri_cache *cache, const tri_chain_args *layers,
                                  uint32_t n_layers, tri_graph **out);
/* Replay a graph on `stream` (asynchronous). RUNTIME if the launch fails. */
tri_status tri_graph_launch(tri_graph *graph, void *stream);
/* Launches the graph holds (the kernels of all its layers). */
uint32_t tri_graph_launch_count(const tri_graph *graph);
void tri_graph_destroy(tri_graph *graph);

/* ---- miss handling, introspection -------------------------------------------- */

/* Install a version for the key of the most recent MISS (Sec. 3.5: growth on
 * a miss): the install policy picks the kernel variant(s) from the key, the
 * kernel handles are resolved once, per-version constants (the RoPE inverse
 * frequencies) are uploaded, and the version is appended (generic under
 * TRI_CACHE_GENERIC). Idempotent: a key that an installed version already
 * matches adds nothing. `out` (nullable) receives the selection a call with
 * the missed arguments will make. Errors: INVALID (no miss yet), FULL,
 * NOMEM, RUNTIME. */
tri_status tri_spec_install_last_miss(tri_cache *cache, tri_selection *out);

/* Copy the selection record of the last entry call (which version of
 * Algorithm 1's ordered list ran, its kernels and launch geometry, the
 * packed key). Not in the paper: introspection for parity with the
 * selection model and for reporting. INVALID for NULL arguments. */
tri_status tri_spec_last_selection(const tri_cache *cache, tri_selection *out);

/* Copy the counters (calls, hits, misses, errors, T == 0 no-ops, installs):
 * the hit rate of Sec. 3.5's three paths. Not in the paper as an interface.
 * INVALID for NULL arguments. */
tri_status tri_spec_stats(const tri_cache *cache, tri_stats *out);

/* Resident argument blocks of a cache (TRI_CACHE_RESIDENT_ARGS). */
typedef struct tri_resident_info {
  int32_t enabled;      /* 1: the flag is set and the device passed the check */
  uint32_t held;        /* blocks the cache holds (both dtypes)              */
  uint64_t launches;    /* launches that took a held block                   */
} tri_resident_info;

/* Copy the cache's resident-block state. Not in the paper: introspection
 * of TRI_CACHE_RESIDENT_ARGS (all zero without the flag). INVALID for NULL
 * arguments. */
tri_status tri_spec_resident_info(const tri_cache *cache, tri_resident_info *out);

/* Describe version `index` (creation order; the versions of Algorithm 1).
 * Not in the paper: introspection. INVALID if out of range. */
tri_status tri_spec_version_info(const tri_cache *cache, uint32_t index,
                                 tri_version_info *out);

/* Copy version `index`'s host copy of its constants (RoPE inverse
 * frequencies, rotary_dim/2 floats; none for other ops or with a cos/sin
 * cache) into out[0..cap); *n gets the count. The paper's captured
 * constants (Sec. 3.3) made visible for parity tests; not an interface of
 * the paper. INVALID if out of range or out is NULL while *n > 0. */
tri_status tri_spec_version_constants(const tri_cache *cache, uint32_t index,
                                      float *out, uint32_t cap, uint32_t *n);

/* With TRI_CACHE_JIT: a directory of compiled code objects shared across
 * caches and processes (the on-disk half of the paper's Sec. 2.2 compile
 * cache). An install first looks for the code object of its exact source
 * (named by a 64-bit hash of the source text, the target and the compiler
 * flags) and loads it; otherwise it compiles and stores the object there
 * (written under a temporary name and renamed). Unreadable or corrupt files
 * are recompiled; write failures are ignored. NULL or "" turns it off; the
 * directory must exist. INVALID for a path of 1024 bytes or more. */
tri_status tri_spec_set_code_dir(tri_cache *cache, const char *dir);

/* The keys of the installed versions in creation order, TRI_KEY_WORDS words
 * each, into keys[0 .. cap * TRI_KEY_WORDS); *n = the number of versions
 * (which may exceed cap). For pre-warming another cache with
 * tri_spec_import_keys. */
tri_status tri_spec_export_keys(const tri_cache *cache, uint64_t *keys, uint32_t cap,
                                uint32_t *n);

/* Install versions for n keys (n * TRI_KEY_WORDS words, e.g. an earlier
 * export), in order, as an install after a miss would (already installed
 * keys add nothing). Each key is checked first -- known op, dtype, token
 * bucket <= 22, flags of the op, sizes within the entry points' limits,
 * consistent RoPE fields (base > 1 and finite unless a cos/sin cache, rotary
 * dim even and <= head_dim, Llama-3 parameters as tri_rope_ext requires),
 * unused fields zero; a malformed key stops the import with INVALID. FULL,
 * NOMEM, RUNTIME as for an install. *done = keys processed before the
 * stop (all n on OK). */
tri_status tri_spec_import_keys(tri_cache *cache, const uint64_t *keys, uint32_t n,
                                uint32_t *done);

/* Install one key (TRI_KEY_WORDS words, checked as tri_spec_import_keys
 * checks them) with a chosen plan: candidate -1 takes the cache's own rule
 * (tuned with TRI_CACHE_AUTOTUNE, else the install policy's plan);
 * 0 .. n_candidates - 1 pins that candidate (tri_version_info reports
 * n_candidates and the chosen index, so a tuned set of versions can be
 * exported and reinstalled without timing). A key already installed adds
 * nothing and keeps its plan. Errors: INVALID (NULL, malformed key,
 * candidate out of range), FULL, NOMEM, RUNTIME. */
tri_status tri_spec_install_key(tri_cache *cache, const uint64_t *key, int32_t candidate);

/* Launch the empty kernel (1 workgroup of 64 work-items, no arguments)
 * through the same launch path: the yardstick for per-call cost. Not in the
 * paper (its measurements compare against eager and torch.compile, Sec. 4);
 * the target of this path is a per-call cost close to this launch's. */
tri_status tri_launch_empty(tri_cache *cache, void *stream);

/* Static name of a status value ("TRI_UNKNOWN" for other values). Not in
 * the paper. */
const char *tri_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* TRI_H */

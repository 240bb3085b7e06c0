// Recording launch backend for CPU tests of the cache core (test double).
//
// Links with the library's host sources in place of the HIP backend. It
// computes nothing: "kernel handles" encode (variant, dtype, sub), launches
// are appended to a log with their grid, block and a copy of the argument
// block, and a launch can be made to fail on purpose (fault injection).
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <string>
#include <vector>

#include "internal.h"

namespace {

struct Rec {
  int32_t kvariant, dtype, ksub;
  uint32_t grid, block;
  unsigned char args[512];
  uint32_t nargs;
  void *stream;
  int32_t slot;   // resident launch: the slot (its block is in args); -1 otherwise
};

std::vector<Rec> g_log;
int64_t g_fail_at = -1;        // launch ordinal that fails, -1 none
int g_init_status = 0;
int64_t g_uploads = 0;
std::vector<std::string> g_jit;   // sources of the code objects loaded, in order
int64_t g_compiles = 0;
int64_t g_unloads = 0;
bool g_jit_fail = false;
int64_t g_captures = 0, g_capture_start = 0, g_graph_launches = 0, g_graph_destroys = 0;
bool g_capture_fail = false;
void *g_capturing = nullptr;   // the capture stream between begin and end

// Resident argument blocks: one host table per family and dtype stands in
// for the device's (shared by every cache, as the device's is).
tri::ResidentBlock g_res_table[tri::kResFamilies][2][tri::kResidentSlots];
bool g_res_check_fail = false, g_res_write_fail = false, g_force_capturing = false;
int64_t g_res_writes = 0, g_res_syncs = 0;

// Scripted launch costs of the tuning timer: the last matching entry wins
// (ksub -1 / grid 0 match any); unmatched launches cost 1 ms.
struct Cost {
  int32_t kvariant, ksub;
  uint32_t grid;
  float ms;
};
std::vector<Cost> g_costs;
std::vector<int64_t> g_marks;
int64_t g_timers = 0, g_timer_destroys = 0, g_scratch_allocs = 0, g_scratch_frees = 0;
uint64_t g_scratch_bytes = 0;
int64_t g_zero_allocs = 0;
uint64_t g_zero_bytes = 0;
bool g_scratch_fail = false;
std::string g_arch = "fake";

uintptr_t encode(int32_t v, uint32_t dt, int32_t sub) {
  return (uintptr_t(uint32_t(v)) << 20) | (uintptr_t(dt) << 16) | uintptr_t(uint32_t(sub) & 0xFFFF) |
         (uintptr_t(1) << 40);
}

}  // namespace

namespace tri {

int be_init(int *device) {
  *device = 0;
  return g_init_status;
}

int be_resolve(int32_t kvariant, uint32_t dtype, int32_t ksub, void **fn) {
  *fn = reinterpret_cast<void *>(encode(kvariant, dtype, ksub));
  return 0;
}

int be_launch(void *fn, uint32_t grid, uint32_t block, const void *args, uint32_t args_size,
              void *stream) {
  const int64_t n = int64_t(g_log.size());
  Rec r;
  memset(&r, 0, sizeof r);
  const uintptr_t h = reinterpret_cast<uintptr_t>(fn);
  if (h & (uintptr_t(1) << 41)) {   // a compiled specialization: -(its source index + 1)
    r.kvariant = -int32_t(((h >> 20) & 0xFFFFF) + 1);
  } else {
    r.kvariant = int32_t((h >> 20) & 0xFFFFF);
    r.dtype = int32_t((h >> 16) & 0xF);
    r.ksub = int32_t(h & 0xFFFF);
  }
  r.grid = grid;
  r.block = block;
  r.stream = stream;
  r.nargs = args && args_size <= sizeof r.args ? args_size : 0;
  if (r.nargs) memcpy(r.args, args, r.nargs);
  r.slot = -1;
  g_log.push_back(r);
  return n == g_fail_at ? -1 : 0;
}

int be_resident_table(int device, uint32_t family, uint32_t dtype, void **table) {
  (void)device;
  *table = nullptr;
  if (g_res_check_fail || family >= kResFamilies || dtype > 1) return TRI_E_RUNTIME;
  *table = g_res_table[family][dtype];
  return 0;
}

int be_resolve_resident(int32_t kvariant, uint32_t dtype, int32_t ksub, void **fn) {
  // as the device library: the plain wide-row norm has no argument-free form
  if (kvariant == RN_WIDE && ksub == 0) {
    *fn = nullptr;
    return TRI_E_RUNTIME;
  }
  *fn = reinterpret_cast<void *>(encode(kvariant, dtype, ksub) | (uintptr_t(1) << 42));
  return 0;
}

int be_resident_write(int device, void *dst, const void *src, uint32_t bytes) {
  (void)device;
  if (g_res_write_fail) return TRI_E_RUNTIME;
  memcpy(dst, src, bytes);
  g_res_writes++;
  return 0;
}

// Logged like a launch with arguments, with the block the kernel would find
// in its slot (none when the slot is out of range or its tag unset).
int be_launch_resident(void *fn, uint32_t grid, uint32_t block, uint32_t slot, void *stream) {
  const int64_t n = int64_t(g_log.size());
  Rec r;
  memset(&r, 0, sizeof r);
  const uintptr_t h = reinterpret_cast<uintptr_t>(fn);
  r.kvariant = int32_t((h >> 20) & 0xFFFFF);
  r.dtype = int32_t((h >> 16) & 0xF);
  r.ksub = int32_t(h & 0xFFFF);
  r.grid = grid;
  r.block = block;
  r.stream = stream;
  r.slot = int32_t(slot);
  const uint32_t fam = resident_family(r.kvariant);
  if (fam < kResFamilies && r.dtype <= 1 && slot < kResidentSlots &&
      g_res_table[fam][r.dtype][slot].tag == kResidentTag + slot) {
    const ResidentBlock &b = g_res_table[fam][r.dtype][slot];
    r.nargs = b.size;
    memcpy(r.args, b.args, b.size);
  }
  g_log.push_back(r);
  return n == g_fail_at ? -1 : 0;
}

int be_stream_capturing(void *stream) {
  return g_force_capturing || (g_capturing && stream == g_capturing) ? 1 : 0;
}

void be_device_sync(int device) {
  (void)device;
  g_res_syncs++;
}

int be_upload(const void *host, uint64_t bytes, void **dev) {
  void *p = malloc(bytes);
  if (!p) return TRI_E_NOMEM;
  memcpy(p, host, bytes);
  *dev = p;
  g_uploads++;
  return 0;
}

// Per-version scratch of split norm rows: zeroed host memory (counted).
int be_alloc_zeroed(uint64_t bytes, void **dev) {
  void *p = calloc(1, bytes);
  if (!p) return TRI_E_NOMEM;
  *dev = p;
  g_zero_allocs++;
  g_zero_bytes += bytes;
  return 0;
}

void be_free(void *dev) { free(dev); }

// The allocation-free entry point's fixed scratch: one host array standing
// in for every device's copy (looked up once, counted).
uint64_t g_noalloc[kNoAllocScratchWords];
int64_t g_noalloc_lookups = 0;
int be_noalloc_scratch(int device, void **ptr) {
  (void)device;
  g_noalloc_lookups++;
  *ptr = g_noalloc;
  return 0;
}

// Runtime compilation: the "code object" is the source behind a 4-byte
// tag; loading records the source and hands out a handle that encodes the
// position of the source in the log (bit 41 marks it).
int be_compile(const char *src, uint64_t len, void **code, uint64_t *code_len) {
  if (g_jit_fail) return TRI_E_RUNTIME;
  g_compiles++;
  char *buf = static_cast<char *>(malloc(size_t(len) + 4));
  if (!buf) return TRI_E_NOMEM;
  memcpy(buf, "CO1:", 4);
  memcpy(buf + 4, src, size_t(len));
  *code = buf;
  *code_len = len + 4;
  return 0;
}

int be_load_code(const void *code, uint64_t code_len, void **fn, void **module) {
  const char *b = static_cast<const char *>(code);
  if (code_len < 4 || memcmp(b, "CO1:", 4) != 0) return TRI_E_RUNTIME;
  g_jit.emplace_back(b + 4, size_t(code_len - 4));
  const uintptr_t idx = uintptr_t(g_jit.size() - 1);
  *fn = reinterpret_cast<void *>((uintptr_t(1) << 41) | (idx << 20));
  *module = reinterpret_cast<void *>(uintptr_t(0x100000 + idx));
  return 0;
}

void be_unload(void *module) {
  (void)module;
  g_unloads++;
}

// Graph capture: launches between begin and end are logged with the
// capture stream's handle; a "graph" remembers how many they were, and a
// graph launch is counted.
int be_capture_begin(void **stream) {
  if (g_capture_fail) return TRI_E_RUNTIME;
  *stream = reinterpret_cast<void *>(uintptr_t(0xCA000000u) + uintptr_t(g_captures++));
  g_capture_start = int64_t(g_log.size());
  g_capturing = *stream;
  return 0;
}

int be_capture_end(void *stream, void **exec) {
  (void)stream;
  g_capturing = nullptr;
  *exec = reinterpret_cast<void *>(uintptr_t(0xE0000000u) +
                                   uintptr_t(int64_t(g_log.size()) - g_capture_start));
  return 0;
}

int be_graph_launch(void *exec, void *stream) {
  (void)exec;
  (void)stream;
  g_graph_launches++;
  return 0;
}

void be_graph_destroy(void *exec) {
  (void)exec;
  g_graph_destroys++;
}

// Tuning: "scratch" is a stand-in address (nothing dereferences it); the
// timer's events mark positions in the launch log and an elapsed time is
// the scripted cost of the launches between two marks.
int be_scratch(uint64_t bytes, void *stream, void **dev) {
  (void)stream;
  if (g_scratch_fail) return TRI_E_NOMEM;
  g_scratch_bytes = bytes;
  g_scratch_allocs++;
  *dev = reinterpret_cast<void *>(uintptr_t(0x5C0000000000ull));
  return 0;
}

void be_scratch_free(void *dev) {
  (void)dev;
  g_scratch_frees++;
}

int be_timer_create(uint32_t n_events, void **timer, void **stream) {
  g_marks.assign(n_events, -1);
  g_timers++;
  *timer = reinterpret_cast<void *>(uintptr_t(0x71000000u) + uintptr_t(g_timers));
  *stream = reinterpret_cast<void *>(uintptr_t(0x72000000u) + uintptr_t(g_timers));
  return 0;
}

int be_timer_record(void *timer, uint32_t i) {
  (void)timer;
  if (i >= g_marks.size()) return TRI_E_INVALID;
  g_marks[i] = int64_t(g_log.size());
  return 0;
}

float launch_cost(const Rec &r) {
  float c = 1.0f;
  for (const Cost &k : g_costs)
    if (k.kvariant == r.kvariant && (k.ksub < 0 || k.ksub == r.ksub) &&
        (k.grid == 0 || k.grid == r.grid))
      c = k.ms;
  return c;
}

int be_timer_elapsed(void *timer, uint32_t i, uint32_t j, float *ms) {
  (void)timer;
  if (i >= g_marks.size() || j >= g_marks.size() || g_marks[i] < 0 || g_marks[j] < 0)
    return TRI_E_INVALID;
  float t = 0.0f;
  for (int64_t n = g_marks[i]; n < g_marks[j]; ++n) t += launch_cost(g_log[size_t(n)]);
  *ms = t;
  return 0;
}

void be_timer_destroy(void *timer) {
  (void)timer;
  g_timer_destroys++;
}

void be_arch(char *out, uint32_t cap) { snprintf(out, cap, "%s", g_arch.c_str()); }

}  // namespace tri

extern "C" {

void trifake_reset() {
  g_log.clear();
  g_fail_at = -1;
  g_init_status = 0;
  g_uploads = 0;
  g_jit.clear();
  g_compiles = 0;
  g_unloads = 0;
  g_jit_fail = false;
  g_captures = g_capture_start = g_graph_launches = g_graph_destroys = 0;
  g_capture_fail = false;
  g_costs.clear();
  g_marks.clear();
  g_timers = g_timer_destroys = g_scratch_allocs = g_scratch_frees = 0;
  g_scratch_bytes = 0;
  g_scratch_fail = false;
  g_zero_allocs = 0;
  g_zero_bytes = 0;
  tri::g_noalloc_lookups = 0;
  g_arch = "fake";
  g_capturing = nullptr;
  g_res_check_fail = g_res_write_fail = g_force_capturing = false;
  g_res_writes = g_res_syncs = 0;
}
// resident blocks: make the device check fail / the block copy fail /
// every stream report a capture; counts of block copies and device syncs
void trifake_resident_check_fail(int on) { g_res_check_fail = on != 0; }
void trifake_resident_write_fail(int on) { g_res_write_fail = on != 0; }
void trifake_force_capturing(int on) { g_force_capturing = on != 0; }
void trifake_resident_counts(int64_t *out) {
  out[0] = g_res_writes;
  out[1] = g_res_syncs;
}
// the stand-in table's slot s of a family and dtype: its tag, grid and
// argument size (-1 out of range)
int64_t trifake_resident_tag(int32_t family, int32_t dtype, int32_t s, uint32_t *grid,
                             uint32_t *size) {
  if (family < 0 || family >= int32_t(tri::kResFamilies) || dtype < 0 || dtype > 1 || s < 0 ||
      s >= int32_t(tri::kResidentSlots))
    return -1;
  const tri::ResidentBlock &b = g_res_table[family][dtype][s];
  if (grid) *grid = b.grid;
  if (size) *size = b.size;
  return int64_t(b.tag);
}
// slot of launch i (-1: a launch with arguments), or -2 if there is no launch i
int32_t trifake_slot(int64_t i) {
  if (i < 0 || i >= int64_t(g_log.size())) return -2;
  return g_log[size_t(i)].slot;
}
// address of the fixed scratch of the allocation-free entry point, and the
// lookups made
void *trifake_noalloc_scratch(int64_t *lookups) {
  if (lookups) *lookups = tri::g_noalloc_lookups;
  return tri::g_noalloc;
}
// zeroed scratch allocations of split norm versions and their total bytes
void trifake_zero_allocs(int64_t *out) {
  out[0] = g_zero_allocs;
  out[1] = int64_t(g_zero_bytes);
}
void trifake_set_cost(int32_t kvariant, int32_t ksub, uint32_t grid, float ms) {
  g_costs.push_back({kvariant, ksub, grid, ms});
}
void trifake_scratch_fail(int on) { g_scratch_fail = on != 0; }
void trifake_set_arch(const char *a) { g_arch = a ? a : ""; }
// timers created, timers destroyed, scratch allocations, frees, last size
void trifake_tune_counts(int64_t *out) {
  out[0] = g_timers;
  out[1] = g_timer_destroys;
  out[2] = g_scratch_allocs;
  out[3] = g_scratch_frees;
  out[4] = int64_t(g_scratch_bytes);
}
int64_t trifake_graph_launches() { return g_graph_launches; }
int64_t trifake_graph_destroys() { return g_graph_destroys; }
void trifake_capture_fail(int on) { g_capture_fail = on != 0; }
int64_t trifake_jit_count() { return int64_t(g_jit.size()); }
int64_t trifake_compile_count() { return g_compiles; }
int64_t trifake_unload_count() { return g_unloads; }
void trifake_jit_fail(int on) { g_jit_fail = on != 0; }
// Source i of the runtime compilations: copies up to cap bytes, returns its
// length (or -1).
int64_t trifake_jit_source(int64_t i, char *buf, int64_t cap) {
  if (i < 0 || i >= int64_t(g_jit.size())) return -1;
  const std::string &s = g_jit[size_t(i)];
  if (buf && cap > 0) memcpy(buf, s.data(), size_t(int64_t(s.size()) < cap ? int64_t(s.size()) : cap));
  return int64_t(s.size());
}
int64_t trifake_launch_count() { return int64_t(g_log.size()); }
int64_t trifake_upload_count() { return g_uploads; }
void trifake_fail_at(int64_t n) { g_fail_at = n; }
void trifake_init_status(int st) { g_init_status = st; }

// Launch i: kernel (variant, dtype, sub), grid, block, stream and the first
// `nbytes` bytes of its argument block (zero beyond its size). Returns the
// argument block's size, or -1 if there is no launch i.
int trifake_get(int64_t i, int32_t *kv, int32_t *dt, int32_t *sub, uint32_t *grid,
                uint32_t *block, void **stream, unsigned char *args, int nbytes) {
  if (i < 0 || i >= int64_t(g_log.size())) return -1;
  const Rec &r = g_log[size_t(i)];
  *kv = r.kvariant;
  *dt = r.dtype;
  *sub = r.ksub;
  *grid = r.grid;
  *block = r.block;
  *stream = r.stream;
  if (args && nbytes > 0) {
    const int n = nbytes > int(sizeof r.args) ? int(sizeof r.args) : nbytes;
    memcpy(args, r.args, size_t(n));
  }
  return int(r.nargs);
}

}  // extern "C"

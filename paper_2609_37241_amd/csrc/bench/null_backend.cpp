// A launch backend that does nothing, for timing the library's own host work
// (bench/hostcost.cpp): kernels resolve to dummy handles, launches return at
// once, device memory is host memory.
#include <stdlib.h>
#include <string.h>

#include "../internal.h"

namespace tri {

int be_init(int *device) {
  *device = 0;
  return 0;
}
int be_resolve(int32_t kvariant, uint32_t, int32_t, void **fn) {
  *fn = reinterpret_cast<void *>(uintptr_t(0x1000) + uintptr_t(uint32_t(kvariant)));
  return 0;
}
int be_launch(void *, uint32_t, uint32_t, const void *, uint32_t, void *) { return 0; }
int be_upload(const void *host, uint64_t bytes, void **dev) {
  void *p = malloc(bytes);
  if (!p) return TRI_E_NOMEM;
  memcpy(p, host, bytes);
  *dev = p;
  return 0;
}
int be_alloc_zeroed(uint64_t bytes, void **dev) {
  *dev = calloc(1, bytes);
  return *dev ? 0 : TRI_E_NOMEM;
}
void be_free(void *dev) { free(dev); }
int be_compile(const char *, uint64_t, void **, uint64_t *) { return TRI_E_RUNTIME; }
int be_load_code(const void *, uint64_t, void **, void **) { return TRI_E_RUNTIME; }
void be_unload(void *) {}
int be_capture_begin(void **) { return TRI_E_RUNTIME; }
int be_capture_end(void *, void **) { return TRI_E_RUNTIME; }
int be_graph_launch(void *, void *) { return TRI_E_RUNTIME; }
void be_graph_destroy(void *) {}
int be_scratch(uint64_t, void *, void **) { return TRI_E_NOMEM; }
void be_scratch_free(void *) {}
int be_timer_create(uint32_t, void **, void **) { return TRI_E_RUNTIME; }
int be_timer_record(void *, uint32_t) { return TRI_E_RUNTIME; }
int be_timer_elapsed(void *, uint32_t, uint32_t, float *) { return TRI_E_RUNTIME; }
void be_timer_destroy(void *) {}
void be_arch(char *out, uint32_t cap) {
  if (cap) out[0] = '\0';
}
// resident argument blocks: host tables stand in for the device's
int be_resident_table(int, uint32_t family, uint32_t dtype, void **table) {
  static ResidentBlock tables[kResFamilies][2][kResidentSlots];
  const bool ok = family < kResFamilies && dtype <= 1;
  *table = ok ? tables[family][dtype] : nullptr;
  return ok ? 0 : TRI_E_RUNTIME;
}
int be_resolve_resident(int32_t, uint32_t, int32_t, void **fn) {
  *fn = reinterpret_cast<void *>(uintptr_t(0x2000));
  return 0;
}
int be_resident_write(int, void *dst, const void *src, uint32_t bytes) {
  memcpy(dst, src, bytes);
  return 0;
}
int be_launch_resident(void *, uint32_t, uint32_t, uint32_t, void *) { return 0; }
int be_stream_capturing(void *) { return 0; }
void be_device_sync(int) {}
int be_noalloc_scratch(int, void **ptr) {
  static uint64_t words[kNoAllocScratchWords];
  *ptr = words;
  return 0;
}

}  // namespace tri

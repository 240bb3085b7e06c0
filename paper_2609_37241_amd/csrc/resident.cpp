// Resident argument blocks (TRI_CACHE_RESIDENT_ARGS).
//
// Not in the paper: it takes away the per-launch placement of kernel
// arguments, part of the per-call launch cost the paper measures (Sec. 2.3).
// Each device has one table of kResidentSlots blocks per kernel family and
// dtype; its slots form a process-wide pool. A cache holds the blocks it has
// written (host copies, so that a call is matched without reading device
// memory) and hands each back to the pool when it is destroyed, after the
// device has finished its work. A held block is never rewritten: a launch
// that reads slot s always finds the block it was issued for.
#include <string.h>

#include <mutex>

#include "internal.h"

namespace tri {
namespace {

constexpr int kMaxDevices = 64;
static_assert(kResidentSlots <= 64, "the pool keeps one bit per slot");
std::mutex g_pool_mu;
uint64_t g_pool_used[kMaxDevices][kResFamilies][2];   // bit s: slot s is held by a cache

bool pool_index_ok(int device, uint32_t fam, uint32_t dt) {
  return device >= 0 && device < kMaxDevices && fam < kResFamilies && dt <= 1;
}

// The lowest free slot below `limit`, or -1.
int32_t pool_claim(int device, uint32_t fam, uint32_t dt, uint32_t limit) {
  if (!pool_index_ok(device, fam, dt)) return -1;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  uint64_t &used = g_pool_used[device][fam][dt];
  for (uint32_t s = 0; s < limit && s < kResidentSlots; ++s) {
    if (!((used >> s) & 1u)) {
      used |= uint64_t(1) << s;
      return int32_t(s);
    }
  }
  return -1;
}

void pool_release(int device, uint32_t fam, uint32_t dt, uint32_t s) {
  if (!pool_index_ok(device, fam, dt) || s >= kResidentSlots) return;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  g_pool_used[device][fam][dt] &= ~(uint64_t(1) << s);
}

inline bool same_block(const ResidentBlock &h, const void *args, uint32_t size, uint32_t grid) {
  return h.grid == grid && h.size == size && memcmp(h.args, args, size) == 0;
}

inline ResidentBlock *held_of(tri_cache *c, uint32_t fam, uint32_t dt) {
  return c->held + (size_t(fam) * 2 + dt) * kResidentSlots;
}

}  // namespace

int32_t resident_slot(tri_cache *c, uint32_t fam, uint32_t dt, const void *args, uint32_t size,
                      uint32_t grid, void *stream, uint32_t limit) {
  if (fam >= kResFamilies || dt > 1 || !c->rtable[fam][dt] || !c->held ||
      size > kResidentArgsMax)
    return -1;
  ResidentBlock *h = held_of(c, fam, dt);
  const uint32_t n = c->n_held[fam][dt];
  // The last match first, then the blocks after it: the layers of a decode
  // step come round in the order they were first seen.
  // A held block's grid is part of it, so its slot is below the limit its
  // launches have.
  for (uint32_t i = 0, j = c->last_held[fam][dt]; i < n; ++i, j = j + 1 == n ? 0 : j + 1) {
    if (same_block(h[j], args, size, grid)) {
      c->last_held[fam][dt] = j;
      return int32_t(h[j].tag - kResidentTag);
    }
  }
  // A new block: written synchronously, so no launch is enqueued ahead of
  // it; never while the caller's stream is captured (the copy is no part of
  // the caller's graph).
  if (n >= kResidentSlots || be_stream_capturing(stream) != 0) return -1;
  const int32_t s = pool_claim(c->device, fam, dt, limit);
  if (s < 0) return -1;
  ResidentBlock b;
  memset(&b, 0, sizeof b);
  memcpy(b.args, args, size);
  b.grid = grid;
  b.tag = kResidentTag + uint32_t(s);
  b.size = size;
  char *dst = static_cast<char *>(c->rtable[fam][dt]) + size_t(s) * sizeof b;
  if (be_resident_write(c->device, dst, &b, uint32_t(sizeof b)) != 0) {
    pool_release(c->device, fam, dt, uint32_t(s));
    return -1;
  }
  h[n] = b;
  c->n_held[fam][dt] = n + 1;
  c->last_held[fam][dt] = n;
  return s;
}

void resident_release_all(tri_cache *c) {
  if (!c->held) return;
  bool any = false;
  for (uint32_t fam = 0; fam < kResFamilies; ++fam)
    any = any || c->n_held[fam][0] || c->n_held[fam][1];
  if (!any) return;
  // no launch that reads one of these slots may still be in flight when
  // another cache rewrites it
  be_device_sync(c->device);
  for (uint32_t fam = 0; fam < kResFamilies; ++fam) {
    for (uint32_t dt = 0; dt < 2; ++dt) {
      const ResidentBlock *h = held_of(c, fam, dt);
      for (uint32_t i = 0; i < c->n_held[fam][dt]; ++i)
        pool_release(c->device, fam, dt, h[i].tag - kResidentTag);
      c->n_held[fam][dt] = 0;
      c->last_held[fam][dt] = 0;
    }
  }
}

}  // namespace tri

// Resident argument blocks of fused-chain launches (TRI_CACHE_RESIDENT_ARGS).
//
// Not in the paper: it takes away the per-launch placement of kernel
// arguments, part of the per-call launch cost the paper measures (Sec. 2.3).
// Each device has one table of kResidentSlots blocks per dtype; its slots
// form a process-wide pool. A cache holds the blocks it has written (host
// copies, so that a call is matched without reading device memory) and
// hands each back to the pool when it is destroyed, after the device has
// finished its work. A held block is never rewritten: a launch that reads
// slot s always finds the block it was issued for.
#include <string.h>

#include <mutex>

#include "internal.h"

namespace tri {
namespace {

constexpr int kMaxDevices = 64;
static_assert(kResidentSlots <= 64, "the pool keeps one bit per slot");
std::mutex g_pool_mu;
uint64_t g_pool_used[kMaxDevices][2];   // bit s: slot s is held by a cache

int32_t pool_claim(int device, uint32_t dt) {
  if (device < 0 || device >= kMaxDevices || dt > 1) return -1;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  for (uint32_t s = 0; s < kResidentSlots; ++s) {
    if (!((g_pool_used[device][dt] >> s) & 1u)) {
      g_pool_used[device][dt] |= uint64_t(1) << s;
      return int32_t(s);
    }
  }
  return -1;
}

void pool_release(int device, uint32_t dt, uint32_t s) {
  if (device < 0 || device >= kMaxDevices || dt > 1 || s >= kResidentSlots) return;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  g_pool_used[device][dt] &= ~(uint64_t(1) << s);
}

inline bool same_block(const ResidentChain &h, const ChainArgs &a, uint32_t grid) {
  return h.grid == grid && memcmp(&h.a, &a, sizeof a) == 0;
}

}  // namespace

int32_t resident_slot(tri_cache *c, uint32_t dt, const ChainArgs &a, uint32_t grid,
                      void *stream) {
  if (dt > 1 || !c->rtable[dt] || !c->held) return -1;
  ResidentChain *h = c->held + size_t(dt) * kResidentSlots;
  const uint32_t n = c->n_held[dt];
  // The last match first, then the blocks after it: the layers of a decode
  // step come round in the order they were first seen.
  for (uint32_t i = 0, j = c->last_held[dt]; i < n; ++i, j = j + 1 == n ? 0 : j + 1) {
    if (same_block(h[j], a, grid)) {
      c->last_held[dt] = j;
      return int32_t(h[j].tag - kResidentTag);
    }
  }
  // A new block: written synchronously, so no launch is enqueued ahead of
  // it; never while the caller's stream is captured (the copy is no part of
  // the caller's graph).
  if (n >= kResidentSlots || be_stream_capturing(stream) != 0) return -1;
  const int32_t s = pool_claim(c->device, dt);
  if (s < 0) return -1;
  ResidentChain b;
  memset(&b, 0, sizeof b);
  b.a = a;
  b.grid = grid;
  b.tag = kResidentTag + uint32_t(s);
  char *dst = static_cast<char *>(c->rtable[dt]) + size_t(s) * sizeof b;
  if (be_resident_write(c->device, dst, &b, uint32_t(sizeof b)) != 0) {
    pool_release(c->device, dt, uint32_t(s));
    return -1;
  }
  h[n] = b;
  c->n_held[dt] = n + 1;
  c->last_held[dt] = n;
  return s;
}

void resident_release_all(tri_cache *c) {
  if (!c->held || (c->n_held[0] == 0 && c->n_held[1] == 0)) return;
  // no launch that reads one of these slots may still be in flight when
  // another cache rewrites it
  be_device_sync(c->device);
  for (uint32_t dt = 0; dt < 2; ++dt) {
    const ResidentChain *h = c->held + size_t(dt) * kResidentSlots;
    for (uint32_t i = 0; i < c->n_held[dt]; ++i)
      pool_release(c->device, dt, h[i].tag - kResidentTag);
    c->n_held[dt] = 0;
    c->last_held[dt] = 0;
  }
}

}  // namespace tri

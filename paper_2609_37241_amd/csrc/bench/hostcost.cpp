// Host cost of one cache hit, step by step, on the CPU: the entry points'
// own source is compiled into this benchmark (its internal steps are not
// exported) over a backend whose launch does nothing, so the figures are
// the library's work alone; the HIP launch itself is what the benchmark's
// native latency loops add on top.
//
// Steps of a decode-chain hit (the Llama-7B 1-token shapes): argument
// validation, guard key packing, version lookup (the op's last key, the
// key memo, and Algorithm 1's scan at n versions), kernel argument fill
// and launch call, and the whole entry call.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <vector>

#include "../api.cpp"

using namespace tri;

namespace {

volatile uint64_t g_sink;
// The arguments are read through volatile pointers, so no step's work on
// them can be hoisted out of the timing loops.
const tri_chain_args *volatile g_pa;
const tri_chain_args *volatile g_pb;

// Median over `rounds` of the mean nanoseconds of one of `n` calls of f.
template <class F>
double ns_per(F f, int n, int rounds = 7) {
  std::vector<double> v;
  for (int r = 0; r < rounds; ++r) {
    const auto t0 = std::chrono::steady_clock::now();
    for (int i = 0; i < n; ++i) f(i);
    const auto t1 = std::chrono::steady_clock::now();
    v.push_back(std::chrono::duration<double, std::nano>(t1 - t0).count() / n);
  }
  std::sort(v.begin(), v.end());
  return v[v.size() / 2];
}

// The 1-token Llama-7B chain: device-like addresses (16-byte aligned).
tri_chain_args chain_args(int64_t I) {
  tri_chain_args a;
  memset(&a, 0, sizeof a);
  const uintptr_t base = uintptr_t(1) << 40;
  auto at = [&](int i) { return reinterpret_cast<void *>(base + uintptr_t(i) * (uintptr_t(1) << 28)); };
  a.dtype = TRI_BF16;
  a.nq = 32, a.nk = 32, a.hd = 128;
  a.T = 1, a.H = 4096, a.I = I;
  a.eps = 1e-6f, a.base = 10000.0f;
  a.x = at(0), a.x_rs = 4096;
  a.res = at(1), a.res_rs = 4096;
  a.w = at(2);
  a.y = at(3), a.y_rs = 4096;
  a.res_out = at(4), a.ro_rs = 4096;
  a.q = at(5), a.q_ts = 32 * 128;
  a.k = at(6), a.k_ts = 32 * 128;
  a.pos = at(7);
  a.gate = at(8), a.g_rs = I;
  a.up = at(9), a.u_rs = I;
  a.out = at(10), a.o_rs = I;
  return a;
}

}  // namespace

extern "C" {

// out[0..5]: ns per hit of validation, key packing, lookup on the op's last
// key, lookup through the key memo, argument fill + launch call, the whole
// entry call; then for each n in ns[0..nn): out[6 + i] = ns of Algorithm 1's
// scan to the last of n versions (no memo). Returns 0, or -1 on failure.
int trib_hostcost(const int32_t *ns, int32_t nn, double *out) {
  const int N = 200000;
  tri_cache *c = nullptr;
  if (tri_spec_cache_create(&c, kMaxCapacity, TRI_CACHE_AUTO_INSTALL) != TRI_OK) return -1;
  tri_chain_args a = chain_args(11008), b = chain_args(11016);
  if (tri_decode_chain(c, &a, nullptr) != TRI_OK || tri_decode_chain(c, &b, nullptr) != TRI_OK)
    return -1;
  Key ka, kb;
  chain_check(&a, &ka);
  chain_check(&b, &kb);
  g_pa = &a;
  g_pb = &b;

  // key packing alone (the flags, the packed words, the RoPE words)
  const double key_ns = ns_per([&](int) {
    const tri_chain_args &x = *g_pa;
    const uint64_t es = 2;
    const unsigned fl =
        res_flags(es, x.x, x.x_rs, x.res, x.res_rs, x.w, x.y, x.y_rs, x.res_out, x.ro_rs, x.H) |
        (rope_flags(es, x.q, x.q_ts, x.k, x.k_ts, x.nq, x.nk, x.hd) << 2) |
        (sw_flags(es, x.gate, x.g_rs, x.up, x.u_rs, x.out, x.o_rs, x.I) << 4);
    Key k = make_key(TRI_OP_CHAIN, uint32_t(x.dtype), x.T, fl, 0, uint64_t(x.H), uint64_t(x.I),
                     uint64_t(x.hd), uint64_t(x.nq), uint64_t(x.nk));
    rope_key_words(k, x.hd, x.base, kRopePlain);
    g_sink += k.k0 ^ k.k1 ^ k.k2 ^ k.k3;
  }, N);
  // validation and key packing together (chain_check)
  const double check_ns = ns_per([&](int) {
    Key k;
    g_sink += uint64_t(chain_check(g_pa, &k)) + k.k0 + k.k1;
  }, N);
  const Key *volatile pka = &ka;
  const Key *volatile pkb = &kb;
  const double last_ns = ns_per([&](int) {
    g_sink += uint64_t(find_version(c, TRI_OP_CHAIN, *pka));
  }, N);
  // alternating keys: the op's last key never matches, the memo does
  const double memo_ns = ns_per([&](int i) {
    g_sink += uint64_t(find_version(c, TRI_OP_CHAIN, (i & 1) ? *pkb : *pka));
  }, N);
  const int32_t vi = find_version(c, TRI_OP_CHAIN, ka);
  const double launch_ns = ns_per([&](int) {
    tri_launch_rec l[3];
    int n = 0;
    g_sink += uint64_t(chain_launch(c, c->versions[vi], *g_pa, nullptr, l, &n)) + l[0].grid_x;
  }, N);
  const double entry_ns = ns_per([&](int) { g_sink += uint64_t(tri_decode_chain(c, g_pa, nullptr)); }, N);
  out[0] = check_ns - key_ns;
  out[1] = key_ns;
  out[2] = last_ns;
  out[3] = memo_ns;
  out[4] = launch_ns;
  out[5] = entry_ns;
  tri_spec_cache_destroy(c);

  // Algorithm 1's scan to the last of n versions: chains differing in I
  for (int32_t j = 0; j < nn; ++j) {
    const int32_t n = ns[j];
    if (n < 1 || uint32_t(n) > kMaxCapacity) return -1;
    tri_cache *s = nullptr;
    if (tri_spec_cache_create(&s, kMaxCapacity, 0) != TRI_OK) return -1;
    Key last{};
    for (int32_t i = 0; i < n; ++i) {
      tri_chain_args x = chain_args(11008 + 8 * int64_t(i));
      Key k;
      chain_check(&x, &k);
      if (install_key(s, k) != TRI_OK) return -1;
      last = k;
    }
    const int reps = n >= 1024 ? 2000 : 20000;
    const Key *volatile pk = &last;
    out[6 + j] = ns_per([&](int) { g_sink += uint64_t(scan_versions(s, *pk)); }, reps);
    tri_spec_cache_destroy(s);
  }
  return 0;
}

// Entry calls on a cache with resident argument blocks (the 1-token chain):
// out[0] ns per call with one held block; out[1] ns per call stepping
// through 40 held blocks in order (the next layer's block is the one after
// the last match); out[2] ns per call alternating between the first and the
// last of the 40 (the longest search). Returns 0, or -1 on failure.
int trib_hostcost_resident(double *out) {
  const int N = 200000;
  tri_cache *c = nullptr;
  if (tri_spec_cache_create(&c, kMaxCapacity, TRI_CACHE_AUTO_INSTALL | TRI_CACHE_RESIDENT_ARGS) !=
      TRI_OK)
    return -1;
  std::vector<tri_chain_args> layers(kResidentSlots);
  for (uint32_t i = 0; i < kResidentSlots; ++i) {
    layers[i] = chain_args(11008);
    layers[i].x = static_cast<char *>(const_cast<void *>(layers[i].x)) + 4096 * i;
    if (tri_decode_chain(c, &layers[i], nullptr) != TRI_OK) return -1;
  }
  tri_resident_info info;
  if (tri_spec_resident_info(c, &info) != TRI_OK || info.held != kResidentSlots) return -1;
  const tri_chain_args *volatile pl = layers.data();
  out[0] = ns_per([&](int) { g_sink += uint64_t(tri_decode_chain(c, pl, nullptr)); }, N);
  out[1] = ns_per([&](int i) {
    g_sink += uint64_t(tri_decode_chain(c, pl + (i % kResidentSlots), nullptr));
  }, N);
  out[2] = ns_per([&](int i) {
    g_sink += uint64_t(tri_decode_chain(c, pl + ((i & 1) ? kResidentSlots - 1 : 0), nullptr));
  }, N);
  if (tri_spec_resident_info(c, &info) != TRI_OK || info.held != kResidentSlots) return -1;
  tri_spec_cache_destroy(c);
  return 0;
}

}  // extern "C"

// Native timing loops for the benchmark: per-call latency with no Python
// between the clock reads and the entry call.
//
// E2E latency of one call = steady_clock around {entry call; stream sync};
// host latency = the clock read right after the entry call returns. The
// empty-kernel yardstick runs the identical loop around tri_launch_empty.
#include <hip/hip_runtime.h>

#include <chrono>

#include "tri.h"

namespace {

using Clock = std::chrono::steady_clock;

inline double us_between(Clock::time_point a, Clock::time_point b) {
  return std::chrono::duration<double, std::micro>(b - a).count();
}

// mode 0: tri_decode_chain(args); mode 1: tri_launch_empty.
inline int one_call(tri_cache *c, int mode, const tri_chain_args *args, void *stream) {
  return mode == 0 ? int(tri_decode_chain(c, args, stream)) : int(tri_launch_empty(c, stream));
}

}  // namespace

extern "C" {

// n_warm untimed calls, then n timed calls, each synchronised. Writes n
// samples to e2e_us and host_us. Returns 0, or the first failing status.
int trib_latency(tri_cache *c, int mode, const tri_chain_args *args, void *stream, int n_warm,
                 int n, double *e2e_us, double *host_us) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int i = 0; i < n_warm; ++i) {
    const int st = one_call(c, mode, args, stream);
    if (st != 0) return st;
    if (hipStreamSynchronize(s) != hipSuccess) return TRI_E_RUNTIME;
  }
  for (int i = 0; i < n; ++i) {
    const Clock::time_point t0 = Clock::now();
    const int st = one_call(c, mode, args, stream);
    const Clock::time_point t1 = Clock::now();
    if (hipStreamSynchronize(s) != hipSuccess) return TRI_E_RUNTIME;
    const Clock::time_point t2 = Clock::now();
    if (st != 0) return st;
    e2e_us[i] = us_between(t0, t2);
    host_us[i] = us_between(t0, t1);
  }
  return 0;
}

// n back-to-back calls and one synchronisation: the pipelined issue rate.
int trib_issue(tri_cache *c, int mode, const tri_chain_args *args, void *stream, int n,
               double *total_us) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipStreamSynchronize(s) != hipSuccess) return TRI_E_RUNTIME;
  const Clock::time_point t0 = Clock::now();
  for (int i = 0; i < n; ++i) {
    const int st = one_call(c, mode, args, stream);
    if (st != 0) return st;
  }
  if (hipStreamSynchronize(s) != hipSuccess) return TRI_E_RUNTIME;
  *total_us = us_between(t0, Clock::now());
  return 0;
}

// Several chains per step: mode 0 issues ONE tri_decode_chain_layers call
// over layers[0 .. n_layers), mode 1 issues n_layers tri_decode_chain calls;
// either way one stream synchronisation ends the step. n_warm untimed steps,
// then n timed ones into e2e_us. Returns 0 or the first failing status.
int trib_layers(tri_cache *c, int mode, const tri_chain_args *layers, int n_layers, void *stream,
                int n_warm, int n, double *e2e_us) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int i = 0; i < n_warm + n; ++i) {
    const Clock::time_point t0 = Clock::now();
    int st = 0;
    if (mode == 0) {
      st = tri_decode_chain_layers(c, layers, uint32_t(n_layers), stream);
    } else {
      for (int l = 0; l < n_layers && st == 0; ++l) st = tri_decode_chain(c, layers + l, stream);
    }
    if (hipStreamSynchronize(s) != hipSuccess) return TRI_E_RUNTIME;
    if (st != 0) return st;
    if (i >= n_warm) e2e_us[i - n_warm] = us_between(t0, Clock::now());
  }
  return 0;
}

// The mixed-shape stream: calls[i] in order, each synchronised. A MISS is
// handled the way a caller of the library handles it (install the missed key,
// call again); missed[i] = 1 marks those calls, whose e2e_us then covers
// miss + install + retry. Returns 0 or the first failing status.
int trib_stream(tri_cache *c, const tri_chain_args *calls, int n, void *stream,
                double *e2e_us, int *missed) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int i = 0; i < n; ++i) {
    const Clock::time_point t0 = Clock::now();
    int st = tri_decode_chain(c, calls + i, stream);
    missed[i] = 0;
    if (st == TRI_MISS) {
      missed[i] = 1;
      st = tri_spec_install_last_miss(c, nullptr);
      if (st == TRI_OK) st = tri_decode_chain(c, calls + i, stream);
    }
    if (hipStreamSynchronize(s) != hipSuccess) return TRI_E_RUNTIME;
    e2e_us[i] = us_between(t0, Clock::now());
    if (st != TRI_OK) return st;
  }
  return 0;
}

}  // extern "C"

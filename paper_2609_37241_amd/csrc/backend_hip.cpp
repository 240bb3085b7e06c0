// HIP launch backend.
//
// Kernels are compiled into this library for gfx950. At install a version's
// kernels are resolved once to hipFunction_t handles (hipGetFuncBySymbol);
// each hit is a single hipModuleLaunchKernel of that handle with a pointer to
// the argument block on the caller's stream -- no symbol lookup, no
// per-argument marshalling, no device query on the hit path.
#include <hip/hip_runtime.h>
#include <hip/hiprtc.h>

#include <stdio.h>
#include <stdlib.h>

#include <mutex>

#include "internal.h"

namespace tri {

const void *rn_kernel(int32_t variant, uint32_t dtype, int32_t res);
const void *rope_kernel(int32_t variant, uint32_t dtype);
const void *sw_kernel(int32_t variant, uint32_t dtype);
const void *chain_kernel_f32(int32_t sub);
const void *chain_kernel_bf16(int32_t sub);
const void *empty_kernel();
const void *elt_kernel(int32_t variant, uint32_t dtype, int32_t op);
const void *emb_kernel(int32_t variant, uint32_t dtype);
const void *rn_kernel_resident(int32_t variant, uint32_t dtype, int32_t res);
const void *rope_kernel_resident(int32_t variant, uint32_t dtype);
const void *sw_kernel_resident(int32_t variant, uint32_t dtype);
const void *chain_kernel_resident_f32(int32_t sub);
const void *chain_kernel_resident_bf16(int32_t sub);
const void *elt_kernel_resident(int32_t variant, uint32_t dtype, int32_t op);
const void *emb_kernel_resident(int32_t variant, uint32_t dtype);
const void *resident_symbol_chain_f32();
const void *resident_symbol_chain_bf16();
const void *resident_symbol_norm();
const void *resident_symbol_rope();
const void *resident_symbol_swiglu();
const void *resident_symbol_elt();
const void *resident_symbol_emb();
int resident_check();

int be_init(int *device) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n < 1) return TRI_E_RUNTIME;
  if (hipGetDevice(device) != hipSuccess) return TRI_E_RUNTIME;
  return 0;
}

int be_resolve(int32_t kvariant, uint32_t dtype, int32_t ksub, void **fn) {
  const void *sym = nullptr;
  if (kvariant >= RN_SCALAR && kvariant <= RN_SPLIT)
    sym = rn_kernel(kvariant, dtype, ksub);
  else if (kvariant >= ROPE_SCALAR && kvariant <= ROPE_QKN_VEC_I)
    sym = rope_kernel(kvariant, dtype);
  else if (kvariant >= SW_SCALAR && kvariant <= SW_ROWS)
    sym = sw_kernel(kvariant, dtype);
  else if (kvariant == CH_FUSED)
    sym = dtype == TRI_F32 ? chain_kernel_f32(ksub) : chain_kernel_bf16(ksub);
  else if (kvariant >= ELT_SCALAR && kvariant <= ELT_ROWS)
    sym = elt_kernel(kvariant, dtype, ksub);
  else if (kvariant == EMB_SCALAR || kvariant == EMB_VEC)
    sym = emb_kernel(kvariant, dtype);
  else if (kvariant == EMPTY)
    sym = empty_kernel();
  if (!sym) return TRI_E_RUNTIME;
  hipFunction_t f = nullptr;
  if (hipGetFuncBySymbol(&f, sym) != hipSuccess || !f) return TRI_E_RUNTIME;
  *fn = reinterpret_cast<void *>(f);
  return 0;
}

int be_launch(void *fn, uint32_t grid, uint32_t block, const void *args, uint32_t,
              void *stream) {
  // The kernels take one by-value struct: the single parameter pointer
  // points at it (the runtime copies args_size bytes from the kernel's
  // parameter metadata).
  void *params[1] = {const_cast<void *>(args)};
  const hipError_t e =
      hipModuleLaunchKernel(reinterpret_cast<hipFunction_t>(fn), grid, 1, 1, block, 1, 1, 0,
                            reinterpret_cast<hipStream_t>(stream), args ? params : nullptr, nullptr);
  return e == hipSuccess ? 0 : -1;
}

// ---- resident argument blocks ----------------------------------------------------------
namespace {
constexpr int kMaxDevices = 64;
std::mutex g_res_mu;
int g_res_check[kMaxDevices];             // 0: not checked; 1: passed; -1: failed
hipStream_t g_res_stream[kMaxDevices];    // private copy stream per device
// device addresses of the tables, per device: [family][dtype]
void *g_res_table[kMaxDevices][kResFamilies][2];

// The table symbol of a family and dtype and the block offset into it: the
// chain has a table per dtype (one per kernel file), the other families one
// dtype-major table.
const void *table_symbol(uint32_t fam, uint32_t dt, uint32_t *first) {
  *first = 0;
  switch (fam) {
    case kResChain: return dt == TRI_F32 ? resident_symbol_chain_f32() : resident_symbol_chain_bf16();
    case kResNorm: *first = dt * kResidentSlots; return resident_symbol_norm();
    case kResRope: *first = dt * kResidentSlots; return resident_symbol_rope();
    case kResSwiglu: *first = dt * kResidentSlots; return resident_symbol_swiglu();
    case kResElt: *first = dt * kResidentSlots; return resident_symbol_elt();
    case kResEmb: *first = dt * kResidentSlots; return resident_symbol_emb();
    default: return nullptr;
  }
}
}  // namespace

// The device's table for a family and dtype, once the device has passed the
// check of the LDS channel (made once per device, with it current).
int be_resident_table(int device, uint32_t family, uint32_t dtype, void **table) {
  *table = nullptr;
  if (device < 0 || device >= kMaxDevices || family >= kResFamilies || dtype > 1)
    return TRI_E_RUNTIME;
  std::lock_guard<std::mutex> lock(g_res_mu);
  if (g_res_check[device] == 0) g_res_check[device] = resident_check() == 0 ? 1 : -1;
  if (g_res_check[device] != 1) return TRI_E_RUNTIME;
  void *&t = g_res_table[device][family][dtype];
  if (!t) {
    uint32_t first = 0;
    const void *sym = table_symbol(family, dtype, &first);
    void *p = nullptr;
    if (!sym || hipGetSymbolAddress(&p, sym) != hipSuccess || !p) return TRI_E_RUNTIME;
    t = static_cast<char *>(p) + size_t(first) * sizeof(ResidentBlock);
  }
  *table = t;
  return 0;
}

int be_resolve_resident(int32_t kvariant, uint32_t dtype, int32_t ksub, void **fn) {
  const void *sym = nullptr;
  if (kvariant >= RN_SCALAR && kvariant <= RN_SPLIT)
    sym = rn_kernel_resident(kvariant, dtype, ksub);
  else if (kvariant >= ROPE_SCALAR && kvariant <= ROPE_QKN_VEC_I)
    sym = rope_kernel_resident(kvariant, dtype);
  else if (kvariant >= SW_SCALAR && kvariant <= SW_ROWS)
    sym = sw_kernel_resident(kvariant, dtype);
  else if (kvariant == CH_FUSED)
    sym = dtype == TRI_F32 ? chain_kernel_resident_f32(ksub) : chain_kernel_resident_bf16(ksub);
  else if (kvariant >= ELT_SCALAR && kvariant <= ELT_ROWS)
    sym = elt_kernel_resident(kvariant, dtype, ksub);
  else if (kvariant == EMB_SCALAR || kvariant == EMB_VEC)
    sym = emb_kernel_resident(kvariant, dtype);
  if (!sym) return TRI_E_RUNTIME;
  hipFunction_t f = nullptr;
  if (hipGetFuncBySymbol(&f, sym) != hipSuccess || !f) return TRI_E_RUNTIME;
  *fn = reinterpret_cast<void *>(f);
  return 0;
}

// A copy into `device`'s table on that device's private stream, complete
// when this returns (the caller's streams are not touched).
int be_resident_write(int device, void *dst, const void *src, uint32_t bytes) {
  if (device < 0 || device >= kMaxDevices) return TRI_E_RUNTIME;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return TRI_E_RUNTIME;
  if (cur != device && hipSetDevice(device) != hipSuccess) return TRI_E_RUNTIME;
  int st = 0;
  {
    std::lock_guard<std::mutex> lock(g_res_mu);
    hipStream_t &s = g_res_stream[device];
    if (!s && hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) {
      s = nullptr;
      st = TRI_E_RUNTIME;
    }
    if (st == 0 && (hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
                    hipStreamSynchronize(s) != hipSuccess))
      st = TRI_E_RUNTIME;
  }
  if (cur != device) (void)hipSetDevice(cur);
  return st;
}

// No kernel arguments: the slot travels as the dynamic LDS size.
int be_launch_resident(void *fn, uint32_t grid, uint32_t block, uint32_t slot, void *stream) {
  if (slot >= kResidentSlots) return -1;
  const hipError_t e = hipModuleLaunchKernel(reinterpret_cast<hipFunction_t>(fn), grid, 1, 1,
                                             block, 1, 1, slot * kLdsGranule,
                                             reinterpret_cast<hipStream_t>(stream), nullptr,
                                             nullptr);
  return e == hipSuccess ? 0 : -1;
}

int be_stream_capturing(void *stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(reinterpret_cast<hipStream_t>(stream), &cs) != hipSuccess) return 1;
  return cs == hipStreamCaptureStatusNone ? 0 : 1;
}

void be_device_sync(int device) {
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return;
  if (cur != device && hipSetDevice(device) != hipSuccess) return;
  (void)hipDeviceSynchronize();
  if (cur != device) (void)hipSetDevice(cur);
}

int be_upload(const void *host, uint64_t bytes, void **dev) {
  void *p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess) return TRI_E_NOMEM;
  if (hipMemcpy(p, host, bytes, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(p);
    return TRI_E_RUNTIME;
  }
  *dev = p;
  return 0;
}

// Zero-filled device memory, ready when this returns (a synchronous fill).
int be_alloc_zeroed(uint64_t bytes, void **dev) {
  void *p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess) return TRI_E_NOMEM;
  // the fill runs on the null stream: wait for it, so that no launch on
  // another stream can reach the memory first
  if (hipMemset(p, 0, bytes) != hipSuccess || hipStreamSynchronize(nullptr) != hipSuccess) {
    (void)hipFree(p);
    return TRI_E_RUNTIME;
  }
  *dev = p;
  return 0;
}

void be_free(void *dev) { (void)hipFree(dev); }

// hipRTC for gfx950 with the device flags of the precompiled kernels (no
// floating-point contraction, packed FP32 instructions off).
int be_compile(const char *src, uint64_t len, void **code, uint64_t *code_len) {
  (void)len;
  hiprtcProgram prog;
  if (hiprtcCreateProgram(&prog, src, "tri_jit.hip", 0, nullptr, nullptr) != HIPRTC_SUCCESS)
    return TRI_E_RUNTIME;
  const char *opts[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"};
  int st = 0;
  if (hiprtcCompileProgram(prog, int(sizeof opts / sizeof opts[0]), opts) != HIPRTC_SUCCESS) {
    st = TRI_E_RUNTIME;
  } else {
    size_t n = 0;
    void *buf = nullptr;
    if (hiprtcGetCodeSize(prog, &n) != HIPRTC_SUCCESS || n == 0 || !(buf = malloc(n))) {
      st = TRI_E_RUNTIME;
    } else if (hiprtcGetCode(prog, static_cast<char *>(buf)) != HIPRTC_SUCCESS) {
      free(buf);
      st = TRI_E_RUNTIME;
    } else {
      *code = buf;
      *code_len = n;
    }
  }
  (void)hiprtcDestroyProgram(&prog);
  return st;
}

// Load a code object and resolve its kernel.
int be_load_code(const void *code, uint64_t code_len, void **fn, void **module) {
  (void)code_len;
  hipModule_t mod = nullptr;
  if (hipModuleLoadData(&mod, code) != hipSuccess) return TRI_E_RUNTIME;
  hipFunction_t f = nullptr;
  if (hipModuleGetFunction(&f, mod, "tri_jit_kernel") != hipSuccess) {
    (void)hipModuleUnload(mod);
    return TRI_E_RUNTIME;
  }
  *fn = reinterpret_cast<void *>(f);
  *module = reinterpret_cast<void *>(mod);
  return 0;
}

void be_unload(void *module) { (void)hipModuleUnload(reinterpret_cast<hipModule_t>(module)); }

// Capture on a private non-blocking stream of default priority, in
// thread-local mode: only this thread's work on that stream is recorded.
int be_capture_begin(void **stream) {
  hipStream_t s = nullptr;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) return TRI_E_RUNTIME;
  if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess) {
    (void)hipStreamDestroy(s);
    return TRI_E_RUNTIME;
  }
  *stream = s;
  return 0;
}

int be_capture_end(void *stream, void **exec) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(s, &g);
  (void)hipStreamDestroy(s);
  if (e != hipSuccess || !g) return TRI_E_RUNTIME;
  hipGraphExec_t x = nullptr;
  const hipError_t ie = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (ie != hipSuccess) return TRI_E_RUNTIME;
  *exec = x;
  return 0;
}

int be_graph_launch(void *exec, void *stream) {
  return hipGraphLaunch(static_cast<hipGraphExec_t>(exec), static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? 0
             : TRI_E_RUNTIME;
}

void be_graph_destroy(void *exec) { (void)hipGraphExecDestroy(static_cast<hipGraphExec_t>(exec)); }

// ---- install-time tuning -------------------------------------------------------
// Zero-filled by a fill on the tuning stream, so the tuning calls that
// follow on that stream see zeros (positions 0: every RoPE table read is in
// range).
int be_scratch(uint64_t bytes, void *stream, void **dev) {
  void *p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess) return TRI_E_NOMEM;
  if (hipMemsetAsync(p, 0, bytes, static_cast<hipStream_t>(stream)) != hipSuccess) {
    (void)hipFree(p);
    return TRI_E_RUNTIME;
  }
  *dev = p;
  return 0;
}

void be_scratch_free(void *dev) { (void)hipFree(dev); }

namespace {
struct Timer {
  hipStream_t stream;
  uint32_t n;
  hipEvent_t ev[1];   // n events
};
}  // namespace

// A private non-blocking stream of default priority and n timing events.
int be_timer_create(uint32_t n_events, void **timer, void **stream) {
  Timer *t = static_cast<Timer *>(calloc(1, sizeof(Timer) + sizeof(hipEvent_t) * n_events));
  if (!t) return TRI_E_NOMEM;
  if (hipStreamCreateWithFlags(&t->stream, hipStreamNonBlocking) != hipSuccess) {
    free(t);
    return TRI_E_RUNTIME;
  }
  for (uint32_t i = 0; i < n_events; ++i) {
    if (hipEventCreate(&t->ev[i]) != hipSuccess) {
      t->n = i;
      be_timer_destroy(t);
      return TRI_E_RUNTIME;
    }
  }
  t->n = n_events;
  *timer = t;
  *stream = t->stream;
  return 0;
}

int be_timer_record(void *timer, uint32_t i) {
  Timer *t = static_cast<Timer *>(timer);
  if (i >= t->n) return TRI_E_INVALID;
  return hipEventRecord(t->ev[i], t->stream) == hipSuccess ? 0 : TRI_E_RUNTIME;
}

int be_timer_elapsed(void *timer, uint32_t i, uint32_t j, float *ms) {
  Timer *t = static_cast<Timer *>(timer);
  if (i >= t->n || j >= t->n) return TRI_E_INVALID;
  if (hipEventSynchronize(t->ev[j]) != hipSuccess) return TRI_E_RUNTIME;
  return hipEventElapsedTime(ms, t->ev[i], t->ev[j]) == hipSuccess ? 0 : TRI_E_RUNTIME;
}

void be_timer_destroy(void *timer) {
  Timer *t = static_cast<Timer *>(timer);
  (void)hipStreamSynchronize(t->stream);
  for (uint32_t i = 0; i < t->n; ++i) (void)hipEventDestroy(t->ev[i]);
  (void)hipStreamDestroy(t->stream);
  free(t);
}

void be_arch(char *out, uint32_t cap) {
  if (!cap) return;
  out[0] = '\0';
  int dev = 0;
  hipDeviceProp_t p;
  if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&p, dev) != hipSuccess) return;
  snprintf(out, cap, "%s", p.gcnArchName);
}

}  // namespace tri

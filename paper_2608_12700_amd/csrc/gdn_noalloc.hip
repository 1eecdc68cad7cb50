// gdn_fwd_noalloc: the forward with its workspace in a fixed, library-owned
// device array instead of a caller buffer, for callers that cannot allocate
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc).  It runs exactly gdn_fwd's kernels.
//
// The array `scratch` below is file-scope device memory: every GPU the library
// runs on holds its own copy, at its own address, until the process ends.  In
// host code its name is only a host-side stand-in, so host code never passes
// it to a kernel or a copy: on the first call on each device (that device
// current) its device address is looked up with hipGetSymbolAddress and kept,
// and only that address is used.
//
// Nothing in the forward's workspace needs to start at any value: every
// region (flags included) is written by the call before it is read, so the
// contents left by an earlier call are harmless.  Calls that overlap on one
// device share the array and race; serialise them (one stream, or events).
#include <hip/hip_runtime.h>

#include <mutex>

#include "gdn.h"

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[GDN_NOALLOC_SCRATCH_BYTES];

std::mutex g_lock;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (nullptr on failure).
void* scratch_of(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> guard(g_lock);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" gdn_status gdn_fwd_noalloc(const gdn_problem* p, const void* q, const void* k, const void* v,
                                      const float* g, const float* beta, const float* S0, void* o,
                                      float* S_T, float* chunk_states, void* stream) {
  try {
    if (!p) return GDN_ERR_NULL;
    if (gdn_num_chunks(p) < 0) return static_cast<gdn_status>(gdn_num_chunks(p));
    const size_t need = gdn_fwd_workspace_size(p);
    if (need > (size_t)GDN_NOALLOC_SCRATCH_BYTES) return GDN_ERR_TOO_LARGE;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return GDN_ERR_HIP;
    void* ws = scratch_of(dev);
    if (ws == nullptr) return GDN_ERR_HIP;
    return gdn_fwd(p, q, k, v, g, beta, S0, o, S_T, chunk_states, ws, (size_t)GDN_NOALLOC_SCRATCH_BYTES, stream);
  } catch (...) {
    return GDN_ERR_HIP;
  }
}

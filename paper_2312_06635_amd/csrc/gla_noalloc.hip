// gla_noalloc.hip -- gla_chunk_fwd_noalloc: the chunkwise forward with its
// workspace in a fixed device array owned by the library, for callers that
// cannot allocate (HIP graph capture, serving loops, harnesses that forbid
// hipMalloc).  It runs exactly the kernels of gla_chunk_fwd.
//
// The array lives in the code object: every GPU the library runs on holds its
// own copy, at its own address, until the process ends.  In host code the
// array's name is only a host-side stand-in for the symbol, so its device
// address is taken once per device with hipGetSymbolAddress (with that device
// current) and only that address is ever handed to kernels.  Nothing here
// allocates, frees or clears memory; the forward's kernels overwrite every
// byte of the workspace they later read, so the array's previous contents
// (the last call's) never matter.  Calls that overlap on one GPU share the
// array and race.
#include <mutex>

#include <hip/hip_runtime.h>

#include "gla.h"

#define GLA_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

constexpr size_t kScratchBytes = GLA_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_ptr[kMaxDevices];  // device address of `scratch` per device (nullptr: not yet taken)

// The current device's address of the scratch array, taken on first use.
gla_status scratch_ptr(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return GLA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GLA_ERR_HIP;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return GLA_OK;
}

}  // namespace

GLA_EXPORT gla_status gla_chunk_fwd_noalloc(const gla_problem *prob, const void *q, const void *k,
                                            const void *v, const void *log_alpha, const float *S0,
                                            void *o, float *S_T, void *stream) {
  if (!prob) return GLA_ERR_NULL;
  const size_t need = gla_workspace_bytes(prob, 0);
  // 0 bytes: an invalid problem (the forward's validation returns its error
  // before any HIP call) or one with nothing to compute
  if (need == 0) return gla_chunk_fwd(prob, q, k, v, log_alpha, S0, o, S_T, nullptr, 0, stream);
  if (need > kScratchBytes) return GLA_ERR_SCRATCH;
  void *ws = nullptr;
  const gla_status st = scratch_ptr(&ws);
  if (st != GLA_OK) return st;
  return gla_chunk_fwd(prob, q, k, v, log_alpha, S0, o, S_T, ws, kScratchBytes, stream);
}

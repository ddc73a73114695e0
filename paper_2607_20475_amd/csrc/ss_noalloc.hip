// ss_noalloc.hip -- ss_sample for callers that cannot allocate: the
// workspace is a fixed array in the library's own device memory.
//
// The array lives in this file's code object, so each GPU that loads the
// library holds its own copy until the process ends.  Host code never uses
// the array's name as a device address: the address of each device's copy
// is queried once per device, with that device current, and that pointer is
// what the kernels receive (exactly where ss_sample receives the caller's
// workspace).  Nothing in the workspace needs to start at any value: every
// call writes what it reads.  All calls on one GPU share its copy, so calls
// that overlap in time on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ss.h"

namespace {

static __device__ __align__(256) unsigned char scratch[SS_NOALLOC_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // per device: the device address of `scratch`

// Address of the current device's copy of `scratch` (queried on the first
// call made with that device current).  nullptr when the query fails.
void* scratch_ptr(ss_status* st) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    *st = SS_ERR_HIP;
    return nullptr;
  }
  if (dev >= kMaxDevices) {
    *st = SS_ERR_UNSUPPORTED;
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      *st = SS_ERR_HIP;
      return nullptr;
    }
    g_scratch[dev] = p;
  }
  *st = SS_OK;
  return g_scratch[dev];
}

}  // namespace

extern "C" ss_status ss_sample_noalloc(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max,
                                       int32_t* out_token, float* out_logprob, int32_t* out_idx, float* out_prob,
                                       int k_out, int32_t* flags, void* stream) {
  if (!p) return SS_ERR_INVALID_ARG;
  const size_t need = ss_workspace_bytes(SS_OP_SAMPLE, p->B, p->V, 0, k_max, dtype);
  if (need == 0) return SS_ERR_INVALID_ARG;
  if (need > (size_t)SS_NOALLOC_BYTES) return SS_ERR_WORKSPACE;
  ss_status st;
  void* ws = scratch_ptr(&st);
  if (!ws) return st;
  return ss_sample(logits, dtype, ld, p, k_max, out_token, out_logprob, out_idx, out_prob, k_out, flags, ws,
                   (size_t)SS_NOALLOC_BYTES, stream);
}

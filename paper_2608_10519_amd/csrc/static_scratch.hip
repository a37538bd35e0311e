// sparstar_score_blocks_static: the selector of sparstar_score_blocks with its
// scratch memory (the pooled blocks qbar and kbar, and the score matrix S when
// the caller does not take S as an output) held by the library, for callers
// that cannot allocate device memory.
//
// The scratch is one file-scope device array per GPU.  Its device address is
// looked up once per device, with that device current, on the first call made
// there, and kept; host code only ever passes that address on (the array's
// name denotes a host-side stand-in in host code).  The call itself allocates
// nothing: it validates its arguments on the host, then launches the same
// kernels as sparstar_score_blocks on the caller's stream.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include <mutex>

#include "../../include/sparstar.h"
#include "host_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[SPARSTAR_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, once looked up

// The current device's scratch address (looked up on its first use there).
int device_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  char msg[256];
  if (e != hipSuccess) {
    snprintf(msg, sizeof msg, "hipGetDevice: %s", hipGetErrorString(e));
    return sparstar::report_error(SPARSTAR_ERR_HIP, msg);
  }
  if (dev < 0 || dev >= kMaxDevices) {
    snprintf(msg, sizeof msg, "device %d is beyond the %d devices the static scratch serves", dev, kMaxDevices);
    return sparstar::report_error(SPARSTAR_ERR_UNSUPPORTED, msg);
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      snprintf(msg, sizeof msg, "hipGetSymbolAddress of the static scratch on device %d: %s", dev,
               e != hipSuccess ? hipGetErrorString(e) : "null address");
      return sparstar::report_error(SPARSTAR_ERR_HIP, msg);
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return SPARSTAR_OK;
}

}  // namespace

extern "C" int sparstar_score_blocks_static(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D,
                                            int block_size, const double* budget, int n_budget,
                                            const sparstar_range* keep, int n_keep, int32_t* kv_num_blocks,
                                            int32_t* kv_indices, int kv_stride, float* scores, void* stream) {
  // every argument, the scratch size included, is checked before any HIP call
  const size_t need = scores != nullptr ? sparstar::score_pooled_bytes(B, H, Lq, Lk, D, block_size)
                                        : sparstar_score_workspace_bytes(B, H, Lq, Lk, D, block_size);
  if (need > SPARSTAR_STATIC_SCRATCH_BYTES) {
    char msg[320];
    snprintf(msg, sizeof msg,
             "these sizes need %zu bytes of scratch%s, more than the %zu bytes the library holds per device",
             need, scores != nullptr ? "" : " (with S; passing `scores` keeps S out of it)",
             (size_t)SPARSTAR_STATIC_SCRATCH_BYTES);
    return sparstar::report_error(SPARSTAR_ERR_WORKSPACE, msg);
  }
  if (int rc = sparstar::score_blocks_internal(q, k, B, H, Lq, Lk, D, block_size, budget, n_budget, keep, n_keep,
                                               kv_num_blocks, kv_indices, kv_stride, scores, nullptr,
                                               SPARSTAR_STATIC_SCRATCH_BYTES, stream, true))
    return rc;
  if (Lq == 0) return SPARSTAR_OK;  // nothing to compute: no HIP call at all
  void* ws = nullptr;
  if (int rc = device_scratch(&ws)) return rc;
  return sparstar::score_blocks_internal(q, k, B, H, Lq, Lk, D, block_size, budget, n_budget, keep, n_keep,
                                         kv_num_blocks, kv_indices, kv_stride, scores, ws,
                                         SPARSTAR_STATIC_SCRATCH_BYTES, stream, false);
}

// Allocation-free variant of the verify pass for callers that cannot allocate
// device memory (code under stream capture, tight serving loops): the pass's
// workspace is a file-scope device array of a fixed size instead of a caller
// buffer. Every GPU the library runs on holds its own copy of the array from
// the first call on that GPU until the process ends; concurrent calls on one
// GPU share it and therefore race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/rksc.h"
#include "api_internal.h"
#include "status.h"

#define RKSC_EXPORT extern "C" __attribute__((visibility("default")))

// The verify pass's workspace for the allocation-free entry point. In host
// code this name is only a stand-in for the device array: its device address
// comes from hipGetSymbolAddress, per device, and only that address is used.
static __device__ __align__(256) unsigned char scratch[RKSC_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};   // device address of `scratch` on each device, once resolved

// The address of this device's copy of `scratch`, resolved once per device with
// that device current.
rksc_status scratch_of(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return rksc::fail(RKSC_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev,
                        hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return RKSC_OK;
}

}  // namespace

RKSC_EXPORT rksc_status rksc_verify_forward_noalloc(const rksc_weights* w, const rksc_prefix_kv* kv,
                                                    const int32_t* branch_tokens, int32_t n_branches,
                                                    int32_t branch_len, float tau, int32_t patience,
                                                    float* entropy, int32_t* exit_layer, float* hidden_last,
                                                    void* stream) {
  if (!w) return rksc::fail(RKSC_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!kv) return rksc::fail(RKSC_ERR_INVALID_ARGUMENT, "prefix_kv is NULL");
  // Size check first (host arithmetic only): larger passes are refused before any HIP call.
  size_t need = 0;
  const rksc_status sz = rksc::verify_workspace(&w->cfg, n_branches, branch_len, kv->n_prefix, &need);
  if (sz != RKSC_OK) return sz;
  if (need > (size_t)RKSC_NOALLOC_SCRATCH_BYTES)
    return rksc::fail(RKSC_ERR_WORKSPACE_TOO_SMALL,
                      "this pass needs %zu bytes of workspace; the allocation-free entry point has %zu "
                      "(use rksc_verify_forward with a caller workspace)",
                      need, (size_t)RKSC_NOALLOC_SCRATCH_BYTES);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return rksc::fail(RKSC_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return rksc::fail(RKSC_ERR_UNSUPPORTED, "device %d out of range", dev);
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev);
    if (e != hipSuccess) return rksc::fail(RKSC_ERR_HIP, "hipStreamGetDevice failed: %s", hipGetErrorString(e));
    if (sdev != dev)
      return rksc::fail(RKSC_ERR_INVALID_ARGUMENT, "the stream belongs to device %d but device %d is current",
                        (int)sdev, dev);
  }
  void* ws = nullptr;
  const rksc_status st = scratch_of(dev, &ws);
  if (st != RKSC_OK) return st;
  return rksc::verify_call(w, kv, branch_tokens, n_branches, branch_len, tau, patience, entropy, exit_layer,
                           hidden_last, ws, (size_t)RKSC_NOALLOC_SCRATCH_BYTES, stream);
}

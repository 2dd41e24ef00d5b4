// noalloc.cpp -- singa_conv_bwd_filter_noalloc: the filter gradient with its
// scratch (split-K partial tiles, the rewritten input and gradient staging)
// in a fixed device array the library owns, for callers that cannot allocate.
#include "singa_mi.h"

#include <hip/hip_runtime.h>

#include <mutex>

namespace {

// One copy per GPU the library runs on, held until the process ends.  In host
// code `scratch` names a host-side stand-in: the device address of each GPU's
// copy comes from hipGetSymbolAddress and is the only form passed to kernels.
static __device__ __align__(256) char scratch[SINGA_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

// The device address of this GPU's scratch array, looked up once per device
// (with that device current).
int scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return SINGA_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SINGA_ERR_HIP;
    g_addr[dev] = p;
  }
  *out = g_addr[dev];
  return SINGA_OK;
}

}  // namespace

extern "C" int singa_conv_bwd_filter_noalloc(singa_dtype dtype, singa_layout layout, const singa_shape4* x,
                                             const void* x_ptr, const singa_filter4* w, const singa_conv_desc* d,
                                             const void* dy_ptr, float* dw, float* db, int accumulate,
                                             singa_stream stream) {
  // the workspace the allocating call would take (with a bias column: never
  // less than without one); validation of shapes, dtype and layout happens
  // here and again in the call below, before anything is enqueued
  size_t need = 0;
  int rc = singa_conv_workspace_bytes(SINGA_OP_BWD_FILTER, dtype, layout, x, w, d, &need);
  if (rc != SINGA_OK) return rc;
  if (need > (size_t)SINGA_NOALLOC_SCRATCH_BYTES) return SINGA_ERR_SCRATCH;
  void* ws = nullptr;
  if (need > 0) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return SINGA_ERR_HIP;
    if (stream) {  // the stream must belong to the current device
      hipDevice_t sd = -1;
      if (hipStreamGetDevice((hipStream_t)stream, &sd) != hipSuccess) return SINGA_ERR_HIP;
      if ((int)sd != cur) return SINGA_ERR_UNSUPPORTED;
    }
    rc = scratch_address(cur, &ws);
    if (rc != SINGA_OK) return rc;
  }
  return singa_conv_bwd_filter(dtype, layout, x, x_ptr, w, d, dy_ptr, dw, db, accumulate, ws, need, stream);
}

// One MGN call (the forward of mgn_forward, without saved activations) whose
// device scratch is a file-scope device array instead of a caller workspace,
// for callers that cannot allocate device memory at call time.
//
// The array lives once per GPU in the loaded code object and is held until
// the process ends.  In host code its name is only a host-side stand-in, so
// its device address is taken once per device with hipGetSymbolAddress (with
// that device current) and only that address is passed to the kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.hpp"

namespace {

constexpr size_t kScratchBytes = (size_t)MGN_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this GPU's copy of the scratch array (looked up on the
// first call made with that device current).
int scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return mgn::fail(MGN_ERR_DEVICE, "mgn_forward_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return mgn::fail(MGN_ERR_DEVICE, "mgn_forward_noalloc: device %d unsupported", dev);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return mgn::fail(MGN_ERR_DEVICE, "mgn_forward_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return MGN_OK;
}

}  // namespace

extern "C" int mgn_forward_noalloc(mgn_ctx* ctx, const mgn_dgraph* g, const float* params, const float* node_in,
                                   const float* efeat, float* out, void* stream) {
  if (!ctx) return mgn::fail(MGN_ERR_ARG, "mgn_forward_noalloc: null ctx");
  // reject a context whose plan exceeds the array before touching the device
  const size_t need = mgn::ctx_workspace_bytes(ctx);
  if (need > kScratchBytes)
    return mgn::fail(MGN_ERR_WORKSPACE,
                     "mgn_forward_noalloc: the context plans %zu bytes of workspace, the static scratch holds %zu "
                     "(plan the context for fewer nodes / edges, or use mgn_forward)",
                     need, kScratchBytes);
  void* ws = nullptr;
  int rc = scratch_ptr(&ws);
  if (rc != MGN_OK) return rc;
  return mgn::forward_in_scratch(ctx, g, params, node_in, efeat, out, ws, kScratchBytes, stream);
}

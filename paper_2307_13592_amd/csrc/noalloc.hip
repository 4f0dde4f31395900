// mgn_forward_noalloc: mgn_forward with its workspace in a statically sized
// device array that the library owns (one copy per GPU), for callers that
// cannot allocate device memory.  Every step of the forward is the same
// launch sequence as mgn_forward's; only the workspace pointer differs.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "mgn_internal.h"

namespace {

// The workspace of mgn_forward_noalloc.  In host code this name is only a
// stand-in for the symbol: host code uses the device address that
// hipGetSymbolAddress returns for the current GPU (scratch_ptr below).
__device__ __align__(256) unsigned char scratch[MGN_NOALLOC_WS_MAX];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};  // device address of `scratch` on each GPU, once looked up

// Device address of `scratch` on the current GPU (looked up once per GPU,
// with that GPU current), or nullptr with `err` set.
void* scratch_ptr(std::string& err) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    err = std::string("hipGetDevice: ") + hipGetErrorString(e);
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    err = "device index " + std::to_string(dev) + " beyond the " + std::to_string(kMaxDevices) + " supported";
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      err = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
      return nullptr;
    }
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" mgn_status mgn_forward_noalloc(mgn_model* m, const mgn_graph* g, const float* node_feat,
                                          const float* edge_feat, const float* halo, float* out, mgn_stream stream) {
  if (!m) return mgn::set_error(nullptr, MGN_E_ARG, "mgn_forward_noalloc: model is NULL");
  if (mgn::timing_enabled(m))
    return mgn::set_error(m, MGN_E_STATE,
                          "mgn_forward_noalloc: launch timing is on (it creates HIP events); disable it first");
  size_t need = 0;
  mgn_status s = mgn_workspace_size(m, g, &need);
  if (s != MGN_OK) return s;
  if (need > (size_t)MGN_NOALLOC_WS_MAX)
    return mgn::set_error(m, MGN_E_NOMEM,
                          "mgn_forward_noalloc: this graph and plan need a workspace of " + std::to_string(need) +
                              " bytes, more than the " + std::to_string((size_t)MGN_NOALLOC_WS_MAX) +
                              " bytes of the static one (use mgn_forward with a caller workspace)");
  std::string err;
  void* ws = scratch_ptr(err);
  if (!ws) return mgn::set_error(m, MGN_E_HIP, "mgn_forward_noalloc: " + err);
  return mgn_forward(m, g, node_feat, edge_feat, halo, out, ws, (size_t)MGN_NOALLOC_WS_MAX, stream);
}

// nacl_evict without a caller workspace, for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops).  The
// score, select and compact kernels take their workspace from `scratch`, a
// fixed device array of NACL_NOALLOC_WORKSPACE_MAX bytes that every GPU the
// library runs on holds until the process ends.  Host code never passes the
// array's name to a kernel: the name is a host-side stand-in.  Its device
// address is taken once per device with hipGetSymbolAddress on the first
// call made with that device current, and kept.

#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/nacl.h"
#include "internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[NACL_NOALLOC_WORKSPACE_MAX];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's copy of `scratch`.
int scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return nacl::fail_status(NACL_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return nacl::fail_status(NACL_ERR_UNSUPPORTED, "device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return nacl::fail_status(NACL_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return NACL_OK;
}

}  // namespace

extern "C" int nacl_evict_noalloc(const nacl_problem* p, const void* q, const void* k, const void* v,
                                  int32_t C, int32_t Cr, int32_t sampling, uint64_t seed, uint32_t layer,
                                  float* scores, int32_t* keep_idx, void* k_out, void* v_out,
                                  uint32_t* health, void* stream) {
  const size_t need = nacl_workspace_bytes(p);
  // An invalid problem: nacl_evict's own checks report it, before any use
  // of the workspace.
  if (need == 0)
    return nacl_evict(p, q, k, v, C, Cr, sampling, seed, layer, scores, keep_idx, k_out, v_out, nullptr,
                      (size_t)NACL_NOALLOC_WORKSPACE_MAX, stream);
  if (need > (size_t)NACL_NOALLOC_WORKSPACE_MAX)
    return nacl::fail_status(NACL_ERR_UNSUPPORTED, "the problem needs %zu bytes of workspace; the built-in scratch holds %zu",
                             need, (size_t)NACL_NOALLOC_WORKSPACE_MAX);
  if (!p->proxy_pos_dev)
    return nacl::fail_status(NACL_ERR_INVALID_ARG, "proxy_pos_dev is required (no host-to-device copy on this path)");
  void* ws = nullptr;
  int st = scratch_of_current_device(&ws);
  if (st) return st;
  st = nacl_evict(p, q, k, v, C, Cr, sampling, seed, layer, scores, keep_idx, k_out, v_out, ws,
                  (size_t)NACL_NOALLOC_WORKSPACE_MAX, stream);
  if (st || !health) return st;
  hipError_t e = hipMemcpyAsync(health, static_cast<char*>(ws) + 4, 2 * sizeof(uint32_t), hipMemcpyDeviceToDevice,
                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return nacl::fail_status(NACL_ERR_HIP, "copying the health words: %s", hipGetErrorString(e));
  return NACL_OK;
}

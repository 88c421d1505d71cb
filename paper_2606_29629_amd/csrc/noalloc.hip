// tri_layer_decode_noalloc: the decode step with its scratch in a file-scope
// device array instead of a caller-provided workspace, for callers that
// cannot allocate (code under HIP graph capture, tight serving loops).
//
// Each GPU the library runs on holds its own copy of `scratch` until the
// process ends.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in for the symbol): the device address is looked up
// once per device with hipGetSymbolAddress, with that device current, and
// that address is what the layer's kernels receive.  Every call on a GPU
// shares its array; no kernel of the decode step needs the scratch cleared
// (every partial it reads was written earlier in the same call), and calls
// that overlap on one GPU race on it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "host.hpp"

namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;  // == TRI_NOALLOC_SCRATCH_BYTES
static_assert(kScratchBytes == TRI_NOALLOC_SCRATCH_BYTES, "scratch size mismatch");

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this GPU's scratch (looked up on its first use here).
tri_status scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TRI_ERR_HIP;
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TRI_ERR_HIP;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return TRI_OK;
}

}  // namespace

extern "C" tri_status tri_layer_decode_noalloc(const tri_layer_config* cfg,
                                               const tri_layer_weights* w,
                                               const tri_kv_cache* cache, const tri_batch* batch,
                                               const void* x_in, void* x_out, int32_t* route_idx,
                                               float* route_w, void* stream) {
  size_t need = 0;
  tri_status st = tri_workspace_size(cfg, batch, &need);
  if (st != TRI_OK) return st;
  if (need > kScratchBytes) return TRI_ERR_SCRATCH;
  if (batch->n_tokens == 0) return TRI_OK;
  void* ws = nullptr;
  if ((st = scratch_ptr(&ws)) != TRI_OK) return st;
  return tri::layer_call(true, false, cfg, w, cache, batch, x_in, x_out, route_idx, route_w, ws,
                         kScratchBytes, stream);
}

// starkv_score_noalloc: starkv_score with its workspace in a library-owned
// device array instead of a caller buffer, for callers that cannot
// allocate.  The array is a file-scope __device__ object, so every GPU the
// library runs on holds its own copy from module load until the process
// ends.  Host code never passes the array's name to a kernel: it takes each
// device's address once with hipGetSymbolAddress (with that device current)
// and passes that pointer, as starkv_score passes its workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace starkv {
namespace {

constexpr size_t kScratchBytes = STARKV_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address per device, guarded by g_scratch_mu

// The current device's copy of `scratch`, looked up on the first call on
// that device.  Returns a HIP error code, or 0.
int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return e != hipSuccess ? (int)e : (int)hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return 0;
}

}  // namespace
}  // namespace starkv

using namespace starkv;

extern "C" starkv_status starkv_score_noalloc(const starkv_dims* dims,
                                              const starkv_params* params,
                                              const void* q, const void* k,
                                              const starkv_kv_layout* k_layout,
                                              float* S, float* sbar, uint8_t* gstar,
                                              void* stream) {
  Geometry g;
  starkv_status st = check_dims(dims, &g);
  if (st != STARKV_OK) return st;
  if ((st = check_pool(params)) != STARKV_OK) return st;
  if (!q || !k || !k_layout || !S || !sbar || !gstar) return STARKV_E_NULL;
  if ((st = check_layout(k_layout, g)) != STARKV_OK) return st;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(S, 4) || !aligned(sbar, 4))
    return STARKV_E_ALIGN;
  // the workspace this call needs must fit the array
  if (ws_layout(g).total > kScratchBytes) return STARKV_E_WORKSPACE;
  void* ws = nullptr;
  if (scratch_address(&ws)) return STARKV_E_HIP;
  // every workspace byte the kernels read is written earlier in the same
  // call (chunk statistics by pass 1, S before pooling by pass 2), so the
  // previous call's contents need no clearing
  return launch_score(g, *params, q, k, *k_layout, S, sbar, gstar, ws, stream)
             ? STARKV_E_HIP
             : STARKV_OK;
}

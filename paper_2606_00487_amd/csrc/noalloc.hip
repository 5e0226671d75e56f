// taps_select for callers that cannot allocate (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc): the selection's scratch (per-chunk top-K
// candidates and normaliser partials) lives in a file-scope device array instead of a
// caller workspace.  Each GPU the library runs on holds its own copy of the array until the
// process ends; its device address is looked up once per device and kept.
#include <atomic>
#include <mutex>

#include "common.h"

namespace taps {

namespace {

static __device__ __align__(256) unsigned char scratch[TAPS_SELECT_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lookup;
std::atomic<void*> g_addr[kMaxDevices];   // device address of `scratch` per device, or null

// The address of the current device's copy of `scratch` (looked up on the first call on
// that device).  In host code the array's name is only a stand-in for the symbol, never a
// device address, so every use goes through the pointer this returns.
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_lookup);
    p = g_addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return hipSuccess;
}

}  // namespace

}  // namespace taps

extern "C" taps_status taps_select_noalloc(const void* marginals, const taps_select_params* p,
                                           const taps_tree* out, hipStream_t stream) {
  const taps_status st = taps_select_validate(p);
  if (st != TAPS_OK) return st;
  if (p->batch == 0) return TAPS_OK;
  if (!marginals || !out || !out->parent || !out->token || !out->depth || !out->rank ||
      !out->q_reach || !out->n_nodes || !out->topk_idx)
    return TAPS_ERR_INVALID_ARG;
  if (taps_select_workspace_bytes(p) > (size_t)TAPS_SELECT_SCRATCH_BYTES) return TAPS_ERR_WORKSPACE;
  void* ws = nullptr;
  if (taps::scratch_address(&ws) != hipSuccess) return TAPS_ERR_HIP;
  // the candidates are written in full by the vocabulary scan before the selection reads
  // them, so nothing left in the array by an earlier call is read
  return taps_select(marginals, p, out, ws, (size_t)TAPS_SELECT_SCRATCH_BYTES, stream);
}

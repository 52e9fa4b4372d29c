// The attention core with its workspace in a fixed device array of the library, for callers
// that cannot allocate device memory (code under graph capture, tight serving loops, harnesses
// that forbid it).  The kernels, their order and their results are those of hspec_paged_attn:
// this entry point only supplies the workspace.
//
// The array `scratch` below lives in every device's copy of the code object.  On the host its
// name is only a stand-in for the symbol, never a device address: the address comes from
// hipGetSymbolAddress, taken once per device (with that device current) on the first call
// there and kept.  Calls on one device share that device's array, so calls that overlap on one
// device (on different streams, or from different threads without ordering) race on it.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "hspec.h"
#include "kernels.h"

#define HSPEC_API extern "C" __attribute__((visibility("default")))

namespace {

static __device__ __align__(256) unsigned char scratch[HSPEC_STATIC_WS_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];   // per-device address of `scratch` (null: not yet taken)
std::mutex g_scratch_mu;                     // serialises the first lookup on a device

hspec_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hspec::api_fail(HSPEC_ERR_LAUNCH, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return hspec::api_fail(HSPEC_ERR_UNSUPPORTED, "device index above 63");
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return hspec::api_fail(HSPEC_ERR_LAUNCH, e != hipSuccess ? hipGetErrorString(e)
                                                                  : "hipGetSymbolAddress returned NULL");
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return HSPEC_OK;
}

}  // namespace

HSPEC_API hspec_status hspec_paged_attn_static(const hspec_attn_cfg* cfg, const void* q, const void* k_blk,
                                               const void* v_blk, const void* k_cache, const void* v_cache,
                                               const int32_t* page_table, const int32_t* ctx_lens, int max_ctx_len,
                                               float* o, int32_t* status, void* stream) {
  if (!cfg) return hspec::api_fail(HSPEC_ERR_NULL, "attention config is NULL");
  const size_t need = hspec_paged_attn_workspace(cfg, max_ctx_len);
  if (need > (size_t)HSPEC_STATIC_WS_BYTES)
    return hspec::api_fail(HSPEC_ERR_WORKSPACE,
                           "this attention needs more workspace than the library's fixed array "
                           "(HSPEC_STATIC_WS_BYTES); call hspec_paged_attn with a workspace");
  void* ws = nullptr;
  if (hspec_status s = scratch_address(&ws)) return s;
  // Every kernel that needs zeroed words in the workspace clears them itself (the work list
  // kernel, the first of the call, clears the status and queue words), so the contents the
  // previous call left behind are harmless.
  if (hspec_status s = hspec_paged_attn(cfg, q, k_blk, v_blk, k_cache, v_cache, page_table, ctx_lens, max_ctx_len,
                                        o, ws, HSPEC_STATIC_WS_BYTES, stream))
    return s;
  if (status) {   // the device status word sits at the start of the workspace
    hipError_t e = hipMemcpyAsync(status, ws, sizeof(int32_t), hipMemcpyDeviceToDevice, (hipStream_t)stream);
    if (e != hipSuccess) return hspec::api_fail(HSPEC_ERR_LAUNCH, hipGetErrorString(e));
  }
  return HSPEC_OK;
}

// fp2_prefill_noalloc: fp2_prefill with its scratch memory in a static device
// array of the library instead of a caller workspace, for callers that cannot
// allocate device memory. Host code plus the array; the kernels are those of
// fp2_prefill, which take the array's device address as their workspace.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include <mutex>

#include "abi.h"

namespace {

// The scratch array. Its name is a host-side stand-in in host code: kernels
// get its device address on the current device, resolved below.
__device__ __align__(256) unsigned char scratch[FP2_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];   // device address of `scratch` per device (null until resolved)
std::mutex g_mu;

// Device address of the array on the current device, resolved once per device.
fp2_status_t scratch_on_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fp2::set_error(FP2_EHIP, "fp2_prefill_noalloc: hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices)
    return fp2::set_error(FP2_EUNSUPPORTED, "fp2_prefill_noalloc: device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      char msg[256];
      snprintf(msg, sizeof(msg), "fp2_prefill_noalloc: hipGetSymbolAddress of the scratch array: %s",
               hipGetErrorString(e));
      return fp2::set_error(FP2_EHIP, msg);
    }
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return FP2_OK;
}

}  // namespace

extern "C" fp2_status_t fp2_prefill_noalloc(const fp2_params_t* params, const void* q,
                                            const int32_t* cu_seqlens,
                                            const int32_t* cu_seqlens_host,
                                            const int32_t* cu_seqlens_k,
                                            const int32_t* cu_seqlens_k_host, const void* k_cache,
                                            const void* v_cache, const int32_t* block_table,
                                            const float* q_scale, const float* k_scale,
                                            const float* v_scale, void* out, float* lse,
                                            uint8_t* block_mask, void* stream) {
  const size_t need = fp2::workspace_need(params);
  if (need > FP2_NOALLOC_SCRATCH_BYTES) {
    char msg[256];
    snprintf(msg, sizeof(msg),
             "fp2_prefill_noalloc: the call needs %zu bytes of scratch, the static array holds %zu "
             "(use fp2_prefill with a workspace)",
             need, (size_t)FP2_NOALLOC_SCRATCH_BYTES);
    return fp2::set_error(FP2_EWORKSPACE, msg);
  }
  void* ws = nullptr;
  if (need > 0) {
    const fp2_status_t st = scratch_on_current_device(&ws);
    if (st != FP2_OK) return st;
  }
  return fp2::prefill_impl(params, q, cu_seqlens, cu_seqlens_host, cu_seqlens_k, cu_seqlens_k_host,
                           k_cache, v_cache, block_table, q_scale, k_scale, v_scale, nullptr, out,
                           lse, block_mask, ws, FP2_NOALLOC_SCRATCH_BYTES, stream);
}

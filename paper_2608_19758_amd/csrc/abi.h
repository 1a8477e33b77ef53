// Host-side pieces of the C ABI shared by its source files (internal).
#pragma once
#include "fp2.h"

namespace fp2 {

// fp2_prefill / fp2_prefill_cached (cache may be null), with validation.
fp2_status_t prefill_impl(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                          const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                          const int32_t* cu_seqlens_k_host, const void* k_cache,
                          const void* v_cache, const int32_t* block_table, const float* q_scale,
                          const float* k_scale, const float* v_scale,
                          const fp2_means_cache_t* cache, void* out, float* lse,
                          uint8_t* block_mask, void* workspace, size_t workspace_bytes,
                          void* stream);

// fp2_workspace_bytes without the C linkage (0 for invalid params).
size_t workspace_need(const fp2_params_t* params);

// Record a failure for fp2_last_error and return st.
fp2_status_t set_error(fp2_status_t st, const char* msg);

}  // namespace fp2

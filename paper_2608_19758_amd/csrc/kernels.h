// Launchers of the libfp2 kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace fp2 {

// Everything a kernel needs to find its rows, shared by all stages.
struct Problem {
  const void* q;            // [total, Hq, d] bf16 or e4m3 codes
  const int32_t* cu;        // [batch + 1] query rows
  const int32_t* cuk;       // [batch + 1] KV tokens (== cu without a prefix); the
                            // queries of sequence b are its last cu-lengths keys
  const void* k;            // pool or contiguous, bf16 or e4m3 codes
  const void* v;
  PageMap pm;
  const float* q_scale;     // fp8 only
  const float* k_scale;
  const float* v_scale;
  int32_t batch, hq, hkv, g;
  int32_t nbmax;            // query blocks per sequence bound (mask rows)
  int32_t nbk;              // key blocks per sequence bound (mask columns, pooled rows)
  int32_t sink, window, recent, corr;
  int32_t splits;           // KV splits per unit (Eq. split), >= 1
  float alpha;
  float scale_log2;         // softmax_scale * log2(e)
  int32_t fp8;
};

// Workspace views.
struct Pooled {
  uint16_t* khat;           // [batch, Hkv, nbk, d] bf16 key means (scoring and correction)
  uint16_t* vbar;           // [batch, Hkv, nbk, d] bf16 value means (correction)
};

struct KeptLists {
  int32_t* idx;             // [batch, Hkv, nbmax, nbk] ascending kept blocks per row
  int32_t* cnt;             // [batch, Hkv, nbmax]
  int32_t* queue;           // work counter of the attention kernel; the kernel that
                            // builds the lists sets it to 0
};

// Partial results of the KV splits of each unit (used when splits > 1): for
// unit row `row` = (b * Hkv + h) * nbmax + I and split u, slot row * splits + u
// holds, per packed row r of the unit, the unnormalised accumulator o (fp32,
// 128 values; value codes for fp8) and {m, l} (running maximum of the base-2
// logits and the denominator).
struct Partials {
  float* o;                 // [rows * splits, g * B, d]
  float* ml;                // [rows * splits, g * B, 2]
};

// Work items of the attention kernel per (sequence, KV head, query block),
// before splitting: row slices of 32 * waves packed rows.
int attend_items_per_unit(int g);

hipError_t launch_pool(const Problem& p, Pooled out, hipStream_t s);
hipError_t launch_estimate(const Problem& p, const Pooled& pooled, uint8_t* mask, KeptLists kl,
                           hipStream_t s);
hipError_t launch_compact(const Problem& p, const uint8_t* mask, KeptLists kl, hipStream_t s);
hipError_t launch_attend(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                         const KeptLists& kl, const Partials& part, void* out, float* lse,
                         hipStream_t s);

}  // namespace fp2

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
  int32_t nbmax;            // query tiles per sequence bound (mask rows)
  int32_t qtile;            // positions per query tile: kBlock, or 128 / g for the
                            // 128-packed-row tile; it divides kBlock, so tile I lies
                            // in key block (prefix + I * qtile) / kBlock
  int32_t nbk;              // key blocks per sequence bound (mask columns, pooled rows)
  int32_t sink, window, recent, corr;
  int32_t splits;           // KV splits: 0 = cost-balanced plan, n >= 1 = n per unit
  int32_t ssplits;          // scoring row parts: 0 = automatic, n >= 1 = at most n
  float alpha;
  float scale_log2;         // softmax_scale * log2(e)
  int32_t fp8;
};

// Workspace views.
struct Pooled {
  uint16_t* khat;           // [batch, Hkv, nbk, d] bf16 key means (scoring; bf16 correction)
  uint16_t* vbar;           // [batch, Hkv, nbk, d] bf16 value means (bf16 correction)
  uint8_t* khat8;           // fp8 inputs: [batch, Hkv, nbk, d] e4m3 code means of the keys,
  uint8_t* vbar8;           // e4m3(khat / k_scale), and of the values (fp8 correction); else null
};

// Block means kept by the caller across calls (chunked prefill, prefix
// caching): slot of key block J of sequence b = page id of its first token
// times per_page plus (offset of that token in its page) / B for a paged pool
// (per_page = ceil(page / B)), b * nbk + J for contiguous KV. Blocks J below
// min(pooled[b], complete blocks of b) are copied from the cache instead of
// being pooled; every pooled block is also written to it. khat == nullptr: no
// cache.
struct MeansCache {
  uint16_t* khat;           // [slots, Hkv, d] bf16
  uint16_t* vbar;           // [slots, Hkv, d] bf16
  const int32_t* pooled;    // [batch] leading blocks already in the cache
  int32_t per_page;
};

struct KeptLists {
  int32_t* idx;             // [batch, Hkv, nbmax, nbk] ascending kept blocks per row
  int32_t* cnt;             // [batch, Hkv, nbmax]
};

// Work plan of the attention kernel (Sec. 3.3 Eq. split and Eq. cost), built
// on the device after the kept lists by plan_kernel. Unit rows are indexed
// row = (b * Hkv + h) * nbmax + I; the attention order is q = (nbmax - 1 - I)
// * (batch * Hkv) + b * Hkv + h (decreasing query block, heaviest first).
struct Plan {
  int4* items;              // [cap_items] {q, k, U, first partial slot or -1}: unit q in
                            // attention order, split k / wpu, row slice k % wpu, and the
                            // unit's rowinfo entry (so one load describes an item)
  int2* rowinfo;            // [rows] {splits U, first partial slot or -1}
  int32_t* splitrows;       // [cap_slots / 2] unit rows with U > 1
  int32_t* counts;          // [0] work counter (zeroed by the plan), [1] items, [2] split rows
  float* part_o;            // [cap_slots, g * B, d] unnormalised partial outputs (fp32;
                            // value codes for fp8)
  float* part_ml;           // [cap_slots, g * B, 2] {running maximum (base 2), denominator}
  int32_t cap_items, cap_slots;
  int32_t target_items;     // work items the cost-balanced plan aims at
};

// Work items of the attention kernel per (sequence, KV head, query block),
// before splitting: row slices of 32 * waves packed rows.
int attend_items_per_unit(int g, int qtile);

// Compute units of the current device (0 if it cannot be queried).
int device_compute_units();

// Rate-calibration loops (calib.hip): kind is an fp2_calib_kind_t; *ops gets
// the operations of the launch (FLOP or exps).
hipError_t launch_calib(int kind, int iters, float* sink, double* ops, hipStream_t s);

hipError_t launch_pool(const Problem& p, Pooled out, hipStream_t s,
                       const MeansCache& cache = MeansCache{nullptr, nullptr, nullptr, 0});
hipError_t launch_estimate(const Problem& p, const Pooled& pooled, uint8_t* mask, KeptLists kl,
                           hipStream_t s, float* scratch = nullptr, size_t scratch_floats = 0);
hipError_t launch_compact(const Problem& p, const uint8_t* mask, KeptLists kl, hipStream_t s);
hipError_t launch_plan(const Problem& p, const KeptLists& kl, const Plan& plan, hipStream_t s);
hipError_t launch_attend(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                         const KeptLists& kl, const Plan& plan, void* out, float* lse,
                         hipStream_t s);
hipError_t launch_combine(const Problem& p, const Plan& plan, void* out, float* lse,
                          hipStream_t s);
hipError_t launch_mask_to_csr(const Problem& p, const uint8_t* mask, int32_t* counts,
                              int32_t* offsets, int32_t* indices, hipStream_t s);

}  // namespace fp2

// C ABI of libfp2: argument validation, workspace layout and the launch
// sequence of each entry point (Algorithm 1 of Sec. 3.4). Host code only.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <string>

#include "fp2.h"
#include "kernels.h"
#include "abi.h"

namespace {

thread_local std::string g_last_error;

// Events of fp2_time_kernels for calls made on this host thread (null: none).
struct KernelEvents {
  hipEvent_t est_begin = nullptr, est_end = nullptr, att_begin = nullptr, att_end = nullptr;
};
thread_local KernelEvents g_events;

hipError_t record(hipEvent_t ev, hipStream_t s) { return ev ? hipEventRecord(ev, s) : hipSuccess; }

fp2_status_t fail(fp2_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

fp2_status_t ok() {
  g_last_error.clear();
  return FP2_OK;
}

constexpr int kMaxSeqLen = fp2::kMaxBlocks * fp2::kBlock;   // 1M tokens

int max_kv_of(const fp2_params_t* p) { return p->max_kv_len > 0 ? p->max_kv_len : p->max_seq_len; }
// query blocks (mask rows) and key blocks (mask columns, pooled rows)
// positions per query tile: a block of B positions, or one 128-packed-row
// M-tile of 128 / g positions
int qtile_of(const fp2_params_t* p) {
  return p->query_tile_rows > 0 ? p->query_tile_rows / (p->num_q_heads / p->num_kv_heads)
                                : fp2::kBlock;
}
int nbq_of(const fp2_params_t* p) { return (p->max_seq_len + qtile_of(p) - 1) / qtile_of(p); }
int nbk_of(const fp2_params_t* p) { return (max_kv_of(p) + fp2::kBlock - 1) / fp2::kBlock; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr int kMaxSplits = 32;            // parts per unit (one per lane of the combine)
constexpr size_t kPartialRows = 65536;    // packed rows of partial outputs, cost-balanced mode

struct Layout {
  size_t khat, vbar, khat8, vbar8, kidx, kcnt, items, rowinfo, splitrows, counts, part_o, part_ml,
      total;
  int32_t cap_items, cap_slots;
};

// Workspace sections. The attention plan holds an item table, per-unit split
// information, the list of split units and the counters; the partial outputs
// of split units take g*B packed rows of d fp32 values and {m, l} per slot.
// kv_splits == 0 (cost-balanced) has kPartialRows packed rows of slots (the
// plan raises its step budget until the parts fit), n > 1 has n per unit,
// n == 1 none.
Layout layout_of(const fp2_params_t* p) {
  Layout l{};
  const size_t heads = (size_t)p->batch * p->num_kv_heads;
  const size_t rows = heads * nbq_of(p);    // (sequence, KV head, query block)
  const size_t krows = heads * nbk_of(p);   // (sequence, KV head, key block)
  const int g = p->num_q_heads / p->num_kv_heads;
  const size_t rpu = (size_t)g * qtile_of(p);
  const size_t wpu = (size_t)fp2::attend_items_per_unit(g, qtile_of(p));
  size_t slots, items;
  if (p->kv_splits == 0) {
    slots = kPartialRows / rpu;
    items = wpu * (rows + slots);
  } else {
    slots = p->kv_splits > 1 ? rows * p->kv_splits : 0;
    items = wpu * rows * p->kv_splits;
  }
  size_t off = 0;
  l.khat = off;
  off = align256(off + krows * fp2::kHeadDim * sizeof(uint16_t));
  l.vbar = off;
  off = align256(off + krows * fp2::kHeadDim * sizeof(uint16_t));
  if (p->dtype == FP2_FP8_E4M3) {   // e4m3 code means for the fp8 correction
    l.khat8 = off;
    off = align256(off + krows * fp2::kHeadDim);
    l.vbar8 = off;
    off = align256(off + krows * fp2::kHeadDim);
  }
  l.kidx = off;
  off = align256(off + rows * nbk_of(p) * sizeof(int32_t));
  l.kcnt = off;
  off = align256(off + rows * sizeof(int32_t));
  l.items = off;
  off = align256(off + items * 4 * sizeof(int32_t));
  l.rowinfo = off;
  off = align256(off + rows * 2 * sizeof(int32_t));
  l.splitrows = off;
  off = align256(off + (slots / 2 + 1) * sizeof(int32_t));
  l.counts = off;
  off += 256;
  if (slots) {
    l.part_o = off;
    off = align256(off + slots * rpu * fp2::kHeadDim * sizeof(float));
    l.part_ml = off;
    off = align256(off + slots * rpu * 2 * sizeof(float));
  }
  l.cap_items = (int32_t)items;
  l.cap_slots = (int32_t)slots;
  l.total = rows ? off : 0;
  return l;
}

fp2_status_t validate_params(const fp2_params_t* p) {
  if (!p) return fail(FP2_EINVAL, "params is null");
  if (p->batch < 0) return fail(FP2_EINVAL, "batch %d < 0", p->batch);
  if (p->num_kv_heads < 1) return fail(FP2_EINVAL, "num_kv_heads %d < 1", p->num_kv_heads);
  if (p->num_kv_heads > 1024)
    return fail(FP2_EUNSUPPORTED, "num_kv_heads %d > 1024", p->num_kv_heads);
  if (p->num_q_heads < 1 || p->num_q_heads % p->num_kv_heads)
    return fail(FP2_EINVAL, "num_q_heads %d is not a positive multiple of num_kv_heads %d",
                p->num_q_heads, p->num_kv_heads);
  const int g = p->num_q_heads / p->num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8)
    return fail(FP2_EUNSUPPORTED, "group size %d not in {1, 2, 4, 8}", g);
  if (p->head_dim <= 0) return fail(FP2_EINVAL, "head_dim %d <= 0", p->head_dim);
  if (p->head_dim != fp2::kHeadDim) return fail(FP2_EUNSUPPORTED, "head_dim %d != 128", p->head_dim);
  if (p->block_size <= 0) return fail(FP2_EINVAL, "block_size %d <= 0", p->block_size);
  if (p->block_size != fp2::kBlock) return fail(FP2_EUNSUPPORTED, "block_size %d != 128", p->block_size);
  if (p->page_size < 0) return fail(FP2_EINVAL, "page_size %d < 0", p->page_size);
  if (p->max_seq_len < 0) return fail(FP2_EINVAL, "max_seq_len %d < 0", p->max_seq_len);
  if (p->max_seq_len > kMaxSeqLen)
    return fail(FP2_EUNSUPPORTED, "max_seq_len %d > %d", p->max_seq_len, kMaxSeqLen);
  if (p->max_kv_len < 0) return fail(FP2_EINVAL, "max_kv_len %d < 0", p->max_kv_len);
  if (p->max_kv_len > 0 && p->max_kv_len < p->max_seq_len)
    return fail(FP2_EINVAL, "max_kv_len %d < max_seq_len %d", p->max_kv_len, p->max_seq_len);
  if (p->max_kv_len > kMaxSeqLen)
    return fail(FP2_EUNSUPPORTED, "max_kv_len %d > %d", p->max_kv_len, kMaxSeqLen);
  if (p->page_size > 0) {
    const int need = (max_kv_of(p) + p->page_size - 1) / p->page_size;
    if (p->max_pages_per_seq < need)
      return fail(FP2_EINVAL, "max_pages_per_seq %d < ceil(max_kv_len / page_size) = %d",
                  p->max_pages_per_seq, need);
  }
  if (!(p->alpha >= 0.f) || !isfinite(p->alpha))
    return fail(FP2_EINVAL, "alpha must be finite and >= 0");
  if (p->sink_blocks < 0 || p->window_blocks < 0 || p->recent_blocks < 0)
    return fail(FP2_EINVAL, "sink/window/recent block counts must be >= 0");
  if (p->mean_correction != 0 && p->mean_correction != 1)
    return fail(FP2_EINVAL, "mean_correction must be 0 or 1");
  if (!isfinite(p->softmax_scale)) return fail(FP2_EINVAL, "softmax_scale is not finite");
  if (p->dtype != FP2_BF16 && p->dtype != FP2_FP8_E4M3)
    return fail(FP2_EINVAL, "dtype %d unknown", p->dtype);
  if (p->kv_splits < 0 || p->kv_splits > kMaxSplits)
    return fail(FP2_EINVAL, "kv_splits %d not in [0, %d]", p->kv_splits, kMaxSplits);
  if (p->score_splits < 0 || p->score_splits > 64)
    return fail(FP2_EINVAL, "score_splits %d not in [0, 64]", p->score_splits);
  if (p->query_tile_rows != 0 && p->query_tile_rows != 128)
    return fail(FP2_EUNSUPPORTED, "query_tile_rows %d not 0 or 128", p->query_tile_rows);
  return FP2_OK;
}

bool aligned16(const void* x) { return ((uintptr_t)x & 15u) == 0; }

// Validation of everything but the workspace; `work` is false when there is
// nothing to compute (no sequence or zero-length bound).
// Host copy of cumulative lengths: starts at 0, non-decreasing, each length
// at most `bound`.
fp2_status_t check_cu(const int32_t* cu, int batch, int bound, const char* name, const char* bname) {
  if (cu[0] != 0) return fail(FP2_EINVAL, "%s[0] = %d != 0", name, cu[0]);
  for (int b = 0; b < batch; ++b) {
    const int len = cu[b + 1] - cu[b];
    if (len < 0) return fail(FP2_EINVAL, "%s decreases at %d", name, b);
    if (len > bound)
      return fail(FP2_EINVAL, "%s: sequence %d has length %d > %s %d", name, b, len, bname, bound);
  }
  return FP2_OK;
}

fp2_status_t validate_common(const fp2_params_t* p, const void* q, const int32_t* cu,
                             const int32_t* cu_host, const int32_t* cuk, const int32_t* cuk_host,
                             const void* k, const void* v, const int32_t* bt, const float* qs,
                             const float* ks, const float* vs, bool need_q, bool* work) {
  fp2_status_t st = validate_params(p);
  if (st != FP2_OK) return st;
  *work = p->batch > 0 && p->max_seq_len > 0;
  if (!*work) return FP2_OK;
  if (!cu) return fail(FP2_EINVAL, "cu_seqlens is null");
  if (need_q && !q) return fail(FP2_EINVAL, "q is null");
  if (!k || !v) return fail(FP2_EINVAL, "k_cache or v_cache is null");
  if ((need_q && !aligned16(q)) || !aligned16(k) || !aligned16(v))
    return fail(FP2_EINVAL, "q, k_cache and v_cache must be 16-byte aligned");
  if (p->page_size > 0 && !bt) return fail(FP2_EINVAL, "block_table is null with page_size > 0");
  if (p->dtype == FP2_FP8_E4M3 && ((need_q && !qs) || !ks || !vs))
    return fail(FP2_EINVAL, "fp8 needs q_scale, k_scale and v_scale");
  if (cuk_host && !cuk) return fail(FP2_EINVAL, "cu_seqlens_k_host given without cu_seqlens_k");
  if (cu_host && (st = check_cu(cu_host, p->batch, p->max_seq_len, "cu_seqlens", "max_seq_len")))
    return st;
  if (cuk_host && (st = check_cu(cuk_host, p->batch, max_kv_of(p), "cu_seqlens_k", "max_kv_len")))
    return st;
  if (cu_host && cuk_host) {
    for (int b = 0; b < p->batch; ++b) {
      const int pre = (cuk_host[b + 1] - cuk_host[b]) - (cu_host[b + 1] - cu_host[b]);
      if (pre < 0)
        return fail(FP2_EINVAL, "sequence %d: KV length < query length (by %d)", b, -pre);
    }
  }
  return FP2_OK;
}

fp2_status_t validate_ws(const fp2_params_t* p, const void* ws, size_t bytes) {
  const size_t need = layout_of(p).total;
  if (need == 0) return FP2_OK;
  if (!ws) return fail(FP2_EWORKSPACE, "workspace is null (need %zu bytes)", need);
  if (((uintptr_t)ws & 255u) != 0) return fail(FP2_EWORKSPACE, "workspace is not 256-byte aligned");
  if (bytes < need) return fail(FP2_EWORKSPACE, "workspace has %zu bytes, need %zu", bytes, need);
  return FP2_OK;
}

int log2_exact(int x) {
  if (x <= 0 || (x & (x - 1))) return -1;
  int s = 0;
  while ((1 << s) < x) ++s;
  return s;
}

fp2::Problem make_problem(const fp2_params_t* p, const void* q, const int32_t* cu,
                          const int32_t* cuk, const void* k, const void* v, const int32_t* bt,
                          const float* qs, const float* ks, const float* vs) {
  fp2::Problem pr{};
  pr.q = q;
  pr.cu = cu;
  pr.cuk = cuk ? cuk : cu;
  pr.k = k;
  pr.v = v;
  pr.pm.table = bt;
  pr.pm.stride = p->max_pages_per_seq;
  pr.pm.page = p->page_size;
  pr.pm.shift = log2_exact(p->page_size);
  pr.q_scale = qs;
  pr.k_scale = ks;
  pr.v_scale = vs;
  pr.batch = p->batch;
  pr.hq = p->num_q_heads;
  pr.hkv = p->num_kv_heads;
  pr.g = p->num_q_heads / p->num_kv_heads;
  pr.nbmax = nbq_of(p);
  pr.qtile = qtile_of(p);
  pr.nbk = nbk_of(p);
  pr.sink = p->sink_blocks;
  pr.window = p->window_blocks;
  pr.recent = p->recent_blocks;
  pr.corr = p->mean_correction;
  pr.splits = p->kv_splits;
  pr.ssplits = p->score_splits;
  pr.alpha = p->alpha;
  const double scale = p->softmax_scale > 0.f ? (double)p->softmax_scale : 1.0 / sqrt((double)p->head_dim);
  pr.scale_log2 = (float)(scale * 1.4426950408889634074);
  pr.fp8 = p->dtype == FP2_FP8_E4M3;
  return pr;
}

struct Views {
  fp2::Pooled pooled;
  fp2::KeptLists kl;
  fp2::Plan plan;
  size_t part_o_floats;   // the partial outputs, also the scoring's row-split scratch
};

Views views_of(const fp2_params_t* p, void* ws) {
  const Layout l = layout_of(p);
  char* base = (char*)ws;
  Views v;
  v.pooled.khat = (uint16_t*)(base + l.khat);
  v.pooled.vbar = (uint16_t*)(base + l.vbar);
  v.pooled.khat8 = l.khat8 ? (uint8_t*)(base + l.khat8) : nullptr;
  v.pooled.vbar8 = l.vbar8 ? (uint8_t*)(base + l.vbar8) : nullptr;
  v.kl.idx = (int32_t*)(base + l.kidx);
  v.kl.cnt = (int32_t*)(base + l.kcnt);
  v.plan.items = (int4*)(base + l.items);
  v.plan.rowinfo = (int2*)(base + l.rowinfo);
  v.plan.splitrows = (int32_t*)(base + l.splitrows);
  v.plan.counts = (int32_t*)(base + l.counts);
  v.plan.part_o = l.part_o ? (float*)(base + l.part_o) : nullptr;
  v.plan.part_ml = l.part_ml ? (float*)(base + l.part_ml) : nullptr;
  v.plan.cap_items = l.cap_items;
  v.plan.cap_slots = l.cap_slots;
  v.plan.target_items = 4 * fp2::device_compute_units();
  const size_t rpu = (size_t)(p->num_q_heads / p->num_kv_heads) * qtile_of(p);
  v.part_o_floats = l.part_o ? (size_t)l.cap_slots * rpu * fp2::kHeadDim : 0;
  return v;
}

fp2_status_t hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(FP2_EHIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

size_t fp2_workspace_bytes(const fp2_params_t* params) {
  if (validate_params(params) != FP2_OK) return 0;
  return layout_of(params).total;
}

}  // extern "C"

namespace fp2 {

fp2_status_t prefill_impl(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                          const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                          const int32_t* cu_seqlens_k_host, const void* k_cache,
                          const void* v_cache, const int32_t* block_table, const float* q_scale,
                          const float* k_scale, const float* v_scale,
                          const fp2_means_cache_t* cache, void* out, float* lse,
                          uint8_t* block_mask, void* workspace, size_t workspace_bytes,
                          void* stream) {
  bool work = false;
  fp2_status_t st = validate_common(params, q, cu_seqlens, cu_seqlens_host, cu_seqlens_k,
                                    cu_seqlens_k_host, k_cache, v_cache, block_table, q_scale,
                                    k_scale, v_scale, true, &work);
  if (st != FP2_OK) return st;
  if (!work) return ok();
  if (!out || !block_mask) return fail(FP2_EINVAL, "out or block_mask is null");
  if (!aligned16(out)) return fail(FP2_EINVAL, "out must be 16-byte aligned");
  if ((st = validate_ws(params, workspace, workspace_bytes)) != FP2_OK) return st;
  const fp2::Problem pr = make_problem(params, q, cu_seqlens, cu_seqlens_k, k_cache, v_cache,
                                       block_table, q_scale, k_scale, v_scale);
  fp2::MeansCache mc{nullptr, nullptr, nullptr, 0};
  if (cache) {
    if (!cache->khat || !cache->vbar || !cache->pooled_blocks)
      return fail(FP2_EINVAL, "means cache: khat, vbar and pooled_blocks must be non-null");
    if (!aligned16(cache->khat) || !aligned16(cache->vbar))
      return fail(FP2_EINVAL, "means cache: khat and vbar must be 16-byte aligned");
    mc = fp2::MeansCache{(uint16_t*)cache->khat, (uint16_t*)cache->vbar, cache->pooled_blocks,
                         params->page_size > 0 ? (params->page_size + fp2::kBlock - 1) / fp2::kBlock
                                               : 0};
  }
  const Views vw = views_of(params, workspace);
  hipStream_t s = (hipStream_t)stream;
  const KernelEvents ev = g_events;
  hipError_t e = record(ev.est_begin, s);
  if (e == hipSuccess) e = fp2::launch_pool(pr, vw.pooled, s, mc);
  if (e == hipSuccess) e = fp2::launch_estimate(pr, vw.pooled, block_mask, vw.kl, s, vw.plan.part_o,
                                                vw.part_o_floats);
  if (e == hipSuccess) e = record(ev.est_end, s);
  if (e == hipSuccess) e = fp2::launch_plan(pr, vw.kl, vw.plan, s);
  if (e == hipSuccess) e = record(ev.att_begin, s);
  if (e == hipSuccess)
    e = fp2::launch_attend(pr, vw.pooled, block_mask, vw.kl, vw.plan, out, lse, s);
  if (e == hipSuccess) e = record(ev.att_end, s);
  if (e == hipSuccess) e = fp2::launch_combine(pr, vw.plan, out, lse, s);
  return hip_status(e, "fp2_prefill launch");
}

size_t workspace_need(const fp2_params_t* params) {
  return validate_params(params) != FP2_OK ? 0 : layout_of(params).total;
}

fp2_status_t set_error(fp2_status_t st, const char* msg) { return fail(st, "%s", msg); }

}  // namespace fp2

namespace {
using fp2::prefill_impl;
}  // namespace

extern "C" {

fp2_status_t fp2_prefill(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                         const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                         const int32_t* cu_seqlens_k_host, const void* k_cache, const void* v_cache,
                         const int32_t* block_table, const float* q_scale, const float* k_scale,
                         const float* v_scale, void* out, float* lse, uint8_t* block_mask,
                         void* workspace, size_t workspace_bytes, void* stream) {
  return prefill_impl(params, q, cu_seqlens, cu_seqlens_host, cu_seqlens_k, cu_seqlens_k_host,
                      k_cache, v_cache, block_table, q_scale, k_scale, v_scale, nullptr, out, lse,
                      block_mask, workspace, workspace_bytes, stream);
}

fp2_status_t fp2_prefill_cached(const fp2_params_t* params, const void* q,
                                const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                                const int32_t* cu_seqlens_k, const int32_t* cu_seqlens_k_host,
                                const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const float* q_scale,
                                const float* k_scale, const float* v_scale,
                                const fp2_means_cache_t* cache, void* out, float* lse,
                                uint8_t* block_mask, void* workspace, size_t workspace_bytes,
                                void* stream) {
  if (!cache) return fail(FP2_EINVAL, "means cache is null");
  return prefill_impl(params, q, cu_seqlens, cu_seqlens_host, cu_seqlens_k, cu_seqlens_k_host,
                      k_cache, v_cache, block_table, q_scale, k_scale, v_scale, cache, out, lse,
                      block_mask, workspace, workspace_bytes, stream);
}

size_t fp2_means_cache_slots(const fp2_params_t* params, int64_t num_pages) {
  if (validate_params(params) != FP2_OK || num_pages < 0) return 0;
  if (params->page_size == 0) return (size_t)params->batch * (size_t)nbk_of(params);
  return (size_t)num_pages * (size_t)((params->page_size + fp2::kBlock - 1) / fp2::kBlock);
}

fp2_status_t fp2_estimate(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                          const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                          const int32_t* cu_seqlens_k_host, const void* k_cache,
                          const void* v_cache, const int32_t* block_table, const float* q_scale,
                          const float* k_scale, const float* v_scale, uint8_t* block_mask,
                          void* workspace, size_t workspace_bytes, void* stream) {
  bool work = false;
  fp2_status_t st = validate_common(params, q, cu_seqlens, cu_seqlens_host, cu_seqlens_k,
                                    cu_seqlens_k_host, k_cache, v_cache, block_table, q_scale,
                                    k_scale, v_scale, true, &work);
  if (st != FP2_OK) return st;
  if (!work) return ok();
  if (!block_mask) return fail(FP2_EINVAL, "block_mask is null");
  if ((st = validate_ws(params, workspace, workspace_bytes)) != FP2_OK) return st;
  const fp2::Problem pr = make_problem(params, q, cu_seqlens, cu_seqlens_k, k_cache, v_cache,
                                       block_table, q_scale, k_scale, v_scale);
  const Views vw = views_of(params, workspace);
  hipStream_t s = (hipStream_t)stream;
  const KernelEvents ev = g_events;
  hipError_t e = record(ev.est_begin, s);
  if (e == hipSuccess) e = fp2::launch_pool(pr, vw.pooled, s);
  if (e == hipSuccess) e = fp2::launch_estimate(pr, vw.pooled, block_mask, vw.kl, s, vw.plan.part_o,
                                                vw.part_o_floats);
  if (e == hipSuccess) e = record(ev.est_end, s);
  return hip_status(e, "fp2_estimate launch");
}

fp2_status_t fp2_attend(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                        const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                        const int32_t* cu_seqlens_k_host, const void* k_cache, const void* v_cache,
                        const int32_t* block_table, const float* q_scale, const float* k_scale,
                        const float* v_scale, const uint8_t* block_mask_in, void* out, float* lse,
                        void* workspace, size_t workspace_bytes, void* stream) {
  bool work = false;
  fp2_status_t st = validate_common(params, q, cu_seqlens, cu_seqlens_host, cu_seqlens_k,
                                    cu_seqlens_k_host, k_cache, v_cache, block_table, q_scale,
                                    k_scale, v_scale, true, &work);
  if (st != FP2_OK) return st;
  if (!work) return ok();
  if (!out || !block_mask_in) return fail(FP2_EINVAL, "out or block_mask_in is null");
  if (!aligned16(out)) return fail(FP2_EINVAL, "out must be 16-byte aligned");
  if ((st = validate_ws(params, workspace, workspace_bytes)) != FP2_OK) return st;
  const fp2::Problem pr = make_problem(params, q, cu_seqlens, cu_seqlens_k, k_cache, v_cache,
                                       block_table, q_scale, k_scale, v_scale);
  const Views vw = views_of(params, workspace);
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (params->mean_correction) e = fp2::launch_pool(pr, vw.pooled, s);
  if (e == hipSuccess) e = fp2::launch_compact(pr, block_mask_in, vw.kl, s);
  if (e == hipSuccess) e = fp2::launch_plan(pr, vw.kl, vw.plan, s);
  const KernelEvents ev = g_events;
  if (e == hipSuccess) e = record(ev.att_begin, s);
  if (e == hipSuccess)
    e = fp2::launch_attend(pr, vw.pooled, block_mask_in, vw.kl, vw.plan, out, lse, s);
  if (e == hipSuccess) e = record(ev.att_end, s);
  if (e == hipSuccess) e = fp2::launch_combine(pr, vw.plan, out, lse, s);
  return hip_status(e, "fp2_attend launch");
}

fp2_status_t fp2_pool(const fp2_params_t* params, const int32_t* cu_seqlens,
                      const int32_t* cu_seqlens_host, const void* k_cache, const void* v_cache,
                      const int32_t* block_table, const float* k_scale, const float* v_scale,
                      void* khat, void* vbar, void* stream) {
  bool work = false;
  // the lengths here are KV lengths, bounded by max_kv_len
  fp2_params_t pp = params ? *params : fp2_params_t{};
  if (params) pp.max_seq_len = max_kv_of(params);
  fp2_status_t st = validate_common(params ? &pp : nullptr, nullptr, cu_seqlens, cu_seqlens_host,
                                    nullptr, nullptr, k_cache, v_cache, block_table, nullptr,
                                    k_scale, v_scale, false, &work);
  if (st != FP2_OK) return st;
  if (!work) return ok();
  if (!khat || !vbar) return fail(FP2_EINVAL, "khat or vbar is null");
  const fp2::Problem pr = make_problem(&pp, nullptr, cu_seqlens, nullptr, k_cache, v_cache,
                                       block_table, nullptr, k_scale, v_scale);
  fp2::Pooled pooled{(uint16_t*)khat, (uint16_t*)vbar, nullptr, nullptr};
  return hip_status(fp2::launch_pool(pr, pooled, (hipStream_t)stream), "fp2_pool launch");
}

size_t fp2_csr_capacity(const fp2_params_t* params) {
  if (validate_params(params) != FP2_OK) return 0;
  return (size_t)params->batch * params->num_kv_heads * nbq_of(params) * 2 * nbk_of(params);
}

fp2_status_t fp2_mask_to_csr(const fp2_params_t* params, const int32_t* cu_seqlens,
                             const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                             const int32_t* cu_seqlens_k_host, const uint8_t* block_mask,
                             int32_t* csr_offsets, int32_t* csr_indices, size_t capacity,
                             void* workspace, size_t workspace_bytes, void* stream) {
  fp2_status_t st = validate_params(params);
  if (st != FP2_OK) return st;
  if (params->batch == 0 || params->max_seq_len == 0) return ok();
  if (!cu_seqlens) return fail(FP2_EINVAL, "cu_seqlens is null");
  if (cu_seqlens_k_host && !cu_seqlens_k)
    return fail(FP2_EINVAL, "cu_seqlens_k_host given without cu_seqlens_k");
  if (cu_seqlens_host &&
      (st = check_cu(cu_seqlens_host, params->batch, params->max_seq_len, "cu_seqlens", "max_seq_len")))
    return st;
  if (cu_seqlens_k_host && (st = check_cu(cu_seqlens_k_host, params->batch, max_kv_of(params),
                                          "cu_seqlens_k", "max_kv_len")))
    return st;
  if (!block_mask || !csr_offsets || !csr_indices)
    return fail(FP2_EINVAL, "block_mask, csr_offsets or csr_indices is null");
  const size_t need = fp2_csr_capacity(params);
  if (capacity < need) return fail(FP2_EINVAL, "csr capacity %zu < %zu", capacity, need);
  if ((st = validate_ws(params, workspace, workspace_bytes)) != FP2_OK) return st;
  const fp2::Problem pr = make_problem(params, nullptr, cu_seqlens, cu_seqlens_k, nullptr, nullptr,
                                       nullptr, nullptr, nullptr, nullptr);
  const Views vw = views_of(params, workspace);
  return hip_status(fp2::launch_mask_to_csr(pr, block_mask, vw.kl.cnt, csr_offsets, csr_indices,
                                            (hipStream_t)stream),
                    "fp2_mask_to_csr launch");
}

fp2_status_t fp2_calibrate(fp2_calib_kind_t kind, int32_t iters, float* sink, double* ops,
                           void* stream) {
  if (kind != FP2_CALIB_MFMA_BF16 && kind != FP2_CALIB_MFMA_FP8 && kind != FP2_CALIB_EXP)
    return fail(FP2_EINVAL, "unknown calibration kind %d", (int)kind);
  if (iters < 1 || iters > (1 << 24)) return fail(FP2_EINVAL, "iters %d outside [1, 2^24]", iters);
  if (!sink || !ops) return fail(FP2_EINVAL, "sink or ops is null");
  return hip_status(fp2::launch_calib((int)kind, iters, sink, ops, (hipStream_t)stream),
                    "fp2_calibrate launch");
}

fp2_status_t fp2_time_kernels(void* estimate_begin, void* estimate_end, void* attend_begin,
                              void* attend_end) {
  if ((estimate_begin == nullptr) != (estimate_end == nullptr) ||
      (attend_begin == nullptr) != (attend_end == nullptr))
    return fail(FP2_EINVAL, "events come in begin/end pairs");
  g_events = KernelEvents{(hipEvent_t)estimate_begin, (hipEvent_t)estimate_end,
                          (hipEvent_t)attend_begin, (hipEvent_t)attend_end};
  return ok();
}

const char* fp2_status_str(fp2_status_t status) {
  switch (status) {
    case FP2_OK: return "ok";
    case FP2_EINVAL: return "invalid argument";
    case FP2_EUNSUPPORTED: return "unsupported configuration";
    case FP2_EWORKSPACE: return "workspace too small";
    case FP2_EHIP: return "HIP error";
  }
  return "unknown status";
}

const char* fp2_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"

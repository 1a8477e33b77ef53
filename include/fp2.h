/*
 * fp2.h -- block-sparse causal GQA prefill attention with max-based block
 * selection and mean correction (FlashPrefill V2), for AMD Instinct MI355X
 * (gfx950). C ABI of libfp2.so.
 *
 * The operator follows Algorithm 1 of the paper (Sec. 3.4): packed queries,
 * a paged KV cache with its page table, per-request lengths and a threshold
 * alpha in; the attention output and the selected-block mask out.
 *
 *   fp2_prefill  = fp2_estimate (pool, score, select) + attention over the
 *                  kept blocks with the mean correction, one call.
 *   fp2_estimate = the index stage only: block means, fused block scoring,
 *                  max-based thresholding, forced blocks, kept-block lists.
 *   fp2_attend   = the attention stage only, under a caller-given mask.
 *   fp2_pool     = the block means alone (exposed for verification).
 *   fp2_prefill_cached = fp2_prefill with block means kept across calls
 *                  (chunked prefill); fp2_means_cache_slots sizes the cache.
 *   fp2_mask_to_csr = a mask as the CSR index of 64-token key tiles;
 *                  fp2_csr_capacity sizes it.
 *   fp2_calibrate = MFMA and exp rate loops (measurement helper).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers (hipMalloc'd or torch CUDA
 *   tensors) unless the name ends in _host. The caller owns every buffer; the
 *   library never allocates, frees or synchronises. Work is enqueued on
 *   `stream` (a hipStream_t; NULL = the default stream) and returns at once.
 * - Scratch memory is the caller's `workspace` of at least
 *   fp2_workspace_bytes(params) bytes (256-byte aligned). It may be reused
 *   across calls and layers on one stream; concurrent calls need distinct
 *   workspaces.
 * - A call only enqueues kernels (no allocation, memset or host
 *   synchronisation; the work counters are reset by a kernel of the call
 *   itself), so it may be captured in a HIP graph and replayed, with every
 *   buffer it names kept at the same address; the host-side arguments
 *   (params, the _host arrays) are read at capture time only.
 * - Errors are reported as fp2_status_t only; nothing aborts. Host-visible
 *   arguments are validated before any launch (FP2_EINVAL, FP2_EUNSUPPORTED,
 *   FP2_EWORKSPACE); a failed launch returns FP2_EHIP. The consistency of
 *   device-resident arrays (cu_seqlens, block_table) with `params` is the
 *   caller's contract; pass cu_seqlens_host to have the lengths checked too.
 *   fp2_last_error() gives a one-line reason for the last failure of the
 *   calling thread.
 *
 * Prefix KV (chunked prefill)
 * ---------------------------
 * A sequence may hold more keys than queries: its L_q queries (cu_seqlens)
 * are the last L_q of its L_kv keys (cu_seqlens_k), i.e. query i sits at
 * absolute position P + i with P = L_kv - L_q >= 0, the tokens already in
 * the KV cache (earlier chunks, a cached prefix). The rows of query block I
 * then lie in key blocks Ja (that of its first row) to Jb (that of its last
 * row): Jb = Ja when P is a multiple of block_size, else possibly Ja + 1. In
 * every rule below, "J <= I" reads J <= Jb, the diagonal "J == I" reads
 * Ja <= J <= Jb, "I - J" reads Jb - J, and "J < I" (blocks every row sees in
 * full) reads J < Ja; positions are absolute. With cu_seqlens_k == NULL,
 * L_kv = L_q (P = 0, Ja = Jb = I). The selection of a query block depends
 * only on its own rows and the keys before them, so with P a multiple of
 * block_size a chunked prefill gives, row for row, the output of one call
 * over the whole sequence (bit for bit with kv_splits == 1 and
 * score_splits == 1, whose work splitting does not depend on the call's
 * size; else up to rounding).
 *
 * KV splits and the work plan (Sec. 3.3 Eq. split and Eq. cost)
 * --------------------------------------------------------------
 * The attention of a (sequence, KV head, query block) unit costs about one
 * 64-key step per half kept block (Eq. cost), which varies a lot between
 * heads. A unit cut into U parts has part u walk kept-list positions
 * [u ceil(T/U), min((u+1) ceil(T/U), T)) of its T kept blocks and correct the
 * pruned blocks of the u-th of U equal ranges of J (Eq. split); each part
 * leaves an unnormalised partial output with its running maximum and
 * denominator in the workspace, and a combine kernel merges them with the
 * usual log-sum-exp weights. The result equals the unsplit one up to
 * rounding (fp8: P~ is rounded against each part's own maximum).
 * kv_splits == 0 (the default) plans on the device after the selection:
 * only units costlier than a step budget are split, the budget being set by
 * the call's total cost over about four items per compute unit (so a short
 * chunk after a long prefix, or a few dense heads, no longer bound the run
 * time). kv_splits == n >= 1 cuts every unit into n parts (1 = no splits).
 *
 * Query tiles (Sec. 3.3 PackGQA and the per-tile index of Eq. csr)
 * --------------------------------------------------------------
 * Selection, attention and the index are per (sequence, KV head, query tile).
 * By default a query tile is a query block: the B = 128 positions
 * [I*B, (I+1)*B) with all g = num_q_heads/num_kv_heads heads of the KV group
 * (g*B packed rows). With query_tile_rows = 128 it is the paper's M-tile of
 * 128 packed rows: the Pt = 128/g positions [I*Pt, (I+1)*Pt) with all g
 * heads. Everything said of a query block holds for a tile: its rows lie in
 * key blocks Ja .. Jb (a single block when the prefix is a multiple of B,
 * since Pt divides B), and the rules below read with them. With g = 1 the
 * two tiles coincide.
 *
 * Layouts (row-major, innermost last)
 * -----------------------------------
 *   q, out       [total_tokens, num_q_heads, head_dim]; sequence b occupies
 *                token rows cu_seqlens[b] .. cu_seqlens[b+1]-1.
 *   k_cache,     page_size > 0: a token pool [num_slots, num_kv_heads,
 *   v_cache      head_dim]; key j (0 <= j < L_kv) of sequence b is slot
 *                block_table[b][j / page_size] * page_size + j % page_size
 *                (Sec. 3.3, Eq. page). page_size == 0: contiguous
 *                [total_kv_tokens, num_kv_heads, head_dim], sequence b at
 *                rows cu_seqlens_k[b] .. cu_seqlens_k[b+1]-1 (cu_seqlens
 *                without a prefix).
 *   block_table  int32 [batch, max_pages_per_seq] (ignored when page_size == 0).
 *   cu_seqlens   int32 [batch + 1], cu_seqlens[0] == 0, non-decreasing:
 *                the query rows.
 *   cu_seqlens_k int32 [batch + 1] or NULL: the KV lengths, same rules;
 *                cu_seqlens_k[b+1] - cu_seqlens_k[b] >= the query length.
 *   q/k/v_scale  fp32 per head ([num_q_heads] / [num_kv_heads] / [num_kv_heads]);
 *                only read when dtype == FP2_FP8_E4M3 (the dequantised value
 *                is scale * code, Sec. 3.3 Eq. fp8; a per-tensor scale is the
 *                all-equal case).
 *   block_mask   uint8 [batch, num_kv_heads, nbq, nbk], nbq = ceil(max_seq_len
 *                / Pt) query tiles (Pt = B by default), nbk = ceil(max_kv_len /
 *                block_size) key blocks (nbk == nbq by default without a
 *                prefix). Entry (b, h, I, J):
 *                bit 0 = key block J is attended exactly by query block I of
 *                KV head h (kept); bit 1 = J is a forced block (sink, window,
 *                diagonal or recent). Zero for J > Ia and for blocks past the
 *                sequence.
 *   lse          fp32 [total_tokens, num_q_heads], natural-log log-sum-exp of
 *                the scaled logits (including the correction masses).
 *
 * Selection semantics (Sec. 3.1 Eq. (1)-(2) and Eq. select, Sec. 3.2)
 * ----------------------------------------------------------------------
 * For query block I (block_size positions x all g = num_q_heads/num_kv_heads
 * query heads of one KV head h) and key block J <= I, the block energy is
 *     E[I][J] = sum over rows r of block I of exp(scale * q_r . khat_J),
 * khat_J = the bf16 rounding (nearest, ties to even) of the mean of the
 * dequantised keys of block J. Block J is kept iff alpha == 0, or
 * E[I][J] >= alpha * max_J' E[I][J'], or J is forced: J < sink_blocks,
 * I - J < window_blocks, J == I, or J >= n_b - recent_blocks (n_b = key
 * blocks of sequence b; with a prefix I reads Ia here and below). With
 * mean_correction, every block J < I that is not kept adds
 * |B_J| * exp(scale * q . kbar_J) * vbar_J to the softmax numerator and
 * |B_J| * exp(scale * q . kbar_J) to its denominator (Sec. 3.2 Eq.
 * correction); kbar/vbar are the block means (stored in bf16 on the GPU; for
 * fp8 inputs the correction uses their e4m3 codes, e4m3(kbar / k_scale) and
 * e4m3(vbar / v_scale), on the fp8 matrix cores).
 *
 * fp8 (Sec. 3.3 Eq. fp8): scores are c_q c_k (q~ . k~) from the e4m3 codes;
 * the probabilities of kept keys are rounded to e4m3 as P~ = e4m3(2^8 *
 * exp(S - m)) before the value product, and the softmax denominator sums
 * those rounded P~ (so out is a convex combination of values); the 2^8 is
 * removed from lse. The reference m_c of the online softmax moves only when
 * a logit passes it by more than tau = 0.8 (base 2), so P~ lies in
 * [0, 2^8.8] (2^8.8 < 446, below 448, the largest e4m3 value); it moves in
 * whole steps k above the accumulators' reference, and the value products
 * lift P~ by 2^k through the MFMA scale operands. Scales must be positive and
 * finite.
 */
#ifndef FP2_H
#define FP2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FP2_OK = 0,
  FP2_EINVAL = 1,        /* a null or inconsistent argument */
  FP2_EUNSUPPORTED = 2,  /* a valid configuration the library does not cover */
  FP2_EWORKSPACE = 3,    /* workspace null or smaller than fp2_workspace_bytes */
  FP2_EHIP = 4           /* a HIP launch or runtime call failed */
} fp2_status_t;

typedef enum {
  FP2_BF16 = 0,          /* q, k, v in bfloat16 */
  FP2_FP8_E4M3 = 1       /* q, k, v in OCP float8 e4m3fn with per-head fp32 scales */
} fp2_dtype_t;

typedef struct {
  int32_t batch;              /* number of sequences, >= 0 */
  int32_t num_q_heads;        /* H_q, a multiple of num_kv_heads */
  int32_t num_kv_heads;       /* 1 <= H_kv <= 1024; g = H_q / H_kv must be 1, 2, 4 or 8 */
  int32_t head_dim;           /* d: must be 128 */
  int32_t block_size;         /* selection block B in tokens: must be 128 */
  int32_t page_size;          /* p >= 1 tokens per page, or 0 for contiguous KV */
  int32_t max_seq_len;        /* upper bound of every query length, <= 1048576 */
  int32_t max_pages_per_seq;  /* block_table row stride, >= ceil(max_kv_len / p) */
  float alpha;                /* threshold ratio >= 0 (0 keeps every causal block) */
  int32_t sink_blocks;        /* forced leading key blocks, >= 0 */
  int32_t window_blocks;      /* forced local band incl. the diagonal, >= 0 */
  int32_t recent_blocks;      /* forced trailing key blocks of the sequence, >= 0 */
  int32_t mean_correction;    /* 0 or 1 */
  float softmax_scale;        /* <= 0 selects 1/sqrt(head_dim) */
  int32_t dtype;              /* fp2_dtype_t */
  int32_t max_kv_len;         /* upper bound of every KV length (prefix + chunk);
                                 0 selects max_seq_len; else >= max_seq_len,
                                 <= 1048576 */
  int32_t kv_splits;          /* 0 = cost-balanced KV splits planned on the
                                 device; n in 1..32 = n parts for every
                                 (sequence, KV head, query block), 1 = none;
                                 see "KV splits" above */
  int32_t query_tile_rows;    /* selection tile: 0 = a query block of B
                                 positions with all g heads; 128 = one
                                 M-tile of 128 packed rows (128/g positions
                                 with all g heads); see "Query tiles" above */
  int32_t score_splits;       /* parts of a unit's query rows in the scoring:
                                 0 = automatic (calls with fewer units than
                                 half the compute units, i.e. short chunks,
                                 split each unit's rows over several
                                 workgroups and merge their block energies);
                                 n in 1..64 = at most n parts, 1 = none.
                                 Results depend on it through rounding only */
} fp2_params_t;

/* Bytes of workspace the entry points need for `params` (0 for a null or
 * invalid params). Covers the pooled key/value means, the kept-block lists
 * and their counts, the attention work plan with its work counter (rebuilt
 * by every call, so a workspace can be reused without clearing) and the
 * partial outputs of split units (520 bytes per packed query row: 34 MB for
 * kv_splits == 0, n x 520 bytes per packed row of the problem for n > 1),
 * which the row-split scoring also uses as its scratch before the attention
 * (it falls back to fewer parts when they do not fit). */
size_t fp2_workspace_bytes(const fp2_params_t* params);

/* Full prefill (Algorithm 1 of Sec. 3.4): block means, fused scoring and
 * selection, then attention over the kept blocks of every (sequence, KV head,
 * query block) with the mean correction for the pruned ones (Sec. 3.2-3.3).
 * Inputs: params, q, cu_seqlens (device), cu_seqlens_host (nullable host
 * copy, validated when given), cu_seqlens_k (device KV lengths, NULL = no
 * prefix), cu_seqlens_k_host (nullable host copy, validated with
 * cu_seqlens_host when given), k_cache, v_cache, block_table (device;
 * ignored if page_size == 0), q_scale/k_scale/v_scale (device; fp8 only,
 * else may be null). Outputs: out (bf16, always), lse (nullable), block_mask
 * (every entry written). Rows of out/lse outside [0, cu_seqlens[batch]) are
 * not touched. */
fp2_status_t fp2_prefill(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                         const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                         const int32_t* cu_seqlens_k_host, const void* k_cache, const void* v_cache,
                         const int32_t* block_table, const float* q_scale, const float* k_scale,
                         const float* v_scale, void* out, float* lse, uint8_t* block_mask,
                         void* workspace, size_t workspace_bytes, void* stream);

/* The index stage alone (Sec. 3.1, Eq. fused_score and Eq. select; Algorithm
 * 1 steps 1-5): writes every entry of block_mask and leaves the pooled means
 * and kept-block lists in the workspace. Arguments as for fp2_prefill. */
fp2_status_t fp2_estimate(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                          const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                          const int32_t* cu_seqlens_k_host, const void* k_cache,
                          const void* v_cache, const int32_t* block_table, const float* q_scale,
                          const float* k_scale, const float* v_scale, uint8_t* block_mask,
                          void* workspace,
                          size_t workspace_bytes, void* stream);

/* The attention stage alone (Sec. 3.2 Eq. correction, Sec. 3.3; the sparse
 * attention of Algorithm 1) under a caller-given mask: bit 0 of block_mask_in[b][h][I][J]
 * selects key block J for query block I (entries with J > Ia are ignored).
 * The caller should select the diagonal J == Ia of every valid block I: the
 * mask is not checked, and a row whose keys are all excluded (no selected
 * key at or before its position and no corrected block) gets an undefined
 * output. Recomputes the block means and the kept lists from the mask in
 * the workspace. Arguments as for fp2_prefill. */
fp2_status_t fp2_attend(const fp2_params_t* params, const void* q, const int32_t* cu_seqlens,
                        const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                        const int32_t* cu_seqlens_k_host, const void* k_cache, const void* v_cache,
                        const int32_t* block_table, const float* q_scale, const float* k_scale,
                        const float* v_scale, const uint8_t* block_mask_in, void* out, float* lse,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Block means of K and V (Sec. 3.2, the pooled statistics of Eq. correction;
 * the block means of Algorithm 1), dequantised for fp8. Here cu_seqlens are the KV
 * lengths (a prefix included) and blocks are counted over max_kv_len. khat
 * [batch, num_kv_heads, nbk, head_dim] receives the bf16 (nearest-even)
 * rounding of the key means, vbar the same layout for the value means;
 * entries of blocks past a sequence are zero. Needs no workspace. */
fp2_status_t fp2_pool(const fp2_params_t* params, const int32_t* cu_seqlens,
                      const int32_t* cu_seqlens_host, const void* k_cache, const void* v_cache,
                      const int32_t* block_table, const float* k_scale, const float* v_scale,
                      void* khat, void* vbar, void* stream);

/* Block means kept across calls (chunked prefill, prefix caching; Sec. 4
 * runs the sparse operator on every extend of a request): the pooled means of
 * a complete key block depend only on its tokens, so a serving engine can keep
 * them beside its paged KV cache and each call pools only the blocks that are
 * new or were incomplete before. One slot per key block of the pool:
 *   page_size p > 0: slot = page_id * ceil(p / 128) + offset / 128, where
 *     page_id = block_table[b][t / p] and offset = t % p for the block's first
 *     token t = 128 J, so a pool of P pages needs P * ceil(p / 128) slots;
 *   page_size == 0: slot = b * ceil(max_kv_len / 128) + J.
 * khat and vbar are bf16 [slots, num_kv_heads, head_dim], device, owned by the
 * caller, one pair per layer (the means are those of that layer's K/V).
 * pooled_blocks is device int32 [batch]: the leading key blocks of sequence b
 * whose slots already hold the means of the same tokens (written by an
 * earlier call); it is clamped to the sequence's complete blocks, so a block
 * that was partial then is pooled again. Blocks below it are copied from the
 * cache; every block pooled by the call is written to its slot. The arrays
 * must cover the slot of every page id that block_table holds (as k_cache and
 * v_cache cover its tokens); the library does not check them. */
typedef struct {
  void* khat;
  void* vbar;
  const int32_t* pooled_blocks;
} fp2_means_cache_t;

/* Slots a means cache needs for `params` and a pool of num_pages pages
 * (num_pages is ignored for contiguous KV); 0 for an invalid params or a
 * negative num_pages. */
size_t fp2_means_cache_slots(const fp2_params_t* params, int64_t num_pages);

/* fp2_prefill with a means cache (cache non-null, all three pointers
 * non-null, khat/vbar 16-byte aligned); results are bitwise those of
 * fp2_prefill whenever the cached slots hold the means of the same tokens. */
fp2_status_t fp2_prefill_cached(const fp2_params_t* params, const void* q,
                                const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                                const int32_t* cu_seqlens_k, const int32_t* cu_seqlens_k_host,
                                const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const float* q_scale,
                                const float* k_scale, const float* v_scale,
                                const fp2_means_cache_t* cache, void* out, float* lse,
                                uint8_t* block_mask, void* workspace, size_t workspace_bytes,
                                void* stream);

/* Entries of csr_indices that always suffice for fp2_mask_to_csr: two
 * 64-token key tiles per key block and query tile, 2 * nbk * nbq * batch *
 * num_kv_heads (0 for an invalid params). */
size_t fp2_csr_capacity(const fp2_params_t* params);

/* The selection as a CSR index of 64-token key tiles (Sec. 3.3 Eq. csr;
 * the compaction of Algorithm 1, logical blocks expanded to B/64 = 2 physical
 * tiles per block): segment s = (b * num_kv_heads + h) * nbq + I, in block_mask row
 * order, owns csr_indices[csr_offsets[s] .. csr_offsets[s+1]), which lists in
 * ascending order the tiles j (keys 64j .. 64j+63 of sequence b) of every key
 * block J with bit 0 of block_mask[b][h][I][J] set and J <= Ia: 2J, and 2J+1
 * when 64(2J+1) < L_kv. Segments of query tiles past their sequence are
 * empty. Inputs: params, cu_seqlens / cu_seqlens_k (device; host copies
 * optional, validated when given), block_mask (device, the layout above).
 * Outputs (device): csr_offsets int32 [batch * num_kv_heads * nbq + 1]
 * (csr_offsets[0] = 0), csr_indices int32 [capacity], capacity >=
 * fp2_csr_capacity(params) (FP2_EINVAL otherwise). Uses the workspace of
 * fp2_workspace_bytes(params) bytes as scratch. */
fp2_status_t fp2_mask_to_csr(const fp2_params_t* params, const int32_t* cu_seqlens,
                             const int32_t* cu_seqlens_host, const int32_t* cu_seqlens_k,
                             const int32_t* cu_seqlens_k_host, const uint8_t* block_mask,
                             int32_t* csr_offsets, int32_t* csr_indices, size_t capacity,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Rate calibration: a measurement helper, not a step of the method. It runs
 * one fixed instruction loop on every compute unit (two workgroups of four
 * waves each, so two waves per SIMD, each wave with independent chains) and
 * sets *ops to the operations the launch performs, so that the caller's
 * timing of `stream` gives the rate this GPU sustains -- the measured
 * counterpart of the vendor peaks a roofline uses:
 *   FP2_CALIB_MFMA_BF16  v_mfma_f32_32x32x16_bf16 (the bf16 attention, the
 *                        correction and the block scoring), 32768 FLOP each;
 *   FP2_CALIB_MFMA_FP8   v_mfma_f32_32x32x64_f8f6f4 on e4m3 codes (the fp8
 *                        attention), 131072 FLOP each;
 *   FP2_CALIB_EXP        v_exp_f32 (the softmax and scoring exponentials),
 *                        64 exps each.
 * iters: loop trips per wave, 1 .. 2^24 (each trip is 4 MFMAs per wave, or
 * 32 exps per lane). sink: one device float, written only if a loop yields a
 * value it never does (it keeps the loop's results live). ops: host double.
 * FP2_EINVAL for an unknown kind, iters out of range or a null pointer. */
typedef enum {
  FP2_CALIB_MFMA_BF16 = 0,
  FP2_CALIB_MFMA_FP8 = 1,
  FP2_CALIB_EXP = 2
} fp2_calib_kind_t;
fp2_status_t fp2_calibrate(fp2_calib_kind_t kind, int32_t iters, float* sink, double* ops,
                           void* stream);

/* Measurement helper, not a step of the method: from this call on, the
 * entry points called on this host thread record the given HIP events
 * (hipEvent_t created by the caller; NULL = none) on the call's stream:
 * estimate_begin right before the block-means kernel and estimate_end right
 * after the scoring and selection kernels (fp2_prefill, fp2_prefill_cached,
 * fp2_estimate), attend_begin right before the attention kernel and
 * attend_end right after it (fp2_prefill, fp2_prefill_cached, fp2_attend).
 * Each call records each event once, so the elapsed time between a pair is
 * the duration of those kernels in that call; time K calls with K pairs set
 * between the calls. Pass all NULL to stop. Events come in begin/end pairs
 * (FP2_EINVAL otherwise). Nothing else about a call changes. */
fp2_status_t fp2_time_kernels(void* estimate_begin, void* estimate_end, void* attend_begin,
                              void* attend_end);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fp2_prefill with its scratch memory in a static device array of the
 * library, FP2_NOALLOC_SCRATCH_BYTES (96 MiB) on each GPU the library runs
 * on, held until the process ends, instead of a caller workspace. Arguments,
 * results and errors otherwise as fp2_prefill (the same kernels, so the same
 * outputs bit for bit). Returns FP2_EWORKSPACE when fp2_workspace_bytes(params)
 * exceeds the array: 128K-token sequences with 8 KV heads need about 69 MiB,
 * and the need grows with batch * num_kv_heads * max_seq_len^2 / 2^14 bytes
 * (the kept lists). The library allocates nothing for this call; the first
 * call on a device resolves the array's address there (make that first call
 * outside a graph capture). Every call on a GPU uses that GPU's one array,
 * which keeps the last call's contents: calls that overlap on one GPU (other
 * streams or host threads) race; calls in order on one stream are safe, since
 * each call's kernels rebuild everything they read from it. */
#define FP2_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)
fp2_status_t fp2_prefill_noalloc(const fp2_params_t* params, const void* q,
                                 const int32_t* cu_seqlens, const int32_t* cu_seqlens_host,
                                 const int32_t* cu_seqlens_k, const int32_t* cu_seqlens_k_host,
                                 const void* k_cache, const void* v_cache,
                                 const int32_t* block_table, const float* q_scale,
                                 const float* k_scale, const float* v_scale, void* out,
                                 float* lse, uint8_t* block_mask, void* stream);

/* Static description of a status code. */
const char* fp2_status_str(fp2_status_t status);

/* One-line reason for the last non-OK status returned on the calling thread
 * ("" if none). The pointer stays valid until the next call on that thread. */
const char* fp2_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FP2_H */

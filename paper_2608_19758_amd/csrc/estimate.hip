// Fused block scoring, max-based thresholding and kept-list compaction
// (Sec. 3.1 Eq. (1)-(2), Eq. fused_score, Eq. select; the scoring, thresholding
// and compaction of Algorithm 1).
//
// A persistent grid (one 8-wave workgroup per compute unit, two for the
// one-chunk variant below) deals the units
// (sequence b, KV head h, query block I) round-robin, heaviest (largest I)
// first. The query rows of block I are the g*B packed rows of Eq. packgqa
// (position I*B + r/g, head h*g + r%g). They stream through LDS in pairs of
// 32-row tiles (one barrier per pair), the global loads one pair ahead; each
// wave keeps four (or, for calls with fewer key blocks, one) 32-wide chunks of
// pooled keys khat in registers (the MFMA B operand) and computes S = Q khat^T with v_mfma_f32_32x32x16_bf16
// (fp32 accumulation). Lane l of the accumulator owns key block J = chunk +
// l%32 and 16 query rows, so the row sum of exp2(S * scale*log2e - m) for its
// block is a per-lane running sum with a per-lane offset m (the role of the
// per-(I,J) maximum of Eq. (1), moved only when a tile's sum would leave a
// safe range; no cross-lane traffic). At the end the two lane halves are
// merged into ell_J = log2 E_J. Calls with few units split a unit's tiles
// over several workgroups (EllParts) and merge the parts in select_kernel.
//
// Selection (Eq. select): J is kept iff alpha == 0, ell_J >= max_J ell +
// log2(alpha), or J is forced (sink, window incl. diagonal, recent). The mask
// row is written in full (zeros past I) and the kept blocks are compacted in
// ascending order with wave ballots into the per-row list of the workspace.
// With a prefix KV (the queries are the last keys of the sequence) the key
// blocks are those of the KV tokens, and the rows of query tile I lie in key
// blocks Ja .. Ia: blocks up to Ia are scored, the band Ja .. Ia is forced
// (the diagonal) and the window counts back from Ia.
//
// Precision: fp8 queries are widened to bf16 exactly, the per-head fp8 scale
// is applied in fp32 after the MFMA, and exponentials use the hardware
// v_exp_f32; block energies match the fp64 definition to ~1e-6 relative.
#include <algorithm>
#include <type_traits>

#include "kernels.h"

namespace fp2 {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
// 32-block chunks of pooled keys per wave: 4 (a pass covers 1024 key blocks,
// one workgroup per CU), or 1 (a pass covers 256), whose smaller register
// budget admits two workgroups per CU: the items of one then run beside
// those of the other, hiding each item's load and selection latencies, at
// the price of streaming a unit's Q tiles once per pass.
constexpr int kChunksPerWave = 4;
constexpr int kQRow = 17;                                  // LDS row stride of a Q tile, 16-byte slots
constexpr int kBufferWord3 = 0x00020000;                   // buffer resource word 3 (gfx9: raw 32-bit data)

// Row split of the scoring for calls with few units (short chunks): part u
// of parts.n scores the unit's 32-row tiles [u ceil(T/n), ...) and writes
// its block log2-energies to buf (one row of nbk floats per item);
// select_kernel merges them per unit. parts.n == 1: one item per unit, the
// selection in the same kernel.
struct EllParts {
  float* buf;
  int n;
};

// Selection of one unit from its block log2-energies ell[0 .. Ia] in LDS
// (Eq. select): J is kept iff alpha == 0, ell_J >= max ell + log2 alpha, or
// J is forced (sink, window counted back from Ia, the band Ja .. Ia, recent).
// Writes the mask row in full and the ascending kept list with its count.
template <class Prob>   // Problem, or the kernel-argument copy of it
__device__ void select_unit(const Prob& p, const float* ell, int Ia, int Ja, int nk,
                            uint8_t* mrow, int32_t* kidx, int32_t* cnt, float* redf, int* redi,
                            int tid) {
  const int lane = tid & 63, w = tid >> 6;
  float mu = -INFINITY;
  for (int J = tid; J <= Ia; J += kThreads) mu = fmaxf(mu, ell[J]);
  mu = wave_max(mu);
  if (lane == 0) redf[w] = mu;
  __syncthreads();
  mu = redf[0];
#pragma unroll
  for (int k = 1; k < kWaves; ++k) mu = fmaxf(mu, redf[k]);
  const bool keep_all = p.alpha == 0.f;
  const float thr = keep_all ? -INFINITY : mu + fast_log2(p.alpha);

  int base = 0;
  for (int J0 = 0; J0 < p.nbk; J0 += kThreads) {
    const int J = J0 + tid;
    const bool valid = J <= Ia;
    const bool forced = valid && (J < p.sink || Ia - J < p.window || J >= Ja || J >= nk - p.recent);
    const bool keep = valid && (keep_all || forced || ell[J] >= thr);
    if (J < p.nbk) mrow[J] = (uint8_t)((keep ? 1 : 0) | (forced ? 2 : 0));
    if (J0 <= Ia) {
      const uint64_t bal = __ballot(keep);
      const int pre = __popcll(bal & ((1ull << lane) - 1ull));
      __syncthreads();
      if (lane == 0) redi[w] = __popcll(bal);
      __syncthreads();
      int wpre = 0, tot = 0;
#pragma unroll
      for (int k = 0; k < kWaves; ++k) {
        wpre += k < w ? redi[k] : 0;
        tot += redi[k];
      }
      if (keep) kidx[base + wpre + pre] = J;
      base += tot;
    }
  }
  if (tid == 0) *cnt = base;
}

// (the second bound is waves per SIMD: four, i.e. two workgroups per CU, for
// the one-chunk variant, so that it keeps within 128 registers)
template <int FP8, int G, int CPW>
__global__ __launch_bounds__(kThreads, CPW == 1 ? 4 : 2) void estimate_kernel(Problem p0, Pooled pooled,
                                                            uint8_t* __restrict__ mask,
                                                            KeptLists kl, EllParts parts) {
  extern __shared__ float ell[];            // [nbk] block log2-energies of this row
  __shared__ uint4 qt[2][64 * kQRow];       // Q tile pairs (double buffer): 2 x 32 rows x 16 chunks of 8 bf16
  __shared__ float redf[kWaves];
  __shared__ int redi[kWaves];

  const int nbh = p0.batch * p0.hkv;
  const int nitems = p0.nbmax * nbh * parts.n;

  // Persistent workgroups, items dealt round-robin in order of decreasing
  // query block: the cost of an item is proportional to (I + 1), so every
  // workgroup gets an almost equal share. Even workgroups take their items
  // heaviest first and odd ones lightest first (the same items, reversed),
  // so that the two workgroups sharing a CU are rarely both on units whose
  // few key-block chunks leave most of their waves idle.
  const int nmine = (nitems - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
#pragma unroll 1
  for (int jj = 0; jj < nmine; ++jj) {
  const int item = (int)blockIdx.x + ((blockIdx.x & 1) ? nmine - 1 - jj : jj) * (int)gridDim.x;
  // Opaque copies of the thread index and of the argument block (the first
  // kernel argument, at offset 0 of the argument segment): values derived
  // from them are recomputed per item instead of living across the loop.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  typedef const __attribute__((address_space(4))) Problem KProblem;
  KProblem* pk = (KProblem*)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(pk));
  KProblem& p = *pk;

  const int uidx = item / parts.n, part = item - uidx * parts.n;   // unit, row-tile part
  const int I = p.nbmax - 1 - uidx / nbh;
  const int bh = uidx % nbh;
  const int b = bh / p.hkv, h = bh % p.hkv;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: branches on it are scalar
  const int half = lane >> 5, l32 = lane & 31;
  const int64_t tok0 = ld_uniform(p.cu, b);
  const int L = ld_uniform(p.cu, b + 1) - (int)tok0;
  const int n = (L + p.qtile - 1) / p.qtile;   // query tiles of the sequence
  // KV tokens and key blocks; the rows of query tile I lie in key blocks
  // Ja .. Ib (Ib = Ja + 1 when the tile straddles a key-block boundary)
  const int Lk = ld_uniform(p.cuk, b + 1) - ld_uniform(p.cuk, b);
  const int nk = (Lk + kBlock - 1) / kBlock;
  const int Ja = (Lk - L + I * p.qtile) / kBlock;
  const int Ia = (Lk - L + min(L, (I + 1) * p.qtile) - 1) / kBlock;   // last visible key block
  const int64_t row = ((int64_t)b * p.hkv + h) * p.nbmax + I;
  uint8_t* mrow = mask + row * p.nbk;

  if (I >= n) {
    if (parts.n == 1) {   // (select_kernel clears the row in the split mode)
      for (int J = tid; J < p.nbk; J += kThreads) mrow[J] = 0;
      if (tid == 0) kl.cnt[row] = 0;
    }
    continue;
  }

  const int npos = min(p.qtile, L - I * p.qtile);
  const int nrows = npos * G;
  const int ntiles = (nrows + 31) / 32;
  // this item's 32-row tiles [tlo, thi): all of them, or part `part` of
  // parts.n; energies of a part go to parts.buf, one row of nbk per item
  const int tper = (ntiles + parts.n - 1) / parts.n;
  const int tlo = min(ntiles, part * tper), thi = min(ntiles, tlo + tper);
  float* pell = parts.buf + (int64_t)item * p.nbk;
  if (tlo >= thi) {   // an empty part adds nothing
    for (int J = tid; J <= Ia; J += kThreads) pell[J] = -INFINITY;
    continue;
  }

  // Row r = 8i + 4*half + j of a 32-row tile has head offset (4*half + j) % G.
  float cs[4];
  if constexpr (FP8) {
    float sc[G];
#pragma unroll
    for (int k = 0; k < G; ++k) sc[k] = p.scale_log2 * ld_uniform(p.q_scale, h * G + k);
#pragma unroll
    for (int j = 0; j < 4; ++j) cs[j] = half ? sc[(4 + j) % G] : sc[j % G];
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) cs[j] = p.scale_log2;
  }

  // Pooled keys through a buffer resource over this unit's blocks 0 .. Ia:
  // blocks past its last one read as zero keys, without a branch.
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(pooled.khat + ((int64_t)b * p.hkv + h) * p.nbk * kHeadDim), (short)0,
      (Ia + 1) * kHeadDim * 2, kBufferWord3);
  // Q rows of this unit as a buffer resource (rows past the tile read as zero).
  constexpr int esz = FP8 ? 1 : 2;
  const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)((const char*)p.q + (tok0 + (int64_t)I * p.qtile) * p.hq * kHeadDim * esz), (short)0,
      npos * p.hq * kHeadDim * esz, kBufferWord3);

  // This thread's 16 bytes of Q tile t (bf16: row tid/16, chunk tid%16;
  // fp8: threads < 256, row tid/8, 16 codes tid%8), zero past the block.
  // Packed row t*32 + r is position t*(32/G) + r/G, head h*G + r%G (G
  // divides 32), so the byte offset is a per-thread constant plus t times
  // the tile stride. fp8 threads past the 256 that cover a tile start past
  // the buffer (2^30, so that no tile's offset wraps): they read zero.
  const int qr = FP8 ? tid >> 3 : tid >> 4;
  const int qoff0 = !FP8 || tid < 256
                        ? ((qr / G) * p.hq + h * G + qr % G) * (kHeadDim * esz) + (FP8 ? tid & 7 : tid & 15) * 16
                        : 0x40000000;
  const int qtstride = (32 / G) * p.hq * kHeadDim * esz;
  auto qload = [&](int t) -> uint4 {
    // tiles past the item's last fetch nothing (an offset past the buffer reads zero)
    const int off = t < thi ? qoff0 + t * qtstride : 0x7ffffff0;
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(qrs, off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
  };
  // Store it into LDS buffer qb (fp8 codes widened to bf16, exact). Rows are
  // kQRow 16-byte slots apart: a lane's eight reads of its row then share
  // one base address, and 16 lanes reading 16 bytes each cover all banks.
  auto qstore = [&](uint4* qb, uint4 v) {
    if (!FP8) {
      const int r = tid >> 4, c = tid & 15;
      qb[r * kQRow + c] = v;
    } else if (tid < 256) {
      const int r = tid >> 3, c8 = tid & 7;
      const uint2 a = e4m3x4_to_bf16(v.x), b2 = e4m3x4_to_bf16(v.y);
      const uint2 c2 = e4m3x4_to_bf16(v.z), d = e4m3x4_to_bf16(v.w);
      qb[r * kQRow + 2 * c8] = make_uint4(a.x, a.y, b2.x, b2.y);
      qb[r * kQRow + 2 * c8 + 1] = make_uint4(c2.x, c2.y, d.x, d.y);
    }
  };

  constexpr int kGroup = kWaves * CPW * 32;   // key blocks per pass
  for (int grp = 0; grp <= Ia; grp += kGroup) {
    bf16x8_t kf[CPW][8];
    float m[CPW], E[CPW];
    bool act[CPW];
    // 32-block chunks of this wave in this group that hold a visible block
    // (chunk c of wave w starts at block grp + 32 (w + 8 c)); a wave without
    // any only takes part in the barriers
    const int ncw = min(CPW, max(0, ((Ia - grp) / 32 - w + kWaves) / kWaves));
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      const int J0 = grp + 32 * (w + kWaves * c);
      act[c] = J0 <= Ia;
      m[c] = -INFINITY;
      E[c] = 0.f;
      const int J = J0 + l32;
      if (act[c]) {   // (an inactive chunk is never scored)
#pragma unroll
        for (int ds = 0; ds < 8; ++ds)
          kf[c][ds] = __builtin_bit_cast(
              bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(krs, J * (kHeadDim * 2) + 32 * ds + 16 * half, 0, 0));
      }
    }

    // Q tiles stream through two LDS buffers of two tiles each, one barrier
    // per pair; the global loads of the next pair are in flight while a pair
    // is scored. Only the last tile can be partial: it runs as a separate
    // instance of the tile body, so the row validity tests stay out of the
    // full tiles. With one chunk per wave a pair of full tiles is scored
    // together, the second tile's MFMAs issued ahead of the first's fold.
    uint4 qa_next = qload(tlo), qa_next2 = qload(tlo + 1);
    auto tile = [&](const uint4* qb, int t, auto partial, auto paired) {
      constexpr bool kPartial = decltype(partial)::value;
      constexpr bool kPair = decltype(paired)::value;   // tiles t and t+1, both full, one chunk

      // Q operand ds of this lane, read from LDS where it is used (two reads
      // in flight ahead of the MFMAs, not the tile's eight held in registers)
      auto qa = [&](const uint4* q, int ds) { return __builtin_bit_cast(bf16x8_t, q[l32 * kQRow + 2 * ds + half]); };
      const int rbase = t * 32 + 4 * half;   // first of this lane's 16 rows

      // Scores of chunk c (the other wave of the SIMD runs its vector work
      // while these MFMAs execute).
      auto score = [&](int c, const uint4* q) -> f32x16_t {
        f32x16_t acc = {};
#pragma unroll
        for (int ds = 0; ds < 8; ++ds)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa(q, ds), kf[c][ds], acc, 0, 0, 0);
        return acc;
      };
      // Fold one chunk's scores into its running (m, E): rows of head
      // offset j carry the scale cs[j] (> 0). Rows past the block (partial
      // tile only) are set to -inf first: they add exp2(-inf) = 0. Once m is
      // set, the sum is taken against it as it stands (E only has to stay
      // finite, so m need not be the exact running maximum); only a tile
      // whose sum exceeds 2^64 moves m to its maximum and is summed again.
      auto fold = [&](int c, f32x16_t& acc) {
        // raised wave priority while folding: the SIMD's arbiter then favours
        // the vector work of a folding wave over the issue of other waves,
        // whose MFMA chains keep the matrix core busy meanwhile
        __builtin_amdgcn_s_setprio(1);
        if constexpr (kPartial) {
          const int rem = nrows - rbase;   // this lane's rows 8i + j < rem lie in the block
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              acc[4 * i + j] = 8 * i + j < rem ? acc[4 * i + j] : -INFINITY;
        }
        auto sum_at = [&](float nb) -> float {
          float s4[4];                                  // four independent partial sums
#pragma unroll
          for (int j = 0; j < 4; ++j) s4[j] = fast_exp2(fmaf(acc[j], cs[j], nb));
#pragma unroll
          for (int i = 1; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) s4[j] += fast_exp2(fmaf(acc[4 * i + j], cs[j], nb));
          return (s4[0] + s4[1]) + (s4[2] + s4[3]);
        };
        float e = m[c] == -INFINITY ? INFINITY : sum_at(-m[c]);
        if (!(e <= 0x1p64f)) {   // no m yet, or the sum grew too large: move m up
          float g[4];
#pragma unroll
          for (int j = 0; j < 4; ++j)
            g[j] = fmaxf(fmaxf(acc[j], acc[4 + j]), fmaxf(acc[8 + j], acc[12 + j])) * cs[j];
          const float mn = fmaxf(m[c], fmaxf(fmaxf(g[0], g[1]), fmaxf(g[2], g[3])));
          if (mn > m[c]) {
            E[c] *= fast_exp2(m[c] - mn);
            m[c] = mn;
          }
          e = mn == -INFINITY ? 0.f : sum_at(-mn);   // no valid row yet: every term is 0
        }
        E[c] += e;
        __builtin_amdgcn_s_setprio(0);
      };
      // the wave's chunks 0 .. NC-1 that hold visible blocks (NC a compile-time
      // count, so the scores of chunk c+1 are issued to the matrix cores
      // before chunk c is folded on the vector ALUs); blocks past the unit's
      // last one score zero keys and are dropped at the end
      auto run = [&](auto nc) {
        constexpr int NC = decltype(nc)::value;
        if constexpr (kPair) {   // the second tile's MFMAs issued before the first tile's fold
          f32x16_t a0 = score(0, qb), a1 = score(0, qb + 32 * kQRow);
          fold(0, a0);
          fold(0, a1);
          return;
        }
        f32x16_t acc = score(0, qb);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          f32x16_t nxt;
          if (c + 1 < NC) nxt = score(c + 1, qb);
          fold(c, acc);
          if (c + 1 < NC) acc = nxt;
        }
      };
      switch (ncw) {
        case 0: break;
        case 1: run(std::integral_constant<int, 1>{}); break;
        case 2: if constexpr (CPW >= 2) run(std::integral_constant<int, 2>{}); break;
        case 3: if constexpr (CPW >= 3) run(std::integral_constant<int, 3>{}); break;
        default: if constexpr (CPW >= 4) run(std::integral_constant<int, 4>{}); break;
      }
    };
    const int nfull = nrows >> 5;
    for (int t0 = tlo; t0 < thi; t0 += 2) {
      uint4* buf = qt[((t0 - tlo) >> 1) & 1];
      __builtin_amdgcn_s_setprio(1);   // the staging waves hold up the barrier below
      qstore(buf, qa_next);
      qstore(buf + 32 * kQRow, qa_next2);
      __builtin_amdgcn_s_setprio(0);
      __syncthreads();   // tiles t0, t0+1 visible; every wave is done with the pair before
      qa_next = qload(t0 + 2);
      qa_next2 = qload(t0 + 3);
      if (CPW == 1 && t0 + 1 < nfull && t0 + 1 < thi) {
        tile(buf, t0, std::false_type{}, std::true_type{});
      } else {
        for (int k = 0; k < 2 && t0 + k < thi; ++k) {
          if (t0 + k < nfull)
            tile(buf + k * 32 * kQRow, t0 + k, std::false_type{}, std::false_type{});
          else
            tile(buf + k * 32 * kQRow, t0 + k, std::true_type{}, std::false_type{});
        }
      }
    }

    // merge the two lane halves (same key block, different rows)
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      if (!act[c]) continue;
      const float m2 = __shfl_xor(m[c], 32, 64);
      const float E2 = __shfl_xor(E[c], 32, 64);
      const float M = fmaxf(m[c], m2);
      float e1 = m[c] == -INFINITY ? 0.f : E[c] * fast_exp2(m[c] - M);
      float e2 = m2 == -INFINITY ? 0.f : E2 * fast_exp2(m2 - M);
      const int J = grp + 32 * (w + kWaves * c) + l32;
      if (half == 0 && J <= Ia) {
        const float v = M + fast_log2(e1 + e2);
        if (parts.n > 1)
          pell[J] = v;
        else
          ell[J] = v;
      }
    }
    __syncthreads();   // every wave is done with the Q tile buffers and ell of this group
  }

  // ---- selection (Eq. select), or the part's energies for select_kernel
  if (parts.n > 1) continue;
  select_unit(p, ell, Ia, Ja, nk, mrow, kl.idx + row * p.nbk, kl.cnt + row, redf, redi, tid);
  }
}

// Merge of the parts' block energies (log-sum-exp over the parts) and the
// selection, one workgroup per unit.
__global__ __launch_bounds__(kThreads) void select_kernel(Problem p, uint8_t* __restrict__ mask,
                                                          KeptLists kl, EllParts parts) {
  extern __shared__ float ell[];
  __shared__ float redf[kWaves];
  __shared__ int redi[kWaves];
  const int nbh = p.batch * p.hkv;
  const int uidx = blockIdx.x;
  const int I = p.nbmax - 1 - uidx / nbh;
  const int bh = uidx % nbh;
  const int b = bh / p.hkv, h = bh % p.hkv;
  const int tid = threadIdx.x;
  const int L = p.cu[b + 1] - p.cu[b];
  const int n = (L + p.qtile - 1) / p.qtile;
  const int64_t row = ((int64_t)b * p.hkv + h) * p.nbmax + I;
  uint8_t* mrow = mask + row * p.nbk;
  if (I >= n) {
    for (int J = tid; J < p.nbk; J += kThreads) mrow[J] = 0;
    if (tid == 0) kl.cnt[row] = 0;
    return;
  }
  const int Lk = p.cuk[b + 1] - p.cuk[b];
  const int nk = (Lk + kBlock - 1) / kBlock;
  const int Ja = (Lk - L + I * p.qtile) / kBlock;
  const int Ia = (Lk - L + min(L, (I + 1) * p.qtile) - 1) / kBlock;
  const float* pe = parts.buf + (int64_t)uidx * parts.n * p.nbk;
  for (int J = tid; J <= Ia; J += kThreads) {
    // running log-sum-exp over the parts, eight loads in flight at a time
    float M = -INFINITY, e = 0.f;
    for (int u0 = 0; u0 < parts.n; u0 += 8) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k)
        v[k] = u0 + k < parts.n ? pe[(int64_t)(u0 + k) * p.nbk + J] : -INFINITY;
      float mk = v[0];
#pragma unroll
      for (int k = 1; k < 8; ++k) mk = fmaxf(mk, v[k]);
      const float Mn = fmaxf(M, mk);
      if (Mn == -INFINITY) continue;
      e = M == -INFINITY ? 0.f : e * fast_exp2(M - Mn);
#pragma unroll
      for (int k = 0; k < 8; ++k) e += fast_exp2(v[k] - Mn);
      M = Mn;
    }
    ell[J] = M == -INFINITY ? M : M + fast_log2(e);
  }
  __syncthreads();
  select_unit(p, ell, Ia, Ja, nk, mrow, kl.idx + row * p.nbk, kl.cnt + row, redf, redi, tid);
}

// Kept lists from a caller-given mask (bit 0), ascending; one workgroup per row.
__global__ __launch_bounds__(256) void compact_kernel(Problem p, const uint8_t* __restrict__ mask,
                                                      KeptLists kl) {
  __shared__ int redi[4];
  const int nbh = p.batch * p.hkv;
  const int I = p.nbmax - 1 - (int)(blockIdx.x / nbh);
  const int bh = blockIdx.x % nbh;
  const int b = bh / p.hkv, h = bh % p.hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int L = p.cu[b + 1] - p.cu[b];
  const int n = (L + p.qtile - 1) / p.qtile;
  // last key block visible to tile I (that of its last row)
  const int Ia = (p.cuk[b + 1] - p.cuk[b] - L + min(L, (I + 1) * p.qtile) - 1) / kBlock;
  const int64_t row = ((int64_t)b * p.hkv + h) * p.nbmax + I;
  if (I >= n) {
    if (tid == 0) kl.cnt[row] = 0;
    return;
  }
  const uint8_t* mrow = mask + row * p.nbk;
  int32_t* kidx = kl.idx + row * p.nbk;
  int base = 0;
  for (int J0 = 0; J0 <= Ia; J0 += 256) {
    const int J = J0 + tid;
    const bool keep = J <= Ia && (mrow[J] & 1);
    const uint64_t bal = __ballot(keep);
    const int pre = __popcll(bal & ((1ull << lane) - 1ull));
    __syncthreads();
    if (lane == 0) redi[w] = __popcll(bal);
    __syncthreads();
    int wpre = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      wpre += k < w ? redi[k] : 0;
      tot += redi[k];
    }
    if (keep) kidx[base + wpre + pre] = J;
    base += tot;
  }
  if (tid == 0) kl.cnt[row] = base;
}

template <int FP8>
hipError_t launch_est_dt(const Problem& p, const Pooled& pooled, uint8_t* mask, KeptLists kl,
                         float* scratch, size_t scratch_floats, hipStream_t s) {
  const int cus = device_compute_units();
  if (cus <= 0) return hipErrorInvalidDevice;
  const int64_t units = (int64_t)p.nbmax * p.batch * p.hkv;
  // few units (short chunks): split their rows so that the grid covers the
  // CUs, if the scratch holds one energy row per item
  EllParts parts{scratch, 1};
  const int tiles = (p.g * p.qtile + 31) / 32;
  if (scratch && (p.ssplits > 1 || (p.ssplits == 0 && units * 2 <= cus))) {
    int n = (int)std::min<int64_t>(tiles, p.ssplits > 0 ? p.ssplits : (cus + units - 1) / units);
    while (n > 1 && (size_t)(units * n) * (size_t)p.nbk > scratch_floats) --n;
    parts.n = std::max(1, n);
  }
  // One chunk per wave (8 x 32 key blocks per pass, two workgroups per CU)
  // up to 1024 key blocks: the latency hidden by the second workgroup
  // outweighs the Q tiles streamed again for every pass (measured at 128K,
  // against four chunks per wave: g = 4 0.83 -> 0.79 ms, g = 8 1.40 -> 1.36
  // ms fp8 and 1.53 -> 1.43 ms bf16).
  const bool small = p.nbk <= 4 * kWaves * 32;
  const unsigned grid = (unsigned)std::min<int64_t>(units * parts.n, (int64_t)cus * (small ? 2 : 1));
  const size_t smem = (size_t)p.nbk * sizeof(float);
  auto go = [&](auto kern) { kern<<<grid, kThreads, smem, s>>>(p, pooled, mask, kl, parts); };
  switch (p.g * (small ? -1 : 1)) {
    case 1: go(estimate_kernel<FP8, 1, kChunksPerWave>); break;
    case 2: go(estimate_kernel<FP8, 2, kChunksPerWave>); break;
    case 4: go(estimate_kernel<FP8, 4, kChunksPerWave>); break;
    case 8: go(estimate_kernel<FP8, 8, kChunksPerWave>); break;
    case -1: go(estimate_kernel<FP8, 1, 1>); break;
    case -2: go(estimate_kernel<FP8, 2, 1>); break;
    case -4: go(estimate_kernel<FP8, 4, 1>); break;
    case -8: go(estimate_kernel<FP8, 8, 1>); break;
    default: return hipErrorInvalidValue;
  }
  if (parts.n > 1) select_kernel<<<(unsigned)units, kThreads, smem, s>>>(p, mask, kl, parts);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_estimate(const Problem& p, const Pooled& pooled, uint8_t* mask, KeptLists kl,
                           hipStream_t s, float* scratch, size_t scratch_floats) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  return p.fp8 ? launch_est_dt<1>(p, pooled, mask, kl, scratch, scratch_floats, s)
               : launch_est_dt<0>(p, pooled, mask, kl, scratch, scratch_floats, s);
}

hipError_t launch_compact(const Problem& p, const uint8_t* mask, KeptLists kl, hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  const unsigned grid = (unsigned)p.nbmax * p.batch * p.hkv;
  compact_kernel<<<grid, 256, 0, s>>>(p, mask, kl);
  return hipGetLastError();
}

}  // namespace fp2

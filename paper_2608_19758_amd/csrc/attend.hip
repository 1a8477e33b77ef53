// Sparse attention over the kept key blocks with the mean correction
// (Sec. 3.2 Eq. correction, Sec. 3.3; the sparse attention of Algorithm 1).
//
// Work unit: (sequence b, KV head h, query block I) of the packed query rows
// of Eq. packgqa. A work item is a slice of 32*W of the g*B packed rows of a
// unit, taken by a workgroup of W waves (W = 8, or 4 for units of 128 packed
// rows: g = 1, or 128-row query tiles), so one K/V tile in LDS serves all g
// query heads of the group. The grid is persistent: one 8-wave workgroup per
// compute unit (its LDS ring admits one), or two 4-wave workgroups on half
// the ring each, so that every SIMD runs two waves; each takes items from an
// atomic counter in order of decreasing query block (heaviest first), so the
// run time of an item never holds up the dispatch of others.
//
// The key sequence of a unit is a list of 64-key steps: both halves of every
// kept block, walked from the last kept index down (Eq. csr), then the pooled
// means of the pruned blocks J < I, 64 per step (the correction). Steps run
// through a ring of LDS stages (128 KiB: 4 bf16 stages or 8 fp8 stages;
// half that for 4-wave workgroups): the
// rows of step s+NST-1 are copied straight from the page-addressed pool
// (Eq. page) into LDS with global_load_lds_dwordx4 while step s is computed,
// with one workgroup barrier per step. The copy addresses come from small LDS
// tables filled once per chunk of steps (kept block index and its page-table
// entries, or the compacted list of pruned blocks), read one step ahead, so
// nothing in the loop waits on a global load.
//
// Per step:
//  - S^T = K Q^T on the matrix cores (A = key rows from LDS, B = the wave's
//    32 query rows held in registers). Lane l then owns query l%32 and 16
//    keys per 32-key subtile, so the row maximum of the online softmax needs
//    one exchange with lane l^32 (v_permlane32_swap);
//  - O^T += V^T P^T: the probabilities go straight from the S^T accumulators
//    into the B operand, and V^T comes from LDS through the gfx950
//    transposing reads ds_read_b64_tr_b16 / _b8 (no transpose pass).
// fp8 (OCP e4m3fn) uses v_mfma_f32_32x32x64_f8f6f4 on the raw codes; the
// per-head scales c_q c_k are applied to the fp32 scores, the probabilities
// are stored as e4m3(2^8 * exp(S - m)) (range [0, 2^(8 + tau)] with the lazy
// rescale below, tau = 0.8: at most 446 < 448) and the denominator
// sums those stored values (Sec. 3.3 Eq. fp8); c_v is applied in the
// epilogue and the 2^8 is removed from the LSE. Within a step the two waves
// of a SIMD overlap each other's matrix and vector work; the vector issue
// count per step is what bounds the fp8 loop, so the softmax is kept lean
// (masking only on the diagonal and last correction steps, constants held
// in registers across steps).
// bf16 uses v_mfma_f32_32x32x16_bf16. Correction steps use the pooled means
// as keys and values, logits shifted by log2|B_J| = 7 (Sec. 3.2
// implementation paragraph): for bf16 the bf16 means khat_J, vbar_J with bf16
// MFMA; for fp8 their e4m3 codes (khat_J / c_k, vbar_J / c_v, quantized as
// Sec. 4 quantizes the pooled statistics under fp8) with the same fp8 steps
// as the kept keys.
//
// Prefix KV (chunked prefill, prefix caching): the queries of a sequence may
// be the last L_q of its L_kv keys. Keys, key blocks and the pooled means are
// then those of the L_kv tokens; the rows of query block (or tile) I lie in
// key blocks Ja .. Jb (two blocks when the prefix is not a multiple of B). The
// causal mask applies to the kept blocks J >= Ja and the correction to the
// pruned J < Ja, with absolute positions; query rows and the LSE are indexed
// by the local position.
#include <algorithm>
#include <utility>

#include "kernels.h"

namespace fp2 {

namespace {

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kStep = 64;            // keys per pipeline step
// LDS ring in 16-byte slots: 128 KiB for one 8-wave workgroup per CU; a
// 4-wave workgroup (128-row items) takes 64 KiB so that two of them share a
// CU and every SIMD still runs two waves (4 fp8 / 2 bf16 stages).
constexpr int ring_u4(int W, int FP8) { return W == 4 ? 4096 : 8192; }
constexpr int wgs_per_cu(int W, int FP8) { return W == 4 ? 2 : 1; }
constexpr int kRec = 768;            // copy-address records per chunk of kept blocks (12 KiB)
constexpr int kPlist = 8 * kRec;     // pruned blocks per correction chunk (u16, same 12 KiB)
#ifndef ATT_W
#define ATT_W 8
#endif

typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef __attribute__((address_space(3))) i32x2_t lds_i32x2_t;
typedef __attribute__((address_space(3))) char lds_char_t;
typedef __attribute__((address_space(3))) void lds_void_t;

// Swizzles: chunk c of row r is stored at slot (c ^ f(r)) of the row, so that
// the MFMA operand reads of one instruction spread over all LDS banks.
__device__ __forceinline__ int kslot16(int r, int c) { return r * 16 + (c ^ (r & 15)); }
__device__ __forceinline__ int vslot16(int r, int c) { return r * 16 + (c ^ (4 * (r & 3))); }
__device__ __forceinline__ int kslot8(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }
__device__ __forceinline__ int vslot8(int r, int c) { return r * 8 + (c ^ (2 * ((r >> 1) & 3))); }

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until a step's copies have landed while `ahead` later steps (D copies
// each, ahead <= 6) stay in flight.
template <int D>
__device__ __forceinline__ void wait_ahead(int ahead) {
  static_assert(6 * D < 64, "ring depth");
  if (ahead <= 0) wait_vmcnt<0>();
  else if (ahead == 1) wait_vmcnt<D>();
  else if (ahead == 2) wait_vmcnt<2 * D>();
  else if (ahead == 3) wait_vmcnt<3 * D>();
  else if (ahead == 4) wait_vmcnt<4 * D>();
  else if (ahead == 5) wait_vmcnt<5 * D>();
  else wait_vmcnt<6 * D>();
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // m0 is reserved; nothing else here uses it
// 16-byte copy global -> LDS (global_load_lds_dwordx4): lane i writes LDS
// bytes [base + 16 i, base + 16 i + 16), base taken from M0. Issued as inline
// assembly so that the compiler does not order every later LDS read behind
// it; completion is tracked explicitly with wait_vmcnt before the barrier
// that publishes a stage.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Copy plan of one 64-row step (K and V): copy instruction j of wave w moves
// rows RPG*(w + W*j) .. +RPG-1, lane i taking 16-byte slot i % CPR of row
// RPG*(w + W*j) + i / CPR.
template <int W, int FP8, int RING>
struct CopyPlan {
  static constexpr int CPR = FP8 ? 8 : 16;          // 16-byte chunks per row
  static constexpr int RPG = 64 / CPR;              // rows per copy instruction
  static constexpr int PER = kStep / RPG / W;       // copies per wave and tensor
  static constexpr int D = 2 * PER;                 // copies per thread and step
  static constexpr int STAGE = 2 * kStep * CPR;     // 16-byte slots per stage
  static constexpr int NST = RING / STAGE;          // ring depth
  __device__ static int row(int j, int tid) { return RPG * ((tid >> 6) + W * j) + (tid & 63) / CPR; }
};

// Start the copies of one step: row row(j) of K / V lies at byte offset
// off[j] from Kb / Vb.
template <int W, int FP8, int RING>
__device__ __forceinline__ void issue_copies(uint32_t st, const uint8_t* Kb, const uint8_t* Vb,
                                             const int64_t (&off)[CopyPlan<W, FP8, RING>::PER], int tid) {
  using P = CopyPlan<W, FP8, RING>;
  const int w = tid >> 6, lane = tid & 63;
  const uint32_t wu = __builtin_amdgcn_readfirstlane(w);   // wave index, uniform
  const int pc = lane % P::CPR;
#pragma unroll
  for (int j = 0; j < P::PER; ++j) {
    const int g = w + W * j;
    const int r = P::RPG * g + lane / P::CPR;
    const int kc = FP8 ? (pc ^ ((r >> 1) & 7)) : (pc ^ (r & 15));
    const int vc = FP8 ? (pc ^ (2 * ((r >> 1) & 3))) : (pc ^ (4 * (r & 3)));
    const uint32_t gl = st + (wu + W * j) * 64 * 16;
    dma16(Kb + off[j] + 16 * kc, gl);
    dma16(Vb + off[j] + 16 * vc, gl + 64 * P::CPR * 16);
  }
}

// Copy addresses of a step come in two parts: fetch(s, r) reads the table
// entry of row r of step s from LDS, addr(entry, s, r) turns it into the byte
// offset. The entries of the next step are fetched before a step is computed
// and converted after the next barrier, so their LDS latency is never waited
// on.
template <int W, int FP8, int RING, class Fetch, class Addr>
struct Addresser {
  using P = CopyPlan<W, FP8, RING>;
  using Raw = decltype(std::declval<Fetch>()(0, 0));
  Fetch fetch;
  Addr addr;
  int tid;
  Raw raw[P::PER];
  int64_t off[P::PER];
  __device__ __forceinline__ void get(int s) {
#pragma unroll
    for (int j = 0; j < P::PER; ++j) raw[j] = fetch(s, P::row(j, tid));
  }
  __device__ __forceinline__ void convert(int s) {
#pragma unroll
    for (int j = 0; j < P::PER; ++j) off[j] = addr(raw[j], s, P::row(j, tid));
  }
};

// Steps whose copies run ahead of the step being computed (at most the
// ring depth less one). Measured on 8-wave items: three steps ahead for fp8
// (of an 8-stage ring) and two for the correction (of a 4-stage ring) are
// 1-2% faster than the whole ring, and the bf16 kept steps take one (set at
// their call); the latency of a step's copies is covered either way. 4-wave
// items keep the whole (half) ring.
constexpr int copy_lead(int W, int FP8, int nst) {
  return W != 8 ? nst - 1 : FP8 ? 3 : 2;
}

// Ring over steps 0 .. n-1 without cross-step overlap of the compute;
// body(stage, s) consumes step s. Ends with a barrier (the ring may be
// refilled).
template <int W, int FP8, int RING, int LEAD_SET = 0, class Fetch, class Addr, class Body>
__device__ __forceinline__ void ring_loop(uint4* ring, int n, const uint8_t* Kb, const uint8_t* Vb,
                                          Fetch fetch, Addr addr, Body body, int tid) {
  using P = CopyPlan<W, FP8, RING>;
  constexpr int LEAD = LEAD_SET > 0 ? LEAD_SET : copy_lead(W, FP8, P::NST);
  static_assert(LEAD >= 1 && LEAD <= P::NST - 1 && LEAD <= 6, "copy lead");
  Addresser<W, FP8, RING, Fetch, Addr> ad{fetch, addr, tid};
  const uint32_t ring_lds = (uint32_t)(uintptr_t)(lds_void_t*)ring;   // LDS byte address
  int ni = 0;
#pragma unroll 1
  for (; ni < LEAD && ni < n; ++ni) {
    ad.get(ni);
    ad.convert(ni);
    issue_copies<W, FP8, RING>(ring_lds + ni * P::STAGE * 16, Kb, Vb, ad.off, tid);
  }
  if (ni < n) ad.get(ni);
#pragma unroll 1
  for (int s = 0; s < n; ++s) {
    wait_ahead<P::D>(ni - 1 - s);
    lds_barrier();   // step s visible to all; every wave is done with step s-1
    if (ni < n) {
      ad.convert(ni);
      issue_copies<W, FP8, RING>(ring_lds + (ni++ % P::NST) * P::STAGE * 16, Kb, Vb, ad.off, tid);
      if (ni < n) ad.get(ni);   // lands while the step is computed
    }
    body(ring + (s % P::NST) * P::STAGE, s);
  }
  lds_barrier();
}

// Larger of a lane's value and that of lane l^32.
__device__ __forceinline__ float xhalf_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  // v_max_f32 directly: the operands are scores (no signalling NaNs), and
  // fmaxf would first canonicalize each of them
  float m;
  asm("v_max_f32 %0, %1, %2" : "=v"(m) : "v"(r[0]), "v"(r[1]));
  return m;
}

// Running state of the RT 32-row tiles of one wave.
template <int RT>
struct RowState {
  f32x16_t o[RT][4];   // O^T accumulators: o[rt][dt][4i+j] = O[row][32dt + 8i + 4*half + j]
  f32x4_t ls[RT];      // fp8: row sums of the last step's P~ from the matrix cores
                       // (element 0, against m + k), folded into l at the next step
  float m[RT];         // reference of the accumulators o and l (log2 units)
  float l[RT];         // bf16: row-sum part of this lane's keys; fp8: the row sums
  int k[RT];           // fp8: P~ is taken against m + k and lifted by 2^k in the PV MFMAs
  float mc[RT];        // fp8: m + k
  float p2k[RT];       // fp8: 2^k
};

// Raw scores S^T of one 64-key step for the RT row tiles: v[rt][u][4i+j] is
// key 32u + 8i + 4*half + j of the lane's query row.
template <int RT>
struct Scores {
  f32x16_t v[RT][2];
};

// Lazy rescale (log2 units): the reference of a row's online softmax only
// moves when a new logit exceeds it by more than tau, so the probabilities
// are 2^(off + x - m) <= 2^(off + tau). bf16 (tau = 8) moves the reference m
// to the new maximum and rescales the accumulators; its probabilities stay
// far from any limit at 2^(8 + 8). fp8 keeps P~ = e4m3(2^8 exp(x - m_c))
// within the e4m3 range, 2^(8 + 0.8) = 445.7 < 448, against a reference
// m_c = m + k that moves in whole steps above the accumulators' reference m:
// the PV MFMAs lift each query's P~ by 2^k through their per-lane E8M0 B
// scales (127 + k: the 32 keys a lane holds belong to its own query), and the
// step's row sums, taken against m + k, join l times 2^k, so a move only
// changes k and the accumulators keep m. A move sets k = ceil(x_max - m) (the
// new maximum then lies in (2^7, 2^8]); only a row without a visible key so
// far, or a lift past 2^64, rebases m to the new maximum and rescales the
// accumulators.
constexpr float kTauFp8 = 0.8f;
constexpr float kTauBf16 = 8.0f;
// Largest lift: with P~ <= 2^8.8, value codes <= 448 and at most 2^17 keys a
// row's accumulators stay below 2^(35 + k), far inside fp32 for k <= 64.
constexpr int kMaxLift = 64;
// Reference of a row that has not seen a visible key yet: finite, so that the
// logit bias stays finite, and far below any logit, so that the first visible
// key moves it (and the rescale by 2^(m_old - m_new) = 0 clears nothing).
constexpr float kNoRef = -1e30f;

// Online-softmax rescale of row tile rt for the raw scores s (-inf where
// masked); the logits are x = cs * s + shift (log2 units, cs > 0). The
// reference m moves to the row's new maximum when that exceeds it by more
// than tau (any visible key moves it from kNoRef; a fully masked row, -inf,
// never does); the accumulators are rescaled only when some row of the wave
// moved. Returns the bias b with x - m + off = cs * s + b.
template <int NU, int RT>
__device__ __forceinline__ float softmax_rescale(const f32x16_t (&s)[NU], RowState<RT>& rs, int rt,
                                                 float cs, float shift, float off, float tau) {
  float mr = -INFINITY;
#pragma unroll
  for (int u = 0; u < NU; ++u)
#pragma unroll
    for (int e = 0; e < 16; ++e) mr = fmaxf(mr, s[u][e]);
  mr = xhalf_max(mr);
  const float mx = fmaf(mr, cs, shift);
  const bool up = mx > rs.m[rt] + tau;
  const float m_new = up ? mx : rs.m[rt];
  if (__any(up)) {
    const float a = fast_exp2(rs.m[rt] - m_new);
    rs.l[rt] *= a;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) rs.o[rt][dt][e] *= a;
  }
  rs.m[rt] = m_new;
  return shift + off - m_new;
}

// fp8 counterpart of softmax_rescale with the lifted reference described
// above: returns the bias b with x - m_c + 8 = cs * s + b.
template <int RT>
__device__ __forceinline__ float softmax_lift_fp8(const f32x16_t (&s)[2], RowState<RT>& rs, int rt,
                                                  float cs, float shift) {
  float mr = -INFINITY;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int e = 0; e < 16; ++e) mr = fmaxf(mr, s[u][e]);
  mr = xhalf_max(mr);
  const float mx = fmaf(mr, cs, shift);   // the row's largest logit; -inf while all are masked
  rs.l[rt] = fmaf(rs.ls[rt][0], rs.p2k[rt], rs.l[rt]);   // the previous step's row sums
  const bool up = mx > rs.mc[rt] + kTauFp8;
  if (__any(up)) {
    // whole steps above m that bring m_c to the new maximum or past it; a
    // row that saw no key yet (m = kNoRef) or a lift past kMaxLift rebases
    const float kf = ceilf(mx - rs.m[rt]);
    const bool rebase = up && !(kf <= (float)kMaxLift);
    if (__any(rebase)) {
      const float m_new = rebase ? mx : rs.m[rt];
      const float a = fast_exp2(rs.m[rt] - m_new);
      rs.l[rt] *= a;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) rs.o[rt][dt][e] *= a;
      rs.m[rt] = m_new;
    }
    rs.k[rt] = rebase ? 0 : up ? (int)fminf(kf, (float)kMaxLift) : rs.k[rt];
    rs.mc[rt] = rs.m[rt] + (float)rs.k[rt];
    rs.p2k[rt] = ldexpf(1.f, rs.k[rt]);
  }
  return shift + 8.f - rs.mc[rt];
}

// Pairwise sum of 16 values.
__device__ __forceinline__ float sum16(const float (&x)[16]) {
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = x[2 * i] + x[2 * i + 1];
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = a[2 * i] + a[2 * i + 1];
  return (a[0] + a[1]) + (a[2] + a[3]);
}

// ---------------------------------------------------------------------------
// bf16 steps of 64 keys for the RT row tiles of the wave; every LDS operand
// read feeds RT MFMAs.
// ---------------------------------------------------------------------------
template <int RT>
__device__ __forceinline__ void qk_bf16(const uint4* st, const bf16x8_t (&qb)[RT][8], Scores<RT>& S,
                                        int lane) {
  const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    bf16x8_t a[8];
#pragma unroll
    for (int ds = 0; ds < 8; ++ds)
      a[ds] = __builtin_bit_cast(bf16x8_t, st[kslot16(32 * u + l32, 2 * ds + half)]);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      S.v[rt][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], qb[rt][0], f32x16_t{}, 0, 0, 0);
#pragma unroll
      for (int ds = 1; ds < 8; ++ds)
        S.v[rt][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ds], qb[rt][ds], S.v[rt][u], 0, 0, 0);
    }
  }
}

// Softmax + PV of a bf16 step from its scores. KIND 0: kept keys key0 ..
// key0+63 (diag: causal mask against pos). KIND 1: correction, column k is
// used iff k < nv (logit shift +7, PV weights x pv_scale). NPRE of the four
// 16-key groups of V^T are read before the softmax, the rest just before
// their MFMAs.
template <int KIND, int RT, int NPRE>
__device__ __forceinline__ void fin_bf16(const uint4* st, Scores<RT>& S, RowState<RT>& rs, float cs,
                                         float off, float pv_scale, int key0, const int (&pos)[RT],
                                         bool diag, int nv, int lane) {
  const int half = lane >> 5;
  const float lg_pv = KIND == 1 ? fast_log2(pv_scale) : 0.f;
  const float inv_pv = KIND == 1 ? 1.f / pv_scale : 1.f;
  // V^T fragment of key group kg (16 keys) and output tile dt: slot i' of
  // lane half H is key 16kg + 8(i'/4) + 4H + i'%4.
  const int g16 = lane >> 4, i16 = lane & 15;
  const int sidx = i16 >> 2, r4 = i16 & 3;
  const uint4* vt = st + kStep * 16;
  auto vread = [&](int kg, int dt) -> bf16x8_t {
    i16x4_t rd[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int key = 16 * kg + 8 * tt + 4 * (g16 >> 1) + sidx;
      const int d = 32 * dt + 16 * (g16 & 1) + 4 * r4;
      const int byte = vslot16(key, d >> 3) * 16 + (d & 7) * 2;
      rd[tt] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)((lds_char_t*)vt + byte));
    }
    const i32x2_t r0 = __builtin_bit_cast(i32x2_t, rd[0]);
    const i32x2_t r1 = __builtin_bit_cast(i32x2_t, rd[1]);
    return __builtin_bit_cast(bf16x8_t, (i32x4_t){r0[0], r0[1], r1[0], r1[1]});
  };
  constexpr int NV = RT > 1 ? 4 : NPRE;   // several row tiles share every fragment
  bf16x8_t va[NV > 0 ? NV : 1][4];
#pragma unroll
  for (int kg = 0; kg < NV; ++kg)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) va[kg][dt] = vread(kg, dt);

  // key of S[rt][u][4i+j] is 32u + 8i + 4*half + j. Per tile: softmax, then
  // its PV MFMAs, which run while the next tile's softmax is computed.
  // only the diagonal step (kept keys) or the last step of the list
  // (correction) has columns to drop
  const bool masked = KIND == 1 ? nv < kStep : diag;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    if (masked) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = 32 * u + 8 * i + 4 * half + j;
            const bool drop = KIND == 1 ? key >= nv : key0 + key > pos[rt];
            S.v[rt][u][4 * i + j] = drop ? -INFINITY : S.v[rt][u][4 * i + j];
          }
    }
    // KIND 1: the PV weight pv_scale (> 0) enters the exponent as log2
    // pv_scale, and the row sum divides it out once.
    const float bias = softmax_rescale<2>(S.v[rt], rs, rt, cs, KIND == 1 ? 7.0f : 0.0f, off,
                                          kTauBf16) +
                       (KIND == 1 ? lg_pv : 0.f);
    float pv[2][16];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 16; ++e) pv[u][e] = fast_exp2(fmaf(S.v[rt][u][e], cs, bias));
    const float psum = sum16(pv[0]) + sum16(pv[1]);
    rs.l[rt] += KIND == 1 ? psum * inv_pv : psum;
    // O^T += V^T P^T, 16 keys per MFMA; B operand of key group kg = 2u + a:
    // slot i' of lane half H is S[u][8a + i']
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      uint32_t pw[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pw[q] = pack_bf16x2(pv[kg >> 1][8 * (kg & 1) + 2 * q], pv[kg >> 1][8 * (kg & 1) + 2 * q + 1]);
      const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const bf16x8_t v = kg < NV ? va[kg < NV ? kg : 0][dt] : vread(kg, dt);
        rs.o[rt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v, pb, rs.o[rt][dt], 0, 0, 0);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp8 pieces: the scores of one 64-key step, then softmax + PV.
// ---------------------------------------------------------------------------
// LDS byte offsets, within a stage, of this lane's fp8 operand reads: the K
// tile (ds, chunk pair; key subtile u = 1 lies 32 rows = 4 KiB further, as
// rows 32 apart share the swizzle) and the V^T fragments (dt; key group t
// lies 16 rows = 2 KiB further, the V tile 8 KiB after the K tile).
// Computed once per item and made opaque, so that a step adds its stage
// base to each with one instruction; the mask keeps the known range, so the
// constant distances fold into the LDS instructions' offsets.
struct Fp8Lane {
  int k[2][2];
  int v[4];
};

__device__ __forceinline__ Fp8Lane fp8_lane_offsets(int lane) {
  Fp8Lane o;
  const int half = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int ds = 0; ds < 2; ++ds)
#pragma unroll
    for (int t = 0; t < 2; ++t) o.k[ds][t] = 16 * kslot8(l32, 4 * ds + 2 * half + t);
  // V^T fragment dt, key group t: byte b of lane half H is key
  // 16t + 8((b%8)/4) + 4H + b%4 (b = 8 r2 + byte of the read)
  const int g16 = lane >> 4, i16 = lane & 15;
  const int sidx = i16 >> 1, r2 = i16 & 1;
  const int key = 8 * (sidx >> 2) + 4 * (g16 >> 1) + (sidx & 3);
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o.v[dt] = 16 * vslot8(key, 2 * dt + (g16 & 1)) + 8 * r2;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    asm volatile("" : "+v"(o.k[i >> 1][i & 1]), "+v"(o.v[i]));
    o.k[i >> 1][i & 1] &= 0x3fff;
    o.v[i] &= 0x3fff;
  }
  return o;
}

template <int RT>
__device__ __forceinline__ void qk_fp8(const uint4* st, const i32x8_t (&qf)[RT][2], Scores<RT>& S,
                                       const Fp8Lane& ol) {
  const char* sb = (const char*)st;
  i32x8_t a[2][2];
#pragma unroll
  for (int ds = 0; ds < 2; ++ds) {
    const char* k0 = sb + ol.k[ds][0];
    const char* k1 = sb + ol.k[ds][1];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const uint4 c0 = *(const uint4*)(k0 + 4096 * u);
      const uint4 c1 = *(const uint4*)(k1 + 4096 * u);
      a[u][ds] = (i32x8_t){(int)c0.x, (int)c0.y, (int)c0.z, (int)c0.w,
                           (int)c1.x, (int)c1.y, (int)c1.z, (int)c1.w};
    }
  }
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      S.v[rt][u] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[u][0], qf[rt][0], f32x16_t{}, 0,
                                                                    0, 0, 0, 0, 0);
      S.v[rt][u] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[u][1], qf[rt][1], S.v[rt][u], 0,
                                                                    0, 0, 0, 0, 0);
    }
}

// V^T fragments of a 64-key fp8 step (the layout of Fp8Lane::v).
__device__ __forceinline__ void vread_fp8(const uint4* st, i32x8_t (&va)[4], const Fp8Lane& ol) {
  const char* vb = (const char*)st + kStep * 8 * 16;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    i32x2_t rd[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
      rd[t] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2_t*)(lds_char_t*)(vb + ol.v[dt] + 2048 * t));
    va[dt] = (i32x8_t){rd[0][0], rd[0][1], rd[1][0], rd[1][1], rd[2][0], rd[2][1], rd[3][0], rd[3][1]};
  }
}

// Four e4m3 codes (round to nearest even) of four non-negative floats <= 448.
// The first conversion writes the low half-word and the second the high one,
// so the register's previous contents never matter (no zeroing move).
__device__ __forceinline__ int pack_e4m3x4(float a, float b, float c, float d) {
  int w;
  asm volatile("" : "=v"(w));
  w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, w, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

// Finish an fp8 step of 64 kept keys key0 .. key0+63 from its scores: per
// row tile the softmax (diag: causal mask against pos) and
// O^T += V^T P~^T with P~ = e4m3(2^8 exp(x - m)); the softmax of one tile
// runs on the vector ALUs while the matrix cores work on the other tile.
// The row sums of P~ come from the matrix cores as well, through one
// v_mfma_f32_16x16x128_f8f6f4 per step: read as its B operand (128 x 16),
// the P~ registers hold in column n the 64 keys of query n (k-groups 0 and 2)
// and of query n+16 (k-groups 1 and 3), so a 0/1 selector A operand whose
// row m picks the k-groups of parity (m/4)%2 leaves in every element of lane
// l the row sum of the lane's own query l%32.
// KIND 0: kept keys key0 .. key0+63, masked against pos when `diag`. KIND 1:
// correction (e4m3 code means as keys and values), column k used iff k < nv
// (masked when `diag`), logits shifted by log2 |B_J| = 7.
template <int KIND, int RT>
__device__ __forceinline__ void fin_fp8(const uint4* st, Scores<RT>& S, RowState<RT>& rs, float cs,
                                        int key0, const int (&pos)[RT], bool diag, int lane,
                                        const i32x8_t& sel, const Fp8Lane& ol, int nv = kStep) {
  const int half = lane >> 5;
  auto& s = S.v;
  i32x8_t va[4];
  vread_fp8(st, va, ol);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    if (diag) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = 32 * u + 8 * i + 4 * half + j;
            const bool drop = KIND == 1 ? key >= nv : key0 + key > pos[rt];
            s[rt][u][4 * i + j] = drop ? -INFINITY : s[rt][u][4 * i + j];
          }
    }
    const float bias = softmax_lift_fp8<RT>(s[rt], rs, rt, cs, KIND == 1 ? 7.0f : 0.0f);
    int pk[8];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pk[4 * u + q] = pack_e4m3x4(fast_exp2(fmaf(s[rt][u][4 * q], cs, bias)),
                                    fast_exp2(fmaf(s[rt][u][4 * q + 1], cs, bias)),
                                    fast_exp2(fmaf(s[rt][u][4 * q + 2], cs, bias)),
                                    fast_exp2(fmaf(s[rt][u][4 * q + 3], cs, bias)));
    const i32x8_t pb = {pk[0], pk[1], pk[2], pk[3], pk[4], pk[5], pk[6], pk[7]};
    // P~ lifted by 2^k (E8M0 B scale of the lane's query, 127 + k; A unscaled,
    // 127). The row-sum MFMA stays unscaled: in its 16x16 shape a B column
    // holds two queries, and its B scale is one per column
    const int sb = 127 + rs.k[rt];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      rs.o[rt][dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(va[dt], pb, rs.o[rt][dt], 0, 0, 0,
                                                                     127, 0, sb);
    rs.ls[rt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(sel, pb, f32x4_t{}, 0, 0, 0, 0, 0,
                                                                 0);
  }
}

// Steps 0 .. n-1 of a ring: the scores of a step (qk) then the rest of it
// (fin). The two waves of a SIMD overlap each other's matrix and vector work.
template <int W, int FP8, int RT, int RING, int LEAD_SET = 0, class Fetch, class Addr, class QK,
          class Fin>
__device__ __forceinline__ void run_steps(uint4* ring, int n, const uint8_t* Kb, const uint8_t* Vb,
                                          Fetch fetch, Addr addr, QK qk, Fin fin, int tid) {
  ring_loop<W, FP8, RING, LEAD_SET>(ring, n, Kb, Vb, fetch, addr, [&](const uint4* st, int s) {
    Scores<RT> S;
    qk(st, S);
    fin(st, S, s);
  }, tid);
}

template <int FP8, int W, int RT>
__global__ __launch_bounds__(64 * W, wgs_per_cu(W, FP8)) void attend_kernel(Problem p0, Pooled pooled,
                                                           const uint8_t* __restrict__ mask,
                                                           KeptLists kl, Plan plan,
                                                           uint16_t* __restrict__ out,
                                                           float* __restrict__ lse) {
  constexpr int RING = ring_u4(W, FP8);
  __shared__ uint4 ring[RING];
  __shared__ uint4 aux[kRec];               // kept: copy-address records; correction: pruned list
  __shared__ int32_t wtot[W];
  __shared__ int4 s_item;

  constexpr int M = 32 * RT * W;            // packed rows per work item
  // V^T key groups read ahead of the softmax (all four only with a wave per SIMD)
  constexpr int NPRE = W > 4 || wgs_per_cu(W, FP8) > 1 ? 2 : 4;
  const int wpu = p0.g * p0.qtile / M;      // row slices per unit
  const int nbh = p0.batch * p0.hkv;
  const int tid0 = threadIdx.x;

  // Persistent workgroups: items of the plan's table (unit, KV split, row
  // slice, and the unit's split count and partial slot; decreasing query
  // block, i.e. heaviest first) are taken in order from a counter; the loop
  // ends for every wave once the counter passes the last item.
#pragma unroll 1
  for (;;) {
    if (tid0 == 0) {
      const int it = atomicAdd(plan.counts, 1);
      int4 v = make_int4(-1, 0, 0, 0);
      if (it < plan.counts[1]) v = plan.items[it];
      s_item = v;
    }
    __syncthreads();
    const int4 cur = s_item;
    __syncthreads();   // every wave has read s_item before it is written again
    if (cur.x < 0) break;
    // Opaque copies of the thread index and of the argument block: what is
    // derived from them is recomputed per item instead of being held in
    // registers across the whole loop. p0 is the first kernel argument, so it
    // sits at offset 0 of the kernel argument segment; its fields are read
    // back from there with scalar loads.
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    typedef const __attribute__((address_space(4))) Problem KProblem;
    KProblem* pk = (KProblem*)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(pk));
    KProblem& p = *pk;

    const int u = cur.x;                     // attention-order index of the unit
    const int sp = cur.y / wpu;              // its part (KV split) ...
    const int msub = cur.y - sp * wpu;       // ... and row slice
    const int nsp = cur.z;                   // parts of the unit
    const int I = p.nbmax - 1 - u / nbh;
    const int bh = u % nbh;
    const int b = bh / p.hkv, h = bh % p.hkv;
    const int Lq = ld_uniform(p.cu, b + 1) - ld_uniform(p.cu, b);
    if (I * p.qtile >= Lq) continue;
    // KV tokens of the sequence (a prefix included) and the key blocks Ja,
    // Jb of the unit's first and last row; positions below are absolute, and
    // query position x is packed row qbase + x
    const int64_t tok0 = ld_uniform(p.cuk, b);
    const int L = ld_uniform(p.cuk, b + 1) - (int)tok0;
    const int Ja = (L - Lq + I * p.qtile) / kBlock;
    const int64_t qbase = (int64_t)ld_uniform(p.cu, b) - (L - Lq);

    const int lane = tid & 63, w = tid >> 6;
    const int half = lane >> 5, l32 = lane & 31;
    const int G = p.g;
    const int64_t row = ((int64_t)b * p.hkv + h) * p.nbmax + I;

    // this lane's query rows (packed rows of Eq. packgqa), one per row tile;
    // G divides 32, so a lane column keeps one query head
    const int pr0 = msub * M + w * 32 * RT + l32;
    const int hq = h * G + pr0 % G;
    int pos[RT];
    bool qvalid[RT];
    int64_t qoff[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      pos[rt] = (L - Lq) + I * p.qtile + (pr0 + 32 * rt) / G;
      qvalid[rt] = pos[rt] < L;
      qoff[rt] = ((qbase + pos[rt]) * p.hq + hq) * kHeadDim;   // element index
    }

    RowState<RT> rs;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) rs.o[rt][dt] = f32x16_t{};
      rs.ls[rt] = f32x4_t{};
      rs.m[rt] = kNoRef;
      rs.l[rt] = 0.f;
      rs.k[rt] = 0;
      rs.mc[rt] = kNoRef;
      rs.p2k[rt] = 1.f;
    }
    float qsc = FP8 ? p.q_scale[hq] : 1.f;
    float vsc = FP8 ? ld_uniform(p.v_scale, h) : 1.f;
    float ksc = FP8 ? ld_uniform(p.k_scale, h) : 1.f;
    const float off = FP8 ? 8.f : 0.f;        // log2 of the probability offset
    asm volatile("" : "+v"(qsc), "+v"(vsc), "+v"(ksc));  // loads complete before the rings

    // fp8: the query codes (B operand of the score products) and the selector
    // A operand of the row-sum MFMA: lane l holds row l%16, k-group l/16 of A,
    // all e4m3 1.0 (0x38) where the row's parity (l%16)/4 matches the
    // k-group's, else 0; opaque so that it stays in registers instead of being
    // rebuilt every step. Both serve the kept keys and the correction.
    i32x8_t qf[FP8 ? RT : 1][2];
    i32x8_t sel;
    if constexpr (FP8) {
      const int selw = (((lane & 15) >> 2) & 1) == ((lane >> 4) & 1) ? 0x38383838 : 0;
#pragma unroll
      for (int k = 0; k < 8; ++k) sel[k] = selw;
      asm volatile("" : "+v"(sel));
    }
    [[maybe_unused]] Fp8Lane ol;
    if constexpr (FP8) ol = fp8_lane_offsets(lane);

    // ---- kept blocks: step s of a chunk -> its block list entry s/2, half s%2
    {
      const uint8_t* K = (const uint8_t*)p.k;
      const uint8_t* V = (const uint8_t*)p.v;
      constexpr int esz = FP8 ? 1 : 2;
      const int cnt = ld_uniform(kl.cnt, row);
      const int32_t* kidx = kl.idx + row * p.nbk;
      // Kept blocks J >= Ja hold keys after some row of the unit and need the
      // causal mask: at most two (Ja and Jb), the first of the descending walk.
      const int e0 = cnt > 0 ? ld_uniform(kidx, cnt - 1) : -1, e1 = cnt > 1 ? ld_uniform(kidx, cnt - 2) : -1;
      const int nmask = (e0 >= Ja) + (e1 >= Ja);
      // Eq. split: part sp walks list positions [lo, hi) of the descending
      // walk, ceil(cnt / nsp) each
      const int per = (cnt + nsp - 1) / nsp;
      const int lo = min(cnt, sp * per), hi = min(cnt, lo + per);
      const int64_t rowbytes = (int64_t)p.hkv * kHeadDim * esz;     // one token slot of the pool
      const int64_t hbytes = (int64_t)h * kHeadDim * esz;
      const int page = p.pm.page, shift = p.pm.shift;
      // Copy-address records: rows of a 64-key half come in groups of G that
      // lie in one page (G = 64 contiguous, min(p, 64) for a power-of-two
      // page, 1 otherwise); one record per (kept block, half, group).
      const int gshift = page == 0 ? 6 : shift >= 0 ? min(shift, 6) : 0;
      const int rph = kStep >> gshift;       // records per half
      const int chunk = kRec / (2 * rph);    // kept blocks per table chunk
      const int32_t* ptab = p.pm.table + (int64_t)b * p.pm.stride;
      auto slot_of = [&](int t) -> uint32_t {
        if (page == 0) return (uint32_t)(tok0 + t);
        const int pi = shift >= 0 ? t >> shift : t / page;
        return (uint32_t)ptab[pi] * (uint32_t)page + (uint32_t)(t - pi * page);
      };

      bf16x8_t qb[FP8 ? 1 : RT][8];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if constexpr (FP8) {
          const uint8_t* qrow = (const uint8_t*)p.q + qoff[rt];
#pragma unroll
          for (int ds = 0; ds < 2; ++ds) {
            uint4 c0 = make_uint4(0, 0, 0, 0), c1 = make_uint4(0, 0, 0, 0);
            if (qvalid[rt]) {
              c0 = *(const uint4*)(qrow + 64 * ds + 32 * half);
              c1 = *(const uint4*)(qrow + 64 * ds + 32 * half + 16);
            }
            qf[rt][ds] = (i32x8_t){(int)c0.x, (int)c0.y, (int)c0.z, (int)c0.w,
                                   (int)c1.x, (int)c1.y, (int)c1.z, (int)c1.w};
            asm volatile("" : "+v"(qf[rt][ds]));
          }
        } else {
          const uint16_t* qrow = (const uint16_t*)p.q + qoff[rt];
#pragma unroll
          for (int ds = 0; ds < 8; ++ds) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (qvalid[rt]) v = *(const uint4*)(qrow + 16 * ds + 8 * half);
            qb[rt][ds] = __builtin_bit_cast(bf16x8_t, v);
            asm volatile("" : "+v"(qb[rt][ds]));
          }
        }
      }
      const float cs = FP8 ? p.scale_log2 * qsc * ksc : p.scale_log2;

#pragma unroll 1
      for (int c0 = lo; c0 < hi; c0 += chunk) {
        const int nbc = min(chunk, hi - c0);
        // Record (block i, half hf, group e) = {byte offset base at which row
        // 0 of the half would lie if the group's page continued down to it
        // (64-bit, may be negative), limit lim >= 0}: row r of the group then
        // lies at base + min(r * rowbytes, lim), with lim the offset of the
        // half's last valid row (at most 63 rows). Rows past the sequence thus
        // repeat its last token (finite data; those keys are masked); a group
        // that starts past it points at that token directly (base = the
        // token, lim = 0). The offset added to base is never negative.
        for (int k = tid; k < nbc * 2 * rph; k += 64 * W) {
          const int i = k / (2 * rph), hk = k - i * 2 * rph;
          const int key0 = kidx[cnt - 1 - (c0 + i)] * kBlock + kStep * (hk >= rph);
          const int last = L - 1 - key0;   // negative when the half starts past the sequence
          const int first = (hk % rph) << gshift;
          int64_t base;
          uint32_t lim;
          if (first <= last) {
            base = ((int64_t)slot_of(key0 + first) - first) * rowbytes + hbytes;
            lim = (uint32_t)(min(last, kStep - 1) * rowbytes);
          } else {
            base = (int64_t)slot_of(L - 1) * rowbytes + hbytes;
            lim = 0u;
          }
          aux[k] = make_uint4((uint32_t)base, (uint32_t)((uint64_t)base >> 32), lim, 0u);
        }
        __syncthreads();
        auto fetch = [&](int s, int r) -> uint4 { return aux[(s * rph) + (r >> gshift)]; };
        const int rowb = (int)rowbytes;   // <= 2^18 (Hkv <= 1024), so 63 * rowb fits int32
        auto addr = [&](uint4 rec, int s, int r) -> int64_t {
          (void)s;
          const int64_t base = (int64_t)(((uint64_t)rec.y << 32) | rec.x);
          // r * rowb is fixed per lane; both operands of min are >= 0
          return base + (uint32_t)min(r * rowb, (int)rec.z);
        };
        const int nst = 2 * nbc;
        if constexpr (FP8) {
          run_steps<W, 1, RT, RING>(
              ring, nst, K, V, fetch, addr,
              [&](const uint4* st, Scores<RT>& S) { qk_fp8<RT>(st, qf, S, ol); },
              [&](const uint4* st, Scores<RT>& S, int s) {
                const int wp = c0 + (s >> 1);   // walk position of the step's block
                fin_fp8<0, RT>(st, S, rs, cs, (wp == 0 ? e0 : e1) * kBlock + kStep * (s & 1), pos,
                               wp < nmask, lane, sel, ol);
              },
              tid);
        } else {
          run_steps<W, 0, RT, RING, W == 8 ? 1 : 0>(   // bf16 kept steps: one step ahead
              ring, nst, K, V, fetch, addr,
              [&](const uint4* st, Scores<RT>& S) { qk_bf16<RT>(st, qb, S, lane); },
              [&](const uint4* st, Scores<RT>& S, int s) {
                const int wp = c0 + (s >> 1);   // walk position of the step's block
                fin_bf16<0, RT, NPRE>(st, S, rs, cs, off, 1.f,
                                      (wp == 0 ? e0 : e1) * kBlock + kStep * (s & 1), pos,
                                      wp < nmask, 0, lane);
              },
              tid);
        }
      }
    }

    // ---- mean correction over the pruned blocks J < Ja (fully visible to
    // every row of the unit), compacted into a list; split sp takes the
    // blocks J in [jlo, jhi)
    const int perj = (Ja + nsp - 1) / nsp;
    const int jlo = min(Ja, sp * perj), jhi = min(Ja, jlo + perj);
    if (p.corr && jhi > jlo) {
      const uint8_t* mrow = mask + row * p.nbk;
      uint16_t* plist = (uint16_t*)aux;
      // bf16: Q and the bf16 means, bf16 steps (the log2 |B_J| = 7 shift in the
      // logits). fp8: the query codes and the e4m3 code means of keys and
      // values, fp8 steps like the kept keys (scores scaled by c_q c_k, value
      // codes by c_v at the end, P~ in e4m3 with its row sums from the
      // selector MFMA).
      bf16x8_t qb[FP8 ? 1 : RT][8];
      if constexpr (!FP8) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int ds = 0; ds < 8; ++ds) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (qvalid[rt]) v = *(const uint4*)((const uint16_t*)p.q + qoff[rt] + 16 * ds + 8 * half);
            qb[rt][ds] = __builtin_bit_cast(bf16x8_t, v);
            asm volatile("" : "+v"(qb[rt][ds]));
          }
      }
      const float cs = FP8 ? p.scale_log2 * qsc * ksc : p.scale_log2;
      const int64_t pbase = ((int64_t)b * p.hkv + h) * p.nbk * kHeadDim;
      const uint8_t* Kh = FP8 ? pooled.khat8 + pbase : (const uint8_t*)(pooled.khat + pbase);
      const uint8_t* Vh = FP8 ? pooled.vbar8 + pbase : (const uint8_t*)(pooled.vbar + pbase);
#pragma unroll 1
      for (int j0 = jlo; j0 < jhi; j0 += kPlist) {
        const int j1 = min(jhi, j0 + kPlist);
        // compaction of the pruned J in [j0, j1), in ascending order
        int np = 0;
#pragma unroll 1
        for (int jb = j0; jb < j1; jb += 64 * W) {
          const int J = jb + tid;
          const bool f = J < j1 && !(mrow[J] & 1);
          const uint64_t bal = __ballot(f);
          const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
          if (lane == 0) wtot[w] = __popcll(bal);
          __syncthreads();
          int base = np, tot = 0;
#pragma unroll
          for (int v = 0; v < W; ++v) {
            base += v < w ? wtot[v] : 0;
            tot += wtot[v];
          }
          if (f) plist[base + before] = (uint16_t)J;
          np += tot;
          __syncthreads();
        }
        if (np == 0) continue;
        // past the list: repeat a valid entry
        auto fetch = [&](int s, int r) -> int { return plist[min(kStep * s + r, np - 1)]; };
        auto addr = [&](int J, int s, int r) -> int64_t {
          (void)s;
          (void)r;
          return (int64_t)J * kHeadDim * (FP8 ? 1 : 2);
        };
        if constexpr (FP8) {
          run_steps<W, 1, RT, RING>(
              ring, (np + kStep - 1) / kStep, Kh, Vh, fetch, addr,
              [&](const uint4* st, Scores<RT>& S) { qk_fp8<RT>(st, qf, S, ol); },
              [&](const uint4* st, Scores<RT>& S, int s) {
                const int nv = np - kStep * s;
                fin_fp8<1, RT>(st, S, rs, cs, 0, pos, nv < kStep, lane, sel, ol, nv);
              },
              tid);
        } else {
          run_steps<W, 0, RT, RING>(
              ring, (np + kStep - 1) / kStep, Kh, Vh, fetch, addr,
              [&](const uint4* st, Scores<RT>& S) { qk_bf16<RT>(st, qb, S, lane); },
              [&](const uint4* st, Scores<RT>& S, int s) {
                fin_bf16<1, RT, NPRE>(st, S, rs, cs, off, 1.f, 0, pos, false, np - kStep * s,
                                      lane);
              },
              tid);
        }
      }
    }

    // fp8: the row sums of P~ from the matrix cores join the denominator
    if constexpr (FP8) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)   // both lane halves hold the row's sums; keep one
        rs.l[rt] = half == 0 ? fmaf(rs.ls[rt][0], rs.p2k[rt], rs.l[rt]) : 0.f;
    }

    // epilogue: O = c_v O^T / l, LSE = (m + log2 l - off) ln 2; with KV
    // splits the unnormalised partials go to the workspace instead
    if (nsp > 1) {
      const int64_t slot = cur.w + sp;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const float l_tot = rs.l[rt] + __shfl_xor(rs.l[rt], 32, 64);
        if (!qvalid[rt]) continue;
        const int64_t prow = slot * (G * p.qtile) + pr0 + 32 * rt;
        float* po = plan.part_o + prow * kHeadDim;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int d = 32 * dt + 8 * i + 4 * half;
            *(float4*)(po + d) = make_float4(rs.o[rt][dt][4 * i + 0], rs.o[rt][dt][4 * i + 1],
                                             rs.o[rt][dt][4 * i + 2], rs.o[rt][dt][4 * i + 3]);
          }
        if (half == 0)   // a part that saw no visible key reports m = -inf
          *(float2*)(plan.part_ml + 2 * prow) = make_float2(l_tot > 0.f ? rs.m[rt] : -INFINITY, l_tot);
      }
      continue;
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const float l_tot = rs.l[rt] + __shfl_xor(rs.l[rt], 32, 64);
      if (!qvalid[rt]) continue;
      const float inv = vsc / l_tot;
      uint16_t* orow = out + qoff[rt];
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = 32 * dt + 8 * i + 4 * half;
          uint2 v;
          v.x = pack_bf16x2(rs.o[rt][dt][4 * i + 0] * inv, rs.o[rt][dt][4 * i + 1] * inv);
          v.y = pack_bf16x2(rs.o[rt][dt][4 * i + 2] * inv, rs.o[rt][dt][4 * i + 3] * inv);
          *(uint2*)(orow + d) = v;
        }
      if (lse && half == 0)
        lse[(qbase + pos[rt]) * p.hq + hq] = (rs.m[rt] + fast_log2(l_tot) - off) * kLn2;
    }
  }
}

template <int FP8, int W, int RT>
hipError_t launch_cfg(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                      const KeptLists& kl, const Plan& plan, void* out, float* lse,
                      hipStream_t s) {
  const int cus = device_compute_units();
  if (cus <= 0) return hipErrorInvalidDevice;
  const unsigned grid = (unsigned)std::min<int64_t>(plan.cap_items, (int64_t)cus * wgs_per_cu(W, FP8));
  attend_kernel<FP8, W, RT><<<grid, 64 * W, 0, s>>>(p, pooled, mask, kl, plan,
                                                          (uint16_t*)out, lse);
  return hipSuccess;
}

// 32 query rows per wave; 8 waves (two per SIMD) when the unit (query tile)
// has at least 256 packed rows, else 4 (a 128-row tile is one work item).
constexpr int waves_for(int rows) { return rows < 256 ? 4 : ATT_W; }

template <int FP8>
hipError_t launch_dt(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                     const KeptLists& kl, const Plan& plan, void* out, float* lse,
                     hipStream_t s) {
  if (p.g * p.qtile < 256)
    return launch_cfg<FP8, waves_for(128), 1>(p, pooled, mask, kl, plan, out, lse, s);
  return launch_cfg<FP8, ATT_W, 1>(p, pooled, mask, kl, plan, out, lse, s);
}

}  // namespace

int attend_items_per_unit(int g, int qtile) { return g * qtile / (32 * waves_for(g * qtile)); }

hipError_t launch_attend(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                         const KeptLists& kl, const Plan& plan, void* out, float* lse,
                         hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  const hipError_t e = p.fp8 ? launch_dt<1>(p, pooled, mask, kl, plan, out, lse, s)
                             : launch_dt<0>(p, pooled, mask, kl, plan, out, lse, s);
  return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace fp2

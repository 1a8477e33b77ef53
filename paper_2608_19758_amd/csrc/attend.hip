// Sparse attention over the kept key blocks with the mean correction
// (Sec. 3.2 Eq. correction, Sec. 3.3; Algorithm 1 steps 6-11).
//
// Work unit: (sequence b, KV head h, query block I) of the packed query rows
// of Eq. packgqa. A workgroup of W waves takes 32*W of the g*B packed rows
// (W = 8, or 4 when g = 1), so one K/V tile in LDS serves all g query heads
// of the group. Units are dealt heaviest-first and the workgroups of a unit
// go to the same XCD (consecutive dispatch slots of one XCD), so they share
// K/V through its L2.
//
// The key sequence of a unit is a list of 64-key steps: both halves of every
// kept block, walked from the last kept index down (Eq. csr), then both
// halves of every 128-block chunk of pooled means that holds a pruned block
// (the correction). Steps run through a ring of LDS stages (128 KiB: 4 bf16
// stages or 8 fp8 stages): the rows of step s+NST-1 are copied straight from
// the page-addressed pool (Eq. page) into LDS with global_load_lds_dwordx4
// while step s is computed, with one workgroup barrier per step. Page-table
// and kept-list reads are scalar loads, so nothing in the loop waits on the
// copies except the explicit count before each barrier.
//
// Per step:
//  - S^T = K Q^T on the matrix cores (A = key rows from LDS, B = the wave's
//    32 query rows held in registers). Lane l then owns query l%32 and 16
//    keys per 32-key subtile, so the row max/sum of the online softmax need
//    one exchange with lane l^32;
//  - O^T += V^T P^T: the probabilities go straight from the S^T accumulators
//    into the B operand, and V^T comes from LDS through the gfx950
//    transposing reads ds_read_b64_tr_b16 / _b8 (no transpose pass).
// bf16 uses v_mfma_f32_32x32x16_bf16. fp8 (OCP e4m3fn) uses
// v_mfma_f32_32x32x64_f8f6f4 on the raw codes; the per-head scales c_q c_k
// are applied to the fp32 scores, the probabilities are stored as
// e4m3(2^8 * exp(S - m)) (range [0, 256], Sec. 3.3 Eq. fp8) and c_v is
// applied in the epilogue; the 2^8 is removed from the LSE.
// Correction steps use the pooled means as keys khat_J and values vbar_J
// (bf16, real units, bf16 MFMA for both dtypes), logits shifted by
// log2|B_J| = 7 (Sec. 3.2 implementation paragraph).
#include "kernels.h"

namespace fp2 {

namespace {

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kStep = 64;           // keys per pipeline step
constexpr int kRingU4 = 8192;       // LDS ring: 128 KiB in 16-byte slots

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

// Wait until the copies of the current step have landed while `ahead` later
// steps (D copies each, at most MAXA of them) stay in flight.
template <int D, int MAXA>
__device__ __forceinline__ void wait_steps_ahead(int ahead) {
  static_assert(MAXA >= 1 && MAXA <= 6 && MAXA * D < 64, "ring depth");
  if (ahead <= 0) wait_vmcnt<0>();
  else if (ahead == 1 || MAXA == 1) wait_vmcnt<D>();
  else if (ahead == 2 || MAXA == 2) wait_vmcnt<2 * D>();
  else if (ahead == 3 || MAXA == 3) wait_vmcnt<3 * D>();
  else if (ahead == 4 || MAXA == 4) wait_vmcnt<4 * D>();
  else if (ahead == 5 || MAXA == 5) wait_vmcnt<5 * D>();
  else wait_vmcnt<6 * D>();
}

// Workgroup barrier for LDS traffic: this wave's LDS operations complete,
// then all waves meet. Outstanding global->LDS copies are not waited for.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // m0 is reserved; nothing else here uses it
// 16-byte copy global -> LDS (global_load_lds_dwordx4): lane i writes LDS
// bytes [base + 16 i, base + 16 i + 16), base taken from M0. Issued as inline
// assembly so that the compiler does not order every later LDS read behind
// it; completion is tracked explicitly with wait_vmcnt before the barrier
// that publishes a stage.
__device__ __forceinline__ void dma16(const void* g, uint4* lds) {
  const uint32_t base = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)lds);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(base)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Scalar (wave-uniform) 32-bit load of read-only data written before the
// kernel started; counted by lgkmcnt, so it never waits on the copies.
__device__ __forceinline__ int sload_i32(const int32_t* ptr) {
  int v;
  asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(ptr));
  return v;
}

// Step ring: steps 0 .. nsteps-1; issue(stage, s) starts the copies of step
// s (D per thread), compute(stage, s) consumes it. Stage of step s: s % NST.
template <int NST, int D, class Issue, class Compute>
__device__ __forceinline__ void run_ring(uint4* ring, int stage_u4, int nsteps, Issue issue,
                                         Compute compute) {
#pragma unroll 1
  for (int s = 0; s < NST - 1 && s < nsteps; ++s) issue(ring + s * stage_u4, s);
#pragma unroll 1
  for (int s = 0; s < nsteps; ++s) {
    wait_steps_ahead<D, NST - 2>(min(NST - 2, nsteps - 1 - s));
    lds_barrier();   // step s visible to all; every wave is done with step s-1
    if (s + NST - 1 < nsteps) issue(ring + ((s + NST - 1) % NST) * stage_u4, s + NST - 1);
    compute(ring + (s % NST) * stage_u4, s);
  }
  lds_barrier();     // the ring may be refilled afterwards
}

// Copy 64 rows (row r: byte offset row_off(r0, r) from Kb / Vb, r0 = first
// row of the copy instruction, wave-uniform) into a stage: K rows at slots
// [0, 64*CPR), V rows at [64*CPR, 128*CPR), CPR 16-byte chunks per row.
template <int W, int FP8, class RowOff>
__device__ __forceinline__ void copy_rows(uint4* st, const uint8_t* Kb, const uint8_t* Vb,
                                          RowOff row_off) {
  constexpr int CPR = FP8 ? 8 : 16;
  constexpr int RPG = 64 / CPR;               // rows per 1 KiB copy
  constexpr int PER = (kStep / RPG) / W;      // copy instructions per wave and tensor
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int pc = lane % CPR;
  int64_t offs[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int r0 = RPG * (w + W * j);
    offs[j] = row_off(r0, r0 + lane / CPR);
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int g = w + W * j;
    const int r = RPG * g + lane / CPR;
    const int kc = FP8 ? (pc ^ ((r >> 1) & 7)) : (pc ^ (r & 15));
    const int vc = FP8 ? (pc ^ (2 * ((r >> 1) & 3))) : (pc ^ (4 * (r & 3)));
    dma16(Kb + offs[j] + 16 * kc, st + g * 64);
    dma16(Vb + offs[j] + 16 * vc, st + 64 * CPR + g * 64);
  }
}

template <int W, int FP8> struct Copies {
  static constexpr int CPR = FP8 ? 8 : 16;
  static constexpr int per_step = 2 * ((kStep / (64 / CPR)) / W);   // per thread
  static constexpr int stage_u4 = 2 * kStep * CPR;
  static constexpr int nst = kRingU4 / stage_u4;
};

// Online-softmax update of one 32-row tile over NU 32-key subtiles. On entry
// s holds raw scores (-inf where masked); the logits are x = cs * s + shift
// (log2 units). On return s holds 2^(x - m + off), their row sum has been
// added to l_i, and o / l_i have been rescaled to the new running maximum.
template <int NU>
__device__ __forceinline__ void softmax_update(f32x16_t (&s)[NU], f32x16_t (&o)[4], float& m_i,
                                               float& l_i, float cs, float shift, float off) {
  float mr = -INFINITY;
#pragma unroll
  for (int u = 0; u < NU; ++u)
#pragma unroll
    for (int e = 0; e < 16; ++e) mr = fmaxf(mr, s[u][e]);
  mr = fmaxf(mr, __shfl_xor(mr, 32, 64));
  const float mx = mr == -INFINITY ? -INFINITY : fmaf(mr, cs, shift);
  // m_new stays -inf only while no key of this row has been visible; the
  // update is then the identity (alpha = 1, p = 0), without branching the
  // wave away from the MFMAs that follow.
  const float m_new = fmaxf(m_i, mx);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  if (__any(m_new != m_i)) {
    const float alpha = fast_exp2(m_i - m_use);
    l_i *= alpha;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
  }
  m_i = m_new;
  const float bias = shift + off - m_use;
  float ls = 0.f;
#pragma unroll
  for (int u = 0; u < NU; ++u)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float pv = fast_exp2(fmaf(s[u][e], cs, bias));
      s[u][e] = pv;
      ls += pv;
    }
  l_i += ls;
}

// Running state of the RT query-row tiles of one wave.
template <int RT>
struct RowState {
  f32x16_t o[RT][4];   // O^T accumulators: o[rt][dt][4i+j] = O[row][32dt + 8i + 4*half + j]
  float m[RT], l[RT];  // running maximum (log2 units) and row sum
};

// One bf16 step of 64 keys for all RT row tiles of the wave; every LDS
// fragment read feeds RT MFMAs. KIND 0: kept keys key0 .. key0+63 (diag:
// causal mask against pos[rt]). KIND 1: correction, column k is used iff
// k < nv and todo[k] (logit shift +7, PV weights x pv_scale).
template <int KIND, int RT>
__device__ __forceinline__ void step_bf16(const uint4* st, const uint8_t* todo, int nv,
                                          const bf16x8_t (&qb)[RT][8], RowState<RT>& rs,
                                          float cs, float off, float pv_scale, int key0,
                                          const int (&pos)[RT], bool diag) {
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5, l32 = lane & 31;
  const int g16 = lane >> 4, i16 = lane & 15;
  const int sidx = i16 >> 2, r4 = i16 & 3;
  const uint4* vt = st + kStep * 16;
#pragma unroll 1
  for (int u = 0; u < 2; ++u) {          // 32 keys at a time
    f32x16_t s[RT][1];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) s[rt][0] = f32x16_t{};
    const int r = 32 * u + l32;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, st[kslot16(r, 2 * ds + half)]);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        s[rt][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[rt][ds], s[rt][0], 0, 0, 0);
    }
    // key of s[rt][0][4i+j] is 32u + 8i + 4*half + j
    if (KIND == 1 || diag) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = 32 * u + 8 * i + 4 * half + j;
            const bool drop = KIND == 1 ? !(key < nv && todo[key]) : (key0 + key > pos[rt]);
            s[rt][0][4 * i + j] = drop ? -INFINITY : s[rt][0][4 * i + j];
          }
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      softmax_update<1>(s[rt], rs.o[rt], rs.m[rt], rs.l[rt], cs, KIND == 1 ? 7.0f : 0.0f, off);

    // O^T += V^T P^T, 16 keys per MFMA: slot i' of lane half H is key
    // 32u + 16a + 8(i'/4) + 4H + i'%4, i.e. s[rt][0][8a + i'].
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      bf16x8_t pb[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        uint32_t pw[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float x0 = s[rt][0][8 * a + 2 * q], x1 = s[rt][0][8 * a + 2 * q + 1];
          pw[q] = KIND == 1 ? pack_bf16x2(x0 * pv_scale, x1 * pv_scale) : pack_bf16x2(x0, x1);
        }
        pb[rt] = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        i16x4_t rd[2];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const int key = 32 * u + 16 * a + 8 * tt + 4 * (g16 >> 1) + sidx;
          const int d = 32 * dt + 16 * (g16 & 1) + 4 * r4;
          const int byte = vslot16(key, d >> 3) * 16 + (d & 7) * 2;
          rd[tt] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)((lds_char_t*)vt + byte));
        }
        const i32x2_t r0 = __builtin_bit_cast(i32x2_t, rd[0]);
        const i32x2_t r1 = __builtin_bit_cast(i32x2_t, rd[1]);
        const bf16x8_t va = __builtin_bit_cast(bf16x8_t, (i32x4_t){r0[0], r0[1], r1[0], r1[1]});
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          rs.o[rt][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[rt], rs.o[rt][dt], 0, 0, 0);
      }
    }
  }
}

// Four e4m3 codes (round to nearest even) of four non-negative floats <= 448.
__device__ __forceinline__ int pack_e4m3x4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

// One fp8 step of 64 kept keys key0 .. key0+63 for all RT row tiles.
template <int RT>
__device__ __forceinline__ void step_fp8(const uint4* st, const i32x8_t (&qf)[RT][2],
                                         RowState<RT>& rs, float cs, int key0,
                                         const int (&pos)[RT], bool diag) {
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5, l32 = lane & 31;
  f32x16_t s[RT][2];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) s[rt][0] = s[rt][1] = f32x16_t{};
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int r = 32 * u + l32;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      const uint4 c0 = st[kslot8(r, 4 * ds + 2 * half)];
      const uint4 c1 = st[kslot8(r, 4 * ds + 2 * half + 1)];
      const i32x8_t av = {(int)c0.x, (int)c0.y, (int)c0.z, (int)c0.w,
                          (int)c1.x, (int)c1.y, (int)c1.z, (int)c1.w};
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        s[rt][u] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, qf[rt][ds], s[rt][u], 0, 0, 0,
                                                                   0, 0, 0);
    }
  }
  if (diag) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = 32 * u + 8 * i + 4 * half + j;
            s[rt][u][4 * i + j] = (key0 + key > pos[rt]) ? -INFINITY : s[rt][u][4 * i + j];
          }
  }
  // O^T += V^T P^T over the 64 keys: byte b of lane half H is the key of
  // s[b/16][b%16], i.e. 16(b/8) + 8((b%8)/4) + 4H + b%4.
  i32x8_t pb[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    softmax_update<2>(s[rt], rs.o[rt], rs.m[rt], rs.l[rt], cs, 0.0f, 8.0f);
    int pk[2][4];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pk[u][q] = pack_e4m3x4(s[rt][u][4 * q], s[rt][u][4 * q + 1], s[rt][u][4 * q + 2],
                               s[rt][u][4 * q + 3]);
    pb[rt] = (i32x8_t){pk[0][0], pk[0][1], pk[0][2], pk[0][3], pk[1][0], pk[1][1], pk[1][2], pk[1][3]};
  }
  const int g16 = lane >> 4, i16 = lane & 15;
  const int sidx = i16 >> 1, r2 = i16 & 1;
  const int H = g16 >> 1;
  const uint4* vt = st + kStep * 8;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    i32x2_t rd[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int key = 16 * t + 8 * (sidx >> 2) + 4 * H + (sidx & 3);
      const int c = 2 * dt + (g16 & 1);
      const int byte = vslot8(key, c) * 16 + 8 * r2;
      rd[t] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2_t*)((lds_char_t*)vt + byte));
    }
    const i32x8_t va = {rd[0][0], rd[0][1], rd[1][0], rd[1][1], rd[2][0], rd[2][1], rd[3][0], rd[3][1]};
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      rs.o[rt][dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(va, pb[rt], rs.o[rt][dt], 0, 0,
                                                                     0, 0, 0, 0);
  }
}

template <int FP8, int W, int RT>
__global__ __launch_bounds__(64 * W, 1) void attend_kernel(Problem p, Pooled pooled,
                                                                const uint8_t* __restrict__ mask,
                                                                KeptLists kl,
                                                                uint16_t* __restrict__ out,
                                                                float* __restrict__ lse) {
  __shared__ uint4 ring[kRingU4];
  __shared__ uint8_t todo[kMaxBlocks];      // correction: J < I not kept
  __shared__ uint8_t cflag[kMaxBlocks / kBlock];
  __shared__ int32_t clist[kMaxBlocks / kBlock];
  __shared__ int ncl;

  constexpr int M = 32 * RT * W;            // packed rows per workgroup
  const int wpu = p.g * kBlock / M;         // workgroups per unit
  const int x = blockIdx.x;
  const int xcd = x & 7, k = x >> 3;
  const int u = 8 * (k / wpu) + xcd;
  const int msub = k % wpu;
  const int nbh = p.batch * p.hkv;
  const int nunits = p.nbmax * nbh;
  if (u >= nunits) return;
  const int I = p.nbmax - 1 - u / nbh;
  const int bh = u % nbh;
  const int b = bh / p.hkv, h = bh % p.hkv;
  const int64_t tok0 = p.cu[b];
  const int L = p.cu[b + 1] - (int)tok0;
  const int n = (L + kBlock - 1) / kBlock;
  if (I >= n) return;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int G = p.g;
  const int64_t row = ((int64_t)b * p.hkv + h) * p.nbmax + I;

  // this lane's query rows (packed rows of Eq. packgqa): one per row tile;
  // all of them belong to the same query head because G divides 32
  int pos[RT];
  bool qvalid[RT];
  int64_t qoff[RT];
  const int pr0 = msub * M + w * 32 * RT + l32;
  const int hq = h * G + pr0 % G;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int pr = pr0 + 32 * rt;
    pos[rt] = I * kBlock + pr / G;
    qvalid[rt] = pos[rt] < L;
    qoff[rt] = ((tok0 + pos[rt]) * p.hq + hq) * kHeadDim;   // element index
  }

  RowState<RT> rs;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) rs.o[rt][dt] = f32x16_t{};
    rs.m[rt] = -INFINITY;
    rs.l[rt] = 0.f;
  }
  float qsc = FP8 ? p.q_scale[hq] : 1.f;
  float vsc = FP8 ? p.v_scale[h] : 1.f;
  float ksc = FP8 ? p.k_scale[h] : 1.f;
  const float off = FP8 ? 8.f : 0.f;        // log2 of the probability offset
  asm volatile("" : "+v"(qsc), "+v"(vsc), "+v"(ksc));  // loads complete before the rings

  // ---- kept blocks: steps s -> kept index cnt-1-s/2, half s%2
  {
    const uint8_t* K = (const uint8_t*)p.k;
    const uint8_t* V = (const uint8_t*)p.v;
    constexpr int esz = FP8 ? 1 : 2;
    const int cnt = kl.cnt[row];
    const int32_t* kidx = kl.idx + row * p.nbmax;
    const int64_t rowbytes = (int64_t)p.hkv * kHeadDim * esz;     // one token slot of the pool
    const int64_t hbytes = (int64_t)h * kHeadDim * esz;
    constexpr int RPG = FP8 ? 8 : 4;
    // a page holding whole copy groups lets one scalar table read serve a copy
    const bool uniform_pages = p.pm.page == 0 || (p.pm.shift >= 0 && p.pm.page >= RPG);
    const int32_t* ptab = p.pm.table + (int64_t)b * p.pm.stride;

    bf16x8_t qb[FP8 ? 1 : RT][8];
    i32x8_t qf[FP8 ? RT : 1][2];
    if (!FP8) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const uint16_t* qrow = (const uint16_t*)p.q + qoff[rt];
#pragma unroll
        for (int ds = 0; ds < 8; ++ds) {
          uint4 v = make_uint4(0, 0, 0, 0);
          if (qvalid[rt]) v = *(const uint4*)(qrow + 16 * ds + 8 * half);
          qb[rt][ds] = __builtin_bit_cast(bf16x8_t, v);
          asm volatile("" : "+v"(qb[rt][ds]));
        }
      }
    } else {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
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
      }
    }
    const float cs = FP8 ? p.scale_log2 * qsc * ksc : p.scale_log2;

    auto issue = [&](uint4* st, int s) {
      const int J = sload_i32(kidx + (cnt - 1 - (s >> 1)));
      const int key0 = J * kBlock + kStep * (s & 1);
      const int nvalid = L - key0;                       // <= 0: the half lies past the sequence
      // rows past the sequence repeat a valid row of the block (finite data)
      const int t0 = nvalid > 0 ? key0 : J * kBlock;
      copy_rows<W, FP8>(st, K, V, [&](int r0, int r) -> int64_t {
        const int rg = nvalid > 0 && r0 < nvalid ? r0 : 0;
        const int rr = nvalid > 0 && r < nvalid ? r : rg;
        int64_t slot;
        if (p.pm.page == 0) {
          slot = tok0 + t0 + rr;
        } else if (uniform_pages) {
          const int pi = __builtin_amdgcn_readfirstlane((t0 + rg) >> p.pm.shift);
          const int64_t pg = sload_i32(ptab + pi);
          slot = pg * p.pm.page + ((t0 + rr) & (p.pm.page - 1));
        } else {
          slot = slot_of(p.pm, b, tok0, t0 + rr);
        }
        return slot * rowbytes + hbytes;
      });
    };
    auto compute = [&](const uint4* st, int s) {
      const int J = sload_i32(kidx + (cnt - 1 - (s >> 1)));
      const int key0 = J * kBlock + kStep * (s & 1);
      if constexpr (FP8) step_fp8<RT>(st, qf, rs, cs, key0, pos, J == I);
      else step_bf16<0, RT>(st, nullptr, 0, qb, rs, cs, off, 1.f, key0, pos, J == I);
    };
    using C = Copies<W, FP8>;
    run_ring<C::nst, C::per_step>(ring, C::stage_u4, 2 * cnt, issue, compute);
  }

  // ---- mean correction over the pruned blocks J < I
  if (p.corr && I > 0) {
    const uint8_t* mrow = mask + row * p.nbmax;
    const int nch = (I + kBlock - 1) / kBlock;
    for (int c = tid; c < nch; c += 64 * W) cflag[c] = 0;
    __syncthreads();
    for (int J = tid; J < I; J += 64 * W) {
      const uint8_t f = !(mrow[J] & 1);
      todo[J] = f;
      if (f) cflag[J / kBlock] = 1;
    }
    __syncthreads();
    if (tid == 0) {
      int c2 = 0;
      for (int c = 0; c < nch; ++c)
        if (cflag[c]) clist[c2++] = c;
      ncl = c2;
    }
    __syncthreads();
    const int nc = ncl;
    if (nc > 0) {
      // Q as bf16 (fp8 codes widen exactly); the fp8 scale goes into cs.
      bf16x8_t qb[RT][8];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int ds = 0; ds < 8; ++ds) {
          uint4 v = make_uint4(0, 0, 0, 0);
          if (qvalid[rt]) {
            if (!FP8) {
              v = *(const uint4*)((const uint16_t*)p.q + qoff[rt] + 16 * ds + 8 * half);
            } else {
              const uint2 cc = *(const uint2*)((const uint8_t*)p.q + qoff[rt] + 16 * ds + 8 * half);
              uint32_t wv[2] = {cc.x, cc.y};
              uint32_t ow[4];
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const uint32_t src = wv[i >> 1] >> (16 * (i & 1));
                ow[i] = e4m3_to_bf16(src & 0xFF) | (e4m3_to_bf16((src >> 8) & 0xFF) << 16);
              }
              v = make_uint4(ow[0], ow[1], ow[2], ow[3]);
            }
          }
          qb[rt][ds] = __builtin_bit_cast(bf16x8_t, v);
          asm volatile("" : "+v"(qb[rt][ds]));
        }
      // fp8: O accumulates code-valued V (c_v applied at the end), so the
      // real-valued vbar enters with weight 1/c_v.
      const float pv_scale = FP8 ? 1.f / vsc : 1.f;
      const float cs = p.scale_log2 * qsc;
      const int64_t pbase = ((int64_t)b * p.hkv + h) * p.nbmax * kHeadDim;
      const uint8_t* Kh = (const uint8_t*)(pooled.khat + pbase);
      const uint8_t* Vh = (const uint8_t*)(pooled.vbar + pbase);
      auto issue = [&](uint4* st, int s) {
        const int c0 = clist[s >> 1] * kBlock;
        const int j0 = c0 + kStep * (s & 1);
        const int nv = I - j0;                           // <= 0: the half is all masked
        copy_rows<W, 0>(st, Kh, Vh, [&](int r0, int r) -> int64_t {
          (void)r0;
          const int jr = r < nv ? j0 + r : c0;            // past I: repeat a valid row
          return (int64_t)jr * kHeadDim * 2;
        });
      };
      auto compute = [&](const uint4* st, int s) {
        const int j0 = clist[s >> 1] * kBlock + kStep * (s & 1);
        step_bf16<1, RT>(st, todo + j0, I - j0, qb, rs, cs, off, pv_scale, 0, pos, false);
      };
      using C = Copies<W, 0>;
      run_ring<C::nst, C::per_step>(ring, C::stage_u4, 2 * nc, issue, compute);
    }
  }

  // epilogue: O = c_v O^T / l, LSE = (m + log2 l - off) ln 2
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
      lse[(tok0 + pos[rt]) * p.hq + hq] = (rs.m[rt] + fast_log2(l_tot) - off) * kLn2;
  }
}

template <int FP8, int W, int RT>
void launch_cfg(const Problem& p, const Pooled& pooled, const uint8_t* mask, const KeptLists& kl,
                void* out, float* lse, hipStream_t s) {
  const int64_t nunits = (int64_t)p.nbmax * p.batch * p.hkv;
  const int64_t units8 = (nunits + 7) / 8 * 8;
  const int wpu = p.g * kBlock / (32 * RT * W);
  const unsigned grid = (unsigned)(units8 * wpu);
  attend_kernel<FP8, W, RT><<<grid, 64 * W, 0, s>>>(p, pooled, mask, kl, (uint16_t*)out, lse);
}

template <int FP8>
void launch_dt(const Problem& p, const Pooled& pooled, const uint8_t* mask, const KeptLists& kl,
               void* out, float* lse, hipStream_t s) {
  // 32 query rows per wave; 8 waves (two per SIMD) when the unit has at
  // least 256 packed rows, else 4
  if (p.g == 1) launch_cfg<FP8, 4, 1>(p, pooled, mask, kl, out, lse, s);
  else launch_cfg<FP8, 8, 1>(p, pooled, mask, kl, out, lse, s);
}

}  // namespace

hipError_t launch_attend(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                         const KeptLists& kl, void* out, float* lse, hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  if (p.fp8) launch_dt<1>(p, pooled, mask, kl, out, lse, s);
  else launch_dt<0>(p, pooled, mask, kl, out, lse, s);
  return hipGetLastError();
}

}  // namespace fp2

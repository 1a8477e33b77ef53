// Sparse attention over the kept key blocks with the mean correction
// (Sec. 3.2 Eq. correction, Sec. 3.3; Algorithm 1 steps 6-11).
//
// Work unit: (sequence b, KV head h, query block I) of the packed query rows
// of Eq. packgqa; each workgroup (4 waves) takes 128 of the g*B packed rows,
// so one K/V tile in LDS serves all g query heads of the group. Units are
// dealt heaviest-first and the g workgroups of a unit go to the same XCD
// (consecutive dispatch slots of one XCD), so they share K/V through its L2.
//
// Per kept block J (walked from the last kept index down, Eq. csr):
//  - the 128 key and value rows are fetched through the page table (Eq.
//    page) into LDS, row-major, with an XOR swizzle of the 16-byte chunks;
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
//
// After the kept blocks, the pruned blocks J < I (mask bit 0 clear) enter as
// extra 128-wide chunks of pooled means: keys khat_J, values vbar_J (bf16,
// real units, bf16 MFMA for both dtypes), logits shifted by log2|B_J| = 7
// (Sec. 3.2 implementation paragraph); chunks without a pruned block are
// skipped.
#include "kernels.h"

namespace fp2 {

namespace {

constexpr int kThreads = 256;   // 4 waves x 32 query rows
constexpr float kLn2 = 0.69314718055994530942f;

typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef __attribute__((address_space(3))) i32x2_t lds_i32x2_t;
typedef __attribute__((address_space(3))) char lds_char_t;

struct Smem {
  union {
    struct {                 // bf16 tile: 128 rows x 16 chunks of 8 values
      uint4 k[kBlock * 16];
      uint4 v[kBlock * 16];
    } h;
    struct {                 // fp8 tile: 128 rows x 8 chunks of 16 codes
      uint4 k[kBlock * 8];
      uint4 v[kBlock * 8];
    } f;
  };
  uint8_t todo[kBlock];      // correction chunk: key column is a pruned block
};

// Swizzles: chunk c of row r is stored at slot (c ^ f(r)) of the row, chosen
// so that the MFMA operand reads of one instruction spread over all banks.
__device__ __forceinline__ int kchunk16(int r, int c) { return r * 16 + (c ^ (r & 15)); }
__device__ __forceinline__ int vchunk16(int r, int c) { return r * 16 + (c ^ (4 * (r & 3))); }
__device__ __forceinline__ int kchunk8(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }
__device__ __forceinline__ int vchunk8(int r, int c) { return r * 8 + (c ^ (2 * ((r >> 1) & 3))); }

// Stage 128 bf16 rows (row r from row_ptr, zero for r >= nvalid) of K and V.
template <class RowPtr>
__device__ __forceinline__ void stage_bf16(Smem& sm, int nvalid, RowPtr row_ptr) {
  const int tid = threadIdx.x;
  const int c = tid & 15;
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    uint4 kv[4], vv[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int r = (part * 4 + it) * 16 + (tid >> 4);
      kv[it] = make_uint4(0, 0, 0, 0);
      vv[it] = make_uint4(0, 0, 0, 0);
      if (r < nvalid) {
        const uint8_t* kp;
        const uint8_t* vp;
        row_ptr(r, kp, vp);
        kv[it] = *(const uint4*)(kp + c * 16);
        vv[it] = *(const uint4*)(vp + c * 16);
      }
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int r = (part * 4 + it) * 16 + (tid >> 4);
      sm.h.k[kchunk16(r, c)] = kv[it];
      sm.h.v[vchunk16(r, c)] = vv[it];
    }
  }
}

// Stage 128 fp8 rows of K and V (8 chunks of 16 codes per row).
template <class RowPtr>
__device__ __forceinline__ void stage_fp8(Smem& sm, int nvalid, RowPtr row_ptr) {
  const int tid = threadIdx.x;
  const int c = tid & 7;
  uint4 kv[4], vv[4];
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int r = it * 32 + (tid >> 3);
    kv[it] = make_uint4(0, 0, 0, 0);
    vv[it] = make_uint4(0, 0, 0, 0);
    if (r < nvalid) {
      const uint8_t* kp;
      const uint8_t* vp;
      row_ptr(r, kp, vp);
      kv[it] = *(const uint4*)(kp + c * 16);
      vv[it] = *(const uint4*)(vp + c * 16);
    }
  }
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int r = it * 32 + (tid >> 3);
    sm.f.k[kchunk8(r, c)] = kv[it];
    sm.f.v[vchunk8(r, c)] = vv[it];
  }
}

// Online-softmax update shared by both dtypes. s holds this lane's 64 logits
// (log2 units, -inf where masked); on return it holds 2^(x - m + off), the
// row sum of which has been added to l_i, and o/l_i have been rescaled.
__device__ __forceinline__ void softmax_update(f32x16_t (&s)[4], f32x16_t (&o)[4], float& m_i,
                                               float& l_i, float off) {
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  // m_new stays -inf only while no key of this row has been visible; the
  // update is then the identity (alpha = 1, p = 0), without branching the
  // wave away from the MFMAs that follow.
  const float m_new = fmaxf(m_i, mx);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = fast_exp2(m_i - m_use);
  m_i = m_new;
  l_i *= alpha;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
  const float mo = m_use - off;
  float ls = 0.f;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float pv = fast_exp2(s[kt][e] - mo);
      s[kt][e] = pv;
      ls += pv;
    }
  l_i += ls;
}

// bf16 tile of 128 keys. KIND 0: kept block (diag: causal mask). KIND 1:
// correction chunk (todo mask, logit shift +7, PV weights scaled by pv_scale).
template <int KIND>
__device__ __forceinline__ void tile_bf16(const Smem& sm, const bf16x8_t (&qb)[8], f32x16_t (&o)[4],
                                          float& m_i, float& l_i, float cscale, float off,
                                          float pv_scale, int key0, int pos, bool diag) {
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5, l32 = lane & 31;
  f32x16_t s[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    s[kt] = f32x16_t{};
    const int r = 32 * kt + l32;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, sm.h.k[kchunk16(r, 2 * ds + half)]);
      s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ds], s[kt], 0, 0, 0);
    }
  }
  // key of s[kt][4i+j] is 32kt + 8i + 4*half + j
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = 32 * kt + 8 * i + 4 * half + j;
        float x = s[kt][4 * i + j] * cscale;
        if (KIND == 1) x = sm.todo[key] ? x + 7.0f : -INFINITY;
        else if (diag) x = (key0 + key > pos) ? -INFINITY : x;
        s[kt][4 * i + j] = x;
      }
  softmax_update(s, o, m_i, l_i, off);

  // O^T += V^T P^T, 16 keys per MFMA: slot i' of lane half H is key
  // 32kt + 16a + 8(i'/4) + 4H + i'%4, i.e. s[kt][8a + i'].
  const int g16 = lane >> 4, i16 = lane & 15;
  const int sidx = i16 >> 2, r4 = i16 & 3;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      uint32_t pw[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pw[q] = KIND == 1 ? pack_bf16x2(s[kt][8 * a + 2 * q] * pv_scale, s[kt][8 * a + 2 * q + 1] * pv_scale)
                          : pack_bf16x2(s[kt][8 * a + 2 * q], s[kt][8 * a + 2 * q + 1]);
      const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        i16x4_t rd[2];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const int key = 32 * kt + 16 * a + 8 * tt + 4 * (g16 >> 1) + sidx;
          const int d = 32 * dt + 16 * (g16 & 1) + 4 * r4;
          const int byte = vchunk16(key, d >> 3) * 16 + (d & 7) * 2;
          rd[tt] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)((lds_char_t*)(sm.h.v) + byte));
        }
        const i32x2_t r0 = __builtin_bit_cast(i32x2_t, rd[0]);
        const i32x2_t r1 = __builtin_bit_cast(i32x2_t, rd[1]);
        const bf16x8_t va = __builtin_bit_cast(bf16x8_t, (i32x4_t){r0[0], r0[1], r1[0], r1[1]});
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[dt], 0, 0, 0);
      }
    }
}

// Four e4m3 codes (round to nearest even) of four non-negative floats <= 448.
__device__ __forceinline__ int pack_e4m3x4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
}

// fp8 kept block of 128 keys.
__device__ __forceinline__ void tile_fp8(const Smem& sm, const i32x8_t (&qf)[2], f32x16_t (&o)[4],
                                         float& m_i, float& l_i, float cscale, int key0, int pos,
                                         bool diag) {
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5, l32 = lane & 31;
  f32x16_t s[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    s[kt] = f32x16_t{};
    const int r = 32 * kt + l32;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      const uint4 c0 = sm.f.k[kchunk8(r, 4 * ds + 2 * half)];
      const uint4 c1 = sm.f.k[kchunk8(r, 4 * ds + 2 * half + 1)];
      const i32x8_t a = {(int)c0.x, (int)c0.y, (int)c0.z, (int)c0.w,
                         (int)c1.x, (int)c1.y, (int)c1.z, (int)c1.w};
      s[kt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, qf[ds], s[kt], 0, 0, 0, 0, 0, 0);
    }
  }
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = 32 * kt + 8 * i + 4 * half + j;
        float x = s[kt][4 * i + j] * cscale;
        if (diag) x = (key0 + key > pos) ? -INFINITY : x;
        s[kt][4 * i + j] = x;
      }
  softmax_update(s, o, m_i, l_i, 8.0f);

  // O^T += V^T P^T, 64 keys per MFMA (a = 0, 1): byte b of lane half H is the
  // key of s[2a + b/16][b%16], i.e. 64a + 16(b/8) + 8((b%8)/4) + 4H + b%4.
  int pk[4][4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      pk[kt][q] = pack_e4m3x4(s[kt][4 * q], s[kt][4 * q + 1], s[kt][4 * q + 2], s[kt][4 * q + 3]);
  const int g16 = lane >> 4, i16 = lane & 15;
  const int sidx = i16 >> 1, r2 = i16 & 1;
  const int H = g16 >> 1;
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const i32x8_t pb = {pk[2 * a][0], pk[2 * a][1], pk[2 * a][2], pk[2 * a][3],
                        pk[2 * a + 1][0], pk[2 * a + 1][1], pk[2 * a + 1][2], pk[2 * a + 1][3]};
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      i32x2_t rd[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = 64 * a + 16 * t + 8 * (sidx >> 2) + 4 * H + (sidx & 3);
        const int c = 2 * dt + (g16 & 1);
        const int byte = vchunk8(key, c) * 16 + 8 * r2;
        rd[t] = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2_t*)((lds_char_t*)(sm.f.v) + byte));
      }
      const i32x8_t va = {rd[0][0], rd[0][1], rd[1][0], rd[1][1], rd[2][0], rd[2][1], rd[3][0], rd[3][1]};
      o[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(va, pb, o[dt], 0, 0, 0, 0, 0, 0);
    }
  }
}

template <int FP8>
__global__ __launch_bounds__(kThreads, 2) void attend_kernel(Problem p, Pooled pooled,
                                                             const uint8_t* __restrict__ mask,
                                                             KeptLists kl,
                                                             uint16_t* __restrict__ out,
                                                             float* __restrict__ lse) {
  __shared__ Smem sm;
  const int G = p.g;
  const int x = blockIdx.x;
  const int xcd = x & 7, k = x >> 3;
  const int u = 8 * (k / G) + xcd;
  const int msub = k % G;
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
  const int64_t row = ((int64_t)b * p.hkv + h) * p.nbmax + I;

  // this lane's query row (packed row pr of Eq. packgqa)
  const int pr = msub * kBlock + w * 32 + l32;
  const int pos = I * kBlock + pr / G;
  const int hq = h * G + pr % G;
  const bool qvalid = pos < L;
  const int64_t qoff = ((tok0 + pos) * p.hq + hq) * kHeadDim;   // element index

  f32x16_t o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16_t{};
  float m_i = -INFINITY, l_i = 0.f;
  const float qsc = FP8 ? p.q_scale[hq] : 1.f;
  const float off = FP8 ? 8.f : 0.f;       // log2 of the probability offset

  const uint8_t* K = (const uint8_t*)p.k;
  const uint8_t* V = (const uint8_t*)p.v;
  constexpr int esz = FP8 ? 1 : 2;
  const int cnt = kl.cnt[row];
  const int16_t* kidx = kl.idx + row * p.nbmax;
  auto kv_row = [&](int key0) {
    return [&, key0](int r, const uint8_t*& kp, const uint8_t*& vp) {
      const int64_t slot = slot_of(p.pm, b, tok0, key0 + r);
      const int64_t off_e = (slot * p.hkv + h) * kHeadDim * esz;
      kp = K + off_e;
      vp = V + off_e;
    };
  };

  if (!FP8) {
    bf16x8_t qb[8];
    const uint16_t* qrow = (const uint16_t*)p.q + qoff;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qvalid) v = *(const uint4*)(qrow + 16 * ds + 8 * half);
      qb[ds] = __builtin_bit_cast(bf16x8_t, v);
    }
    for (int t = cnt - 1; t >= 0; --t) {
      const int J = kidx[t];
      const int key0 = J * kBlock;
      __syncthreads();
      stage_bf16(sm, min(kBlock, L - key0), kv_row(key0));
      __syncthreads();
      tile_bf16<0>(sm, qb, o, m_i, l_i, p.scale_log2, 0.f, 1.f, key0, pos, J == I);
    }
  } else {
    i32x8_t qf[2];
    const uint8_t* qrow = (const uint8_t*)p.q + qoff;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      uint4 c0 = make_uint4(0, 0, 0, 0), c1 = make_uint4(0, 0, 0, 0);
      if (qvalid) {
        c0 = *(const uint4*)(qrow + 64 * ds + 32 * half);
        c1 = *(const uint4*)(qrow + 64 * ds + 32 * half + 16);
      }
      qf[ds] = (i32x8_t){(int)c0.x, (int)c0.y, (int)c0.z, (int)c0.w,
                         (int)c1.x, (int)c1.y, (int)c1.z, (int)c1.w};
    }
    const float cqk = p.scale_log2 * qsc * p.k_scale[h];
    for (int t = cnt - 1; t >= 0; --t) {
      const int J = kidx[t];
      const int key0 = J * kBlock;
      __syncthreads();
      stage_fp8(sm, min(kBlock, L - key0), kv_row(key0));
      __syncthreads();
      tile_fp8(sm, qf, o, m_i, l_i, cqk, key0, pos, J == I);
    }
  }

  if (p.corr && I > 0) {
    // Q as bf16 (fp8 codes widen exactly); the fp8 scale goes into cscale.
    bf16x8_t qb[8];
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qvalid) {
        if (!FP8) {
          v = *(const uint4*)((const uint16_t*)p.q + qoff + 16 * ds + 8 * half);
        } else {
          const uint2 c = *(const uint2*)((const uint8_t*)p.q + qoff + 16 * ds + 8 * half);
          uint32_t wv[2] = {c.x, c.y};
          uint32_t ow[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t src = wv[i >> 1] >> (16 * (i & 1));
            ow[i] = e4m3_to_bf16(src & 0xFF) | (e4m3_to_bf16((src >> 8) & 0xFF) << 16);
          }
          v = make_uint4(ow[0], ow[1], ow[2], ow[3]);
        }
      }
      qb[ds] = __builtin_bit_cast(bf16x8_t, v);
    }
    // fp8: O accumulates code-valued V (c_v applied at the end), so the
    // real-valued vbar enters with weight 1/c_v.
    const float pv_scale = FP8 ? 1.f / p.v_scale[h] : 1.f;
    const float cs = p.scale_log2 * qsc;
    const uint8_t* mrow = mask + row * p.nbmax;
    const int64_t pbase = ((int64_t)b * p.hkv + h) * p.nbmax * kHeadDim;
    for (int c0 = 0; c0 < I; c0 += kBlock) {
      __syncthreads();
      int flag = 0;
      if (tid < kBlock) {
        const int J = c0 + tid;
        flag = (J < I) && !(mrow[J] & 1);
        sm.todo[tid] = (uint8_t)flag;
      }
      if (!__syncthreads_or(flag)) continue;
      stage_bf16(sm, min(kBlock, I - c0), [&](int r, const uint8_t*& kp, const uint8_t*& vp) {
        kp = (const uint8_t*)(pooled.khat + pbase + (int64_t)(c0 + r) * kHeadDim);
        vp = (const uint8_t*)(pooled.vbar + pbase + (int64_t)(c0 + r) * kHeadDim);
      });
      __syncthreads();
      tile_bf16<1>(sm, qb, o, m_i, l_i, cs, off, pv_scale, 0, pos, false);
    }
  }

  // epilogue: O = c_v O^T / l, LSE = (m + log2 l - off) ln 2
  const float l_tot = l_i + __shfl_xor(l_i, 32, 64);
  if (!qvalid) return;
  const float inv = (FP8 ? p.v_scale[h] : 1.f) / l_tot;
  uint16_t* orow = out + ((tok0 + pos) * p.hq + hq) * kHeadDim;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = 32 * dt + 8 * i + 4 * half;
      uint2 v;
      v.x = pack_bf16x2(o[dt][4 * i + 0] * inv, o[dt][4 * i + 1] * inv);
      v.y = pack_bf16x2(o[dt][4 * i + 2] * inv, o[dt][4 * i + 3] * inv);
      *(uint2*)(orow + d) = v;
    }
  if (lse && half == 0) lse[(tok0 + pos) * p.hq + hq] = (m_i + fast_log2(l_tot) - off) * kLn2;
}

}  // namespace

hipError_t launch_attend(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                         const KeptLists& kl, void* out, float* lse, hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  const int64_t nunits = (int64_t)p.nbmax * p.batch * p.hkv;
  const int64_t units8 = (nunits + 7) / 8 * 8;
  const unsigned grid = (unsigned)(units8 * p.g);
  if (p.fp8)
    attend_kernel<1><<<grid, kThreads, 0, s>>>(p, pooled, mask, kl, (uint16_t*)out, lse);
  else
    attend_kernel<0><<<grid, kThreads, 0, s>>>(p, pooled, mask, kl, (uint16_t*)out, lse);
  return hipGetLastError();
}

}  // namespace fp2

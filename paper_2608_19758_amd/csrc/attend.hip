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
//  - S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = key rows from LDS,
//    B = the wave's 32 query rows held in registers). Lane l then owns query
//    l%32 and 16 keys per 32-key subtile, so the row max/sum of the online
//    softmax need one exchange with lane l^32;
//  - O^T += V^T P^T: the probabilities are packed to bf16 straight from the
//    S^T accumulators into the B operand, and V^T comes from LDS with the
//    gfx950 transposing read ds_read_b64_tr_b16 (no transpose pass).
// After the kept blocks, the pruned blocks J < I (mask bit 0 clear) enter as
// extra 128-wide chunks of pooled means: keys khat_J, values vbar_J, logits
// shifted by log2|B_J| = 7 (Sec. 3.2 implementation paragraph); chunks
// without a pruned block are skipped.
#include "kernels.h"

namespace fp2 {

namespace {

constexpr int kThreads = 256;   // 4 waves x 32 query rows
constexpr float kLn2 = 0.69314718055994530942f;

typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

struct Smem {
  uint4 k[kBlock * 16];   // key rows: chunk c of key row r at r*16 + (c ^ (r & 15))
  uint4 v[kBlock * 16];   // value rows: chunk c of row r at r*16 + (c ^ (4*(r & 3)))
  uint8_t todo[kBlock];   // correction chunk: key column is a pruned block
};

__device__ __forceinline__ int kchunk(int r, int c) { return r * 16 + (c ^ (r & 15)); }
__device__ __forceinline__ int vchunk(int r, int c) { return r * 16 + (c ^ (4 * (r & 3))); }

// Stage 128 rows (row r from `src_row(r)` or zero) of K and V into LDS.
template <class RowPtr>
__device__ __forceinline__ void stage_rows(Smem& sm, int nvalid, RowPtr row_ptr) {
  const int tid = threadIdx.x;
  const int c = tid & 15;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    uint4 kv[4], vv[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int r = (half * 4 + it) * 16 + (tid >> 4);
      kv[it] = make_uint4(0, 0, 0, 0);
      vv[it] = make_uint4(0, 0, 0, 0);
      if (r < nvalid) {
        const uint16_t* kp;
        const uint16_t* vp;
        row_ptr(r, kp, vp);
        kv[it] = *(const uint4*)(kp + c * 8);
        vv[it] = *(const uint4*)(vp + c * 8);
      }
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int r = (half * 4 + it) * 16 + (tid >> 4);
      sm.k[kchunk(r, c)] = kv[it];
      sm.v[vchunk(r, c)] = vv[it];
    }
  }
}

// One 128-key tile: S^T, online softmax update, O^T += V^T P^T.
// kind 0: ordinary block (diag = causal mask needed); kind 1: correction chunk.
template <int KIND>
__device__ __forceinline__ void tile_step(const Smem& sm, const bf16x8_t (&qb)[8], f32x16_t (&o)[4],
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
    for (int ds = 0; ds < 8; ++ds) {
      const bf16x8_t a = __builtin_bit_cast(bf16x8_t, sm.k[kchunk(r, 2 * ds + half)]);
      s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ds], s[kt], 0, 0, 0);
    }
  }
  // logits in log2 units; key of s[kt][4i+j] is 32kt + 8i + 4*half + j
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = 32 * kt + 8 * i + 4 * half + j;
        float x = s[kt][4 * i + j] * cscale;
        if (KIND == 1) {
          x = sm.todo[key] ? x + 7.0f : -INFINITY;
        } else if (diag) {
          x = (key0 + key > pos) ? -INFINITY : x;
        }
        s[kt][4 * i + j] = x;
        mx = fmaxf(mx, x);
      }
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  // m_new stays -inf only while no key of this row has been visible; the
  // update is then the identity (alpha = 1, p = 0), without branching the
  // wave away from the MFMAs below.
  const float m_new = fmaxf(m_i, mx);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = fast_exp2(m_i - m_use);
  m_i = m_new;
  l_i *= alpha;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
  float ls = 0.f;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float pv = fast_exp2(s[kt][e] - m_use);
      s[kt][e] = pv;
      ls += pv;
    }
  l_i += ls;

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
      for (int q = 0; q < 4; ++q) pw[q] = pack_bf16x2(s[kt][8 * a + 2 * q], s[kt][8 * a + 2 * q + 1]);
      const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, make_uint4(pw[0], pw[1], pw[2], pw[3]));
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        i16x4_t rd[2];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const int key = 32 * kt + 16 * a + 8 * tt + 4 * (g16 >> 1) + sidx;
          const int d = 32 * dt + 16 * (g16 & 1) + 4 * r4;
          const int byte = vchunk(key, d >> 3) * 16 + (d & 7) * 2;
          rd[tt] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t*)((__attribute__((address_space(3))) char*)(sm.v) + byte));
        }
        const bf16x8_t va = __builtin_bit_cast(
            bf16x8_t, (i32x4_t){__builtin_bit_cast(i32x2_t, rd[0])[0], __builtin_bit_cast(i32x2_t, rd[0])[1],
                                __builtin_bit_cast(i32x2_t, rd[1])[0], __builtin_bit_cast(i32x2_t, rd[1])[1]});
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[dt], 0, 0, 0);
      }
    }
}

__global__ __launch_bounds__(kThreads, 2) void attend_bf16_kernel(Problem p, Pooled pooled,
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
  bf16x8_t qb[8];
  {
    const uint16_t* qrow = (const uint16_t*)p.q + ((tok0 + pos) * p.hq + hq) * kHeadDim;
#pragma unroll
    for (int ds = 0; ds < 8; ++ds) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qvalid) v = *(const uint4*)(qrow + 16 * ds + 8 * half);
      qb[ds] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x16_t o[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o[dt] = f32x16_t{};
  float m_i = -INFINITY, l_i = 0.f;
  const float cscale = p.scale_log2;

  const uint16_t* K = (const uint16_t*)p.k;
  const uint16_t* V = (const uint16_t*)p.v;
  const int cnt = kl.cnt[row];
  const int16_t* kidx = kl.idx + row * p.nbmax;

  for (int t = cnt - 1; t >= 0; --t) {
    const int J = kidx[t];
    const int key0 = J * kBlock;
    const int nvalid = min(kBlock, L - key0);
    __syncthreads();
    stage_rows(sm, nvalid, [&](int r, const uint16_t*& kp, const uint16_t*& vp) {
      const int64_t slot = slot_of(p.pm, b, tok0, key0 + r);
      const int64_t off = (slot * p.hkv + h) * kHeadDim;
      kp = K + off;
      vp = V + off;
    });
    __syncthreads();
    tile_step<0>(sm, qb, o, m_i, l_i, cscale, key0, pos, J == I);
  }

  if (p.corr && I > 0) {
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
      const int nv = min(kBlock, I - c0);
      stage_rows(sm, nv, [&](int r, const uint16_t*& kp, const uint16_t*& vp) {
        kp = pooled.khat + pbase + (int64_t)(c0 + r) * kHeadDim;
        vp = pooled.vbar + pbase + (int64_t)(c0 + r) * kHeadDim;
      });
      __syncthreads();
      tile_step<1>(sm, qb, o, m_i, l_i, cscale, 0, pos, false);
    }
  }

  // epilogue: O = O^T / l, LSE = (m + log2 l) ln 2
  const float l_tot = l_i + __shfl_xor(l_i, 32, 64);
  if (!qvalid) return;
  const float inv = 1.0f / l_tot;
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
  if (lse && half == 0) lse[(tok0 + pos) * p.hq + hq] = (m_i + fast_log2(l_tot)) * kLn2;
}

}  // namespace

hipError_t launch_attend(const Problem& p, const Pooled& pooled, const uint8_t* mask,
                         const KeptLists& kl, void* out, float* lse, hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  if (p.fp8) return hipErrorInvalidValue;   // fp8 attention not built yet
  const int64_t nunits = (int64_t)p.nbmax * p.batch * p.hkv;
  const int64_t units8 = (nunits + 7) / 8 * 8;
  const unsigned grid = (unsigned)(units8 * p.g);
  attend_bf16_kernel<<<grid, kThreads, 0, s>>>(p, pooled, mask, kl, (uint16_t*)out, lse);
  return hipGetLastError();
}

}  // namespace fp2

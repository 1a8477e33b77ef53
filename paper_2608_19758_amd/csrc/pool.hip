// Block means of K and V (Sec. 3.2, the pooled statistics kbar_J, vbar_J of
// Eq. correction; the block means of Algorithm 1). HBM-bound: every K/V byte of the
// sequence is read once with 16-byte loads through the page table.
//
// One workgroup per (key block J, KV head h, sequence b), 256 threads, over
// the sequence's KV tokens (a prefix included).
//  - bf16: thread (row group rg = tid/16, column chunk c = tid%16) sums tokens
//    rg, rg+16, ... of the block for columns 8c..8c+7 in fp64. Every bf16
//    value is exact in fp64 and so are the partial sums of realistic data, so
//    the mean does not depend on the summation order.
//  - fp8: each e4m3 value is an exact multiple of 2^-9 (the hardware decode
//    v_cvt_pk_f32_fp8 is exact); per-thread sums of 4 rows are exact in fp32,
//    the block sums exact 32-bit integers in units of 2^-9, and the mean is
//    (sum * 2^-9 * scale) / count in fp64 (the product is exact, the
//    division rounds once).
// The rounded key mean khat (bf16, one rounding from fp64) is the scoring key
// of Eq. fused_score and the surrogate key of the correction; vbar is the
// value mean in bf16. For fp8 inputs the correction runs on the matrix cores
// in fp8 like the kept keys (the pooled statistics quantized as Sec. 4 does
// under fp8): the kernel also writes the e4m3 code means e4m3(khat / k_scale)
// and e4m3(vbar / v_scale), derived from the bf16 means so that blocks taken
// from a means cache give the same codes. With a caller's means cache (chunked prefill), complete
// blocks it already holds are copied from it (512 bytes per block and head
// instead of the block's K/V), and every block pooled here is written to it.
#include "kernels.h"

namespace fp2 {

namespace {

constexpr int kThreads = 256;

// Element offset of (key block J of sequence b, KV head h) in the caller's
// means cache.
__device__ __forceinline__ int64_t cache_offset(const Problem& p, const MeansCache& mc, int b,
                                                int J, int h) {
  int64_t slot;
  if (p.pm.page == 0) {
    slot = (int64_t)b * p.nbk + J;
  } else {
    const int t = J * kBlock;
    const int pg = p.pm.shift >= 0 ? t >> p.pm.shift : t / p.pm.page;
    const int off = t - pg * p.pm.page;
    slot = (int64_t)p.pm.table[(int64_t)b * p.pm.stride + pg] * mc.per_page + off / kBlock;
  }
  return (slot * p.hkv + h) * kHeadDim;
}

template <int FP8>
__global__ __launch_bounds__(kThreads) void pool_kernel(Problem p, Pooled out, MeansCache mc) {
  const int J = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int64_t tok0 = p.cuk[b];
  const int L = p.cuk[b + 1] - (int)tok0;     // KV tokens, a prefix included
  const int64_t obase = (((int64_t)b * p.hkv + h) * p.nbk + J) * kHeadDim;
  const int n = (L + kBlock - 1) / kBlock;
  // fp8: the e4m3 code means, from the bf16 means (|mean code| <= 448)
  auto store8 = [&](uint16_t kh, uint16_t vb) {
    if (FP8 && out.khat8) {
      const float kc = __uint_as_float((uint32_t)kh << 16) / p.k_scale[h];
      const float vc = __uint_as_float((uint32_t)vb << 16) / p.v_scale[h];
      out.khat8[obase + tid] = (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(
                                             fminf(fmaxf(kc, -448.f), 448.f), 0.f, 0, false) & 0xFF);
      out.vbar8[obase + tid] = (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(
                                             fminf(fmaxf(vc, -448.f), 448.f), 0.f, 0, false) & 0xFF);
    }
  };
  if (J >= n) {
    if (tid < kHeadDim) {
      out.khat[obase + tid] = 0;
      out.vbar[obase + tid] = 0;
      store8(0, 0);
    }
    return;
  }
  const int64_t cbase = mc.khat ? cache_offset(p, mc, b, J, h) : 0;
  if (mc.khat && J < min(mc.pooled[b], L / kBlock)) {   // complete block, already pooled
    if (tid < kHeadDim) {
      const uint16_t kh = mc.khat[cbase + tid], vb = mc.vbar[cbase + tid];
      out.khat[obase + tid] = kh;
      out.vbar[obase + tid] = vb;
      store8(kh, vb);
    }
    return;
  }
  // the means go to the workspace and, with a cache, to the block's slot
  auto store = [&](uint16_t kh, uint16_t vb) {
    out.khat[obase + tid] = kh;
    out.vbar[obase + tid] = vb;
    store8(kh, vb);
    if (mc.khat) {
      mc.khat[cbase + tid] = kh;
      mc.vbar[cbase + tid] = vb;
    }
  };
  const int cnt = min(kBlock, L - J * kBlock);

  if constexpr (!FP8) {
    __shared__ double redk[16][kHeadDim];
    __shared__ double redv[16][kHeadDim];
    const int c = tid & 15, rg = tid >> 4;
    double ak[8], av[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) ak[i] = av[i] = 0.0;
    const uint16_t* K = (const uint16_t*)p.k;
    const uint16_t* V = (const uint16_t*)p.v;
    // all 2 x 8 loads of this thread in flight before the first sum; rows
    // past the block read nothing and add zero
    uint4 kv[8], vv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = rg + 16 * i;
      kv[i] = vv[i] = make_uint4(0, 0, 0, 0);
      if (r < cnt) {
        const int64_t off = (slot_of(p.pm, b, tok0, J * kBlock + r) * p.hkv + h) * kHeadDim + c * 8;
        kv[i] = *(const uint4*)(K + off);
        vv[i] = *(const uint4*)(V + off);
      }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint32_t kw[4] = {kv[r].x, kv[r].y, kv[r].z, kv[r].w};
      const uint32_t vw[4] = {vv[r].x, vv[r].y, vv[r].z, vv[r].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ak[2 * i] += (double)__uint_as_float(kw[i] << 16);
        ak[2 * i + 1] += (double)__uint_as_float(kw[i] & 0xFFFF0000u);
        av[2 * i] += (double)__uint_as_float(vw[i] << 16);
        av[2 * i + 1] += (double)__uint_as_float(vw[i] & 0xFFFF0000u);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      redk[rg][c * 8 + i] = ak[i];
      redv[rg][c * 8 + i] = av[i];
    }
    __syncthreads();
    if (tid < kHeadDim) {
      double sk = 0.0, sv = 0.0;
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        sk += redk[g][tid];
        sv += redv[g][tid];
      }
      store(f64_to_bf16(sk / (double)cnt), f64_to_bf16(sv / (double)cnt));
    }
  } else {
    // 8 threads per token row (16 codes each), 32 row groups.
    const int c = tid & 7, rg = tid >> 3;
    const uint8_t* K = (const uint8_t*)p.k;
    const uint8_t* V = (const uint8_t*)p.v;
    uint4 kv[4], vv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = rg + 32 * i;
      kv[i] = vv[i] = make_uint4(0, 0, 0, 0);
      if (r < cnt) {
        const int64_t off = (slot_of(p.pm, b, tok0, J * kBlock + r) * p.hkv + h) * kHeadDim + c * 16;
        kv[i] = *(const uint4*)(K + off);
        vv[i] = *(const uint4*)(V + off);
      }
    }
    // Codes decoded by the hardware (v_cvt_pk_f32_fp8, exact) and summed in
    // fp32 over the thread's 4 rows: every e4m3 value is a multiple of 2^-9
    // below 448 in magnitude, so a sum of 4 needs at most 20 significant
    // bits and is exact; times 512 it is an exact integer.
    float fk[16], fv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) fk[i] = fv[i] = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t kw[4] = {kv[r].x, kv[r].y, kv[r].z, kv[r].w};
      const uint32_t vw[4] = {vv[r].x, vv[r].y, vv[r].z, vv[r].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x2_t k0 = __builtin_amdgcn_cvt_pk_f32_fp8((int)kw[q], false);
        const f32x2_t k1 = __builtin_amdgcn_cvt_pk_f32_fp8((int)kw[q], true);
        const f32x2_t v0 = __builtin_amdgcn_cvt_pk_f32_fp8((int)vw[q], false);
        const f32x2_t v1 = __builtin_amdgcn_cvt_pk_f32_fp8((int)vw[q], true);
        fk[4 * q] += k0.x;
        fk[4 * q + 1] += k0.y;
        fk[4 * q + 2] += k1.x;
        fk[4 * q + 3] += k1.y;
        fv[4 * q] += v0.x;
        fv[4 * q + 1] += v0.y;
        fv[4 * q + 2] += v1.x;
        fv[4 * q + 3] += v1.y;
      }
    }
    int ak[16], av[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      ak[i] = (int)(fk[i] * 512.f);
      av[i] = (int)(fv[i] * 512.f);
    }
    // integer sums (exact): over the wave's 8 row groups with lane
    // exchanges, then over the 4 waves through LDS (4 KiB, so LDS does not
    // bound the workgroups per CU)
    __shared__ int redki[4][kHeadDim];
    __shared__ int redvi[4][kHeadDim];
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int o = 8; o < 64; o <<= 1) {
        ak[i] += __shfl_xor(ak[i], o, 64);
        av[i] += __shfl_xor(av[i], o, 64);
      }
    const int w = tid >> 6;
    if ((tid & 63) < 8) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        redki[w][c * 16 + i] = ak[i];
        redvi[w][c * 16 + i] = av[i];
      }
    }
    __syncthreads();
    if (tid < kHeadDim) {
      const int sk = (redki[0][tid] + redki[1][tid]) + (redki[2][tid] + redki[3][tid]);
      const int sv = (redvi[0][tid] + redvi[1][tid]) + (redvi[2][tid] + redvi[3][tid]);
      double ks = (double)p.k_scale[h], vs = (double)p.v_scale[h];
      store(f64_to_bf16(((double)sk * 0x1p-9 * ks) / (double)cnt),
            f64_to_bf16(((double)sv * 0x1p-9 * vs) / (double)cnt));
    }
  }
}

}  // namespace

hipError_t launch_pool(const Problem& p, Pooled out, hipStream_t s, const MeansCache& cache) {
  if (p.batch == 0 || p.nbk == 0) return hipSuccess;
  dim3 grid(p.nbk, p.hkv, p.batch);
  if (p.fp8)
    pool_kernel<1><<<grid, kThreads, 0, s>>>(p, out, cache);
  else
    pool_kernel<0><<<grid, kThreads, 0, s>>>(p, out, cache);
  return hipGetLastError();
}

}  // namespace fp2

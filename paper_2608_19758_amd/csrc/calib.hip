// Rate calibration: fixed instruction loops that keep every SIMD of the GPU
// busy with one kind of work, so that timing a call gives the rate this GPU
// sustains for it (the measured counterpart of the vendor peaks a roofline is
// priced against).
//
//   bf16 MFMA  v_mfma_f32_32x32x16_bf16         2*32*32*16 = 32768 FLOP per wave instruction
//   fp8 MFMA   v_mfma_f32_32x32x64_f8f6f4 (e4m3) 2*32*32*64 = 131072 FLOP per wave instruction
//   exp        v_exp_f32                         64 exps per wave instruction
//
// The matrix loops are the instructions the attention and scoring kernels
// issue. Each wave runs four independent accumulator chains (an MFMA never
// waits for its predecessor's result), the exp loop 32 independent chains
// per lane, x <- exp2(-x), which stay in (1/2, 1] (v_exp_f32's latency is
// several times its issue interval: eight chains on two waves per SIMD reach
// only about 60% of the rate). Two workgroups of four
// waves per compute unit: two waves per SIMD, as in the kernels. A result
// reaches memory only if it equals a tag the loops never produce (-1), so the
// work is kept and nothing is written.
#include "common.h"
#include "kernels.h"
#include "fp2.h"

namespace fp2 {
namespace {

constexpr int kCalThreads = 256;
constexpr int kCalWgPerCu = 2;
constexpr int kExpChains = 32;

template <int KIND>
__global__ __launch_bounds__(kCalThreads) void calib_kernel(int iters, float tag, float* sink) {
  const int lane = threadIdx.x & 63;
  float r;
  if constexpr (KIND == FP2_CALIB_MFMA_BF16) {
    bf16x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = (__bf16)(0.5f + 0.001f * (lane + i));
      b[i] = (__bf16)(0.25f - 0.001f * (lane ^ i));
    }
    f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
#pragma unroll 1
    for (int it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    }
    r = c0[lane & 15] + c1[lane & 15] + c2[lane & 15] + c3[lane & 15];
  } else if constexpr (KIND == FP2_CALIB_MFMA_FP8) {
    i32x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = 0x38383838 + ((lane + i) & 7);   // e4m3 codes near 1.0
      b[i] = 0x30303030 + ((lane ^ i) & 7);   // near 0.25
    }
    f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
#pragma unroll 1
    for (int it = 0; it < iters; ++it) {
      c0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c0, 0, 0, 0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c1, 0, 0, 0, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c2, 0, 0, 0, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c3, 0, 0, 0, 0, 0, 0);
    }
    r = c0[lane & 15] + c1[lane & 15] + c2[lane & 15] + c3[lane & 15];
  } else {
    float x[kExpChains];
#pragma unroll
    for (int i = 0; i < kExpChains; ++i) x[i] = 0.5f + 0.01f * i + 0.0001f * lane;
#pragma unroll 1
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int i = 0; i < kExpChains; ++i) x[i] = __builtin_amdgcn_exp2f(-x[i]);
    }
    r = 0.f;
#pragma unroll
    for (int i = 0; i < kExpChains; ++i) r += x[i];
  }
  if (r == tag) *sink = r;
}

}  // namespace

hipError_t launch_calib(int kind, int iters, float* sink, double* ops, hipStream_t s) {
  const int cus = device_compute_units();
  if (cus <= 0) return hipErrorNoDevice;
  const int grid = cus * kCalWgPerCu;
  const double waves = (double)grid * (kCalThreads / 64);
  const float tag = -1.f;   // every loop result is positive
  switch (kind) {
    case FP2_CALIB_MFMA_BF16:
      calib_kernel<FP2_CALIB_MFMA_BF16><<<grid, kCalThreads, 0, s>>>(iters, tag, sink);
      *ops = waves * iters * 4 * (2.0 * 32 * 32 * 16);
      break;
    case FP2_CALIB_MFMA_FP8:
      calib_kernel<FP2_CALIB_MFMA_FP8><<<grid, kCalThreads, 0, s>>>(iters, tag, sink);
      *ops = waves * iters * 4 * (2.0 * 32 * 32 * 64);
      break;
    default:
      calib_kernel<FP2_CALIB_EXP><<<grid, kCalThreads, 0, s>>>(iters, tag, sink);
      *ops = waves * 64 * iters * (double)kExpChains;
      break;
  }
  return hipGetLastError();
}

}  // namespace fp2

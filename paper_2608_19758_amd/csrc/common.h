// Device helpers shared by the gfx950 kernels of libfp2.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp2 {

constexpr int kHeadDim = 128;   // d
constexpr int kBlock = 128;     // selection block B (tokens)
constexpr int kMaxBlocks = 8192;  // blocks per sequence (max_seq_len <= 1M tokens)

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(8))) int i32x8_t;
typedef __attribute__((ext_vector_type(4))) int i32x4_t;
typedef __attribute__((ext_vector_type(2))) int i32x2_t;
typedef __attribute__((ext_vector_type(4))) short i16x4_t;

// ---------------------------------------------------------------------------
// Number formats
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// Two floats -> packed bf16 pair (v_cvt_pk_bf16_f32: round to nearest even).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// fp64 -> bf16 with a single rounding (nearest, ties to even), from the
// double's bit pattern: the exponent and 7 mantissa bits are kept, the 45
// dropped bits round the kept field (a carry moves into the exponent).
// Below 2^-126 the bf16 spacing is 2^-133: round x * 2^133 to an integer,
// which is then the encoding itself. Overflow gives infinity.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  uint32_t sign = (uint32_t)(u >> 63) << 15;
  uint64_t mag = u & 0x7FFFFFFFFFFFFFFFull;
  if (mag > 0x7FF0000000000000ull) return 0x7FC0;  // NaN
  double ax = __longlong_as_double((long long)mag);
  if (ax < 0x1p-126) return (uint16_t)(sign | (uint32_t)rint(ax * 0x1p133));
  uint64_t keep = mag >> 45;
  uint64_t rem = mag & ((1ull << 45) - 1);
  const uint64_t half = 1ull << 44;
  if (rem > half || (rem == half && (keep & 1))) keep += 1;
  int e = (int)(keep >> 7) - 1023 + 127;
  if (e >= 255) return (uint16_t)(sign | 0x7F80);
  return (uint16_t)(sign | ((uint32_t)e << 7) | (uint32_t)(keep & 0x7F));
}

typedef __attribute__((ext_vector_type(2))) float f32x2_t;

// Four OCP e4m3fn codes (the bytes of w, lowest first) -> two packed bf16
// pairs, two codes per v_cvt_scalef32_pk_bf16_fp8 (scale 1). Exact: every
// e4m3 value, subnormals included, is a bf16 value, and the instruction
// returns it for every non-NaN code (checked against an exact decode of all
// 256 codes).
__device__ __forceinline__ uint2 e4m3x4_to_bf16(uint32_t w) {
  typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));
  const bf16x2v_t lo = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, false);
  const bf16x2v_t hi = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, true);
  return make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

// ---------------------------------------------------------------------------
// Paged addressing (Sec. 3.3, Eq. page)
// ---------------------------------------------------------------------------

struct PageMap {
  const int32_t* table;   // [batch, stride]
  int32_t stride;         // max_pages_per_seq
  int32_t page;           // p (0: contiguous)
  int32_t shift;          // log2(p) when p is a power of two, else -1
};

// Pool slot of token t of sequence b whose first token row is tok0.
__device__ __forceinline__ int64_t slot_of(const PageMap& pm, int b, int64_t tok0, int t) {
  if (pm.page == 0) return tok0 + t;
  int pg, off;
  if (pm.shift >= 0) {
    pg = t >> pm.shift;
    off = t & (pm.page - 1);
  } else {
    pg = t / pm.page;
    off = t - pg * pm.page;
  }
  return (int64_t)pm.table[(int64_t)b * pm.stride + pg] * pm.page + off;
}

// ---------------------------------------------------------------------------
// Wave helpers (wave64)
// ---------------------------------------------------------------------------

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Workgroup barrier for LDS traffic: this wave's LDS operations complete,
// then all waves meet. Unlike __syncthreads(), outstanding global loads (and
// global->LDS copies) are not waited for, so prefetches stay in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Read-only metadata (sequence offsets, per-head scales) at a wave-uniform
// index through the constant address space: a scalar load, which waits only
// on the scalar counter, not behind the vector loads a kernel has in flight.
template <class T>
__device__ __forceinline__ T ld_uniform(const T* ptr, int64_t i) {
  return ((const __attribute__((address_space(4))) T*)ptr)[i];
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

}  // namespace fp2

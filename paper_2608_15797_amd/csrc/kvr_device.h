// Device-side helpers shared by the gfx950 kernels of libkvr.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvr {

typedef uint16_t bf16_t;  // raw bfloat16 bits
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef float float2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Cache-policy operand of the buffer loads of data that one launch reads once
// (cache rows, logits rows): the nt (streaming) hint, so the lines do not
// displace reused data in L2.
constexpr int kStreamLoad = 2;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two float32 -> bfloat16 (lo in the low half) with the hardware's
// round-to-nearest-even pack conversion (NaN stays a NaN). A bit-level
// software rounding compiles to a divergent branch per element, which made the
// output epilogue of the attention kernels about as long as a chunk's work.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((float2_t){lo, hi}, bf16x2_t));
}

template <typename T>
__device__ __forceinline__ T shfl_xor(T v, int mask) {
  return __shfl_xor(v, mask, kWave);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Wave-wide reductions.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, shfl_xor(v, m));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}

}  // namespace kvr

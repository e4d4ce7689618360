// Device helpers shared by the gfx950 kernels of the carryover drafter step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/carryover.h"

namespace co {

constexpr int kPage = 16;
constexpr int32_t kSkip = INT32_MIN;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

// fp32 -> bf16, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return static_cast<uint16_t>(b >> 16);
}

// Element conversions for the two storage types (fp32, bf16 bits).
template <typename T> __device__ __forceinline__ T to_elem(float v);
template <> __device__ __forceinline__ float to_elem<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t to_elem<uint16_t>(float v) { return f2bf(v); }

__device__ __forceinline__ bf16x8 as_bf16x8(u16x8 v) { return __builtin_bit_cast(bf16x8, v); }

// v_mfma_f32_16x16x32_bf16: acc[16x16] += A[16x32] * B[32x16].
// Lane l holds A row (l % 16), k = 8*(l/16) .. +7; B column (l % 16), same k;
// acc column (l % 16), rows 4*(l/16) .. +3.
__device__ __forceinline__ f32x4 mfma16x16x32(u16x8 a, u16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// Rotary angle of pair index i at position pos: pos * theta^(-2i/hd).  The product
// and the reduction to [-pi, pi] are done in fp64 so that positions of 10^5 keep
// fp32 accuracy after the reduction; sin/cos are then taken in fp32.
__device__ __forceinline__ double rope_inv_freq(int i, int hd, double log2_theta) {
  return exp2(-(2.0 * i / hd) * log2_theta);
}

__device__ __forceinline__ void rope_cos_sin(int pos, double inv_freq, float* c, float* s) {
  const double two_pi = 6.283185307179586476925286766559;
  double a = static_cast<double>(pos) * inv_freq;
  double k = rint(a * (1.0 / two_pi));
  float r = static_cast<float>(fma(-k, two_pi, a));
  sincosf(r, s, c);
}

__device__ __forceinline__ void set_status(int32_t* status, int32_t code) {
  if (status) atomicCAS(status, 0, code);
}

}  // namespace co

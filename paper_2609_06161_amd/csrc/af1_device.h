// Device-side helpers shared by the AF1 kernels: 16-bit float conversions
// and wave-level reductions for gfx950 (64-lane wavefronts).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace af1 {

constexpr int kWave = 64;

// bfloat16 pattern -> fp32 (exact: bfloat16 is the top half of binary32).
__device__ __forceinline__ float bf16_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// binary16 pattern -> fp32 (exact, hardware conversion).
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  _Float16 v = __builtin_bit_cast(_Float16, h);
  return (float)v;
}

// fp32 -> binary16 pattern, round to nearest even (hardware conversion).
__device__ __forceinline__ uint16_t f32_to_f16(float f) {
  _Float16 v = (_Float16)f;
  return __builtin_bit_cast(uint16_t, v);
}

// fp32 -> bfloat16 pattern, round to nearest even; NaN stays a quiet NaN
// with its payload (hardware conversion, one instruction on gfx950; checked
// identical to rounding the pattern by hand, u + 0x7fff + bit 16, on every
// upper half of the fp32 pattern with 128 lower halves each).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 v = (__bf16)f;
  return __builtin_bit_cast(uint16_t, v);
}

// Sum over the 64 lanes of a wave; every lane receives the total.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

}  // namespace af1

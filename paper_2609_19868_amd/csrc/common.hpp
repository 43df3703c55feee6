// Device helpers shared by the gfx950 kernels of libzarya.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zarya {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Finite stand-in for -inf as a running maximum: exp2(x - kNegBig) stays 0
// for masked scores (-inf) and never produces inf - inf.
constexpr float kNegBig = -1.0e30f;

// bf16 bits -> float (exact).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bf16 bits, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Two floats -> packed bf16x2 (low half = a), round to nearest even.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
}

__device__ __forceinline__ f32x16 mfma32x32x16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Work-item index for workgroup `bid` of a grid of `8 * per_xcd` workgroups.
// Workgroups are dispatched round-robin over the 8 XCDs (bid % 8); this gives
// each XCD a contiguous run of work items so that neighbouring items (which
// share operands) meet in the same L2.  Returns -1 for padding workgroups.
__device__ __forceinline__ int xcd_work_index(int bid, int per_xcd, int n_items) {
  const int w = (bid & 7) * per_xcd + (bid >> 3);
  return w < n_items ? w : -1;
}

}  // namespace zarya

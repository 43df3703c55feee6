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

typedef __attribute__((address_space(3))) void* lds_ptr;

// Direct global -> LDS load of 16 bytes per lane: lane l's bytes land at
// lds_base + 16*l (lds_base must be wave-uniform).  A plain (non-template)
// function: the builtin called straight from a kernel template stops clang
// from emitting that template's host-side launch stub.
__device__ __forceinline__ void dma16(const void* src, void* lds_base) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr)lds_base, 16, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are in flight
// (direct global->LDS loads count until their data is in LDS).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier that orders LDS accesses (this wave's LDS operations are
// complete) without waiting for the wave's outstanding global->LDS prefetches,
// which the __syncthreads() fence would drain.
__device__ __forceinline__ void block_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_ptr)p; }

// 16-byte LDS read issued exactly where it stands in the program (the
// compiler sinks plain LDS loads next to their use, which exposes the LDS
// latency in MFMA loops).  The result is only valid after a matching
// lds_wait<N>() that also names the fragment.
template <int OFF>
__device__ __forceinline__ bf16x8 lds_read_b128(uint32_t addr) {
  bf16x8 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

// Transposing 8-byte LDS read (ds_read_b64_tr_b16), issued where it stands;
// valid after a matching lds_wait<N>() / lds_tie.  In each 16-lane group,
// output lane i, element j comes from input lane 4*j + i/4, element i%4.
template <int OFF>
__device__ __forceinline__ v4i16 lds_read_tr16_b64(uint32_t addr) {
  v4i16 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

// Wait until at most N LDS operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void lds_wait() {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}

// Order a use of `x` after the preceding lds_wait (volatile asm statements
// keep their relative order; the tie makes x's consumers depend on it).
__device__ __forceinline__ void lds_tie(bf16x8& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void lds_tie(v4i16& x) { asm volatile("" : "+v"(x)); }

// max(a, b, c) in one v_max3_f32.  fmaxf() of values the compiler cannot
// prove quiet (MFMA results, say) costs an extra canonicalising max per
// operand; the operands here are finite.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Two floats -> packed bf16x2 (low half = a) with the hardware conversion
// (round to nearest even).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2_hw(float a, float b) {
  bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Work-item index for workgroup `bid` of a grid of `8 * per_xcd` workgroups.
// Workgroups are dispatched round-robin over the 8 XCDs (bid % 8); this gives
// each XCD a contiguous run of work items so that neighbouring items (which
// share operands) meet in the same L2.  Returns -1 for padding workgroups.
__device__ __forceinline__ int xcd_work_index(int bid, int per_xcd, int n_items) {
  const int w = (bid & 7) * per_xcd + (bid >> 3);
  return w < n_items ? w : -1;
}

}  // namespace zarya

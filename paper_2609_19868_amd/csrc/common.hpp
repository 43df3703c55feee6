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

// Buffer resource of `bytes` (< 4 GiB) bytes at `base` for raw byte-offset
// loads (stride 0; loads past the end return zeros).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Direct buffer->LDS copy of 16 bytes per lane: lane l reads the bytes at
// byte offset voffset + soffset of `rsrc` and writes them to LDS at
// lds_base + 16*l (lds_base wave-uniform).  Addresses are 32-bit offsets, so
// no 64-bit address arithmetic per load.  Only voffset is checked against the
// buffer's size (soffset is not): an access whose voffset is past the end
// reads zeros, while one whose soffset carries it past the end is not caught.
// AUX: cache-policy bits of the load (0: default; kLoadNonTemporal).
constexpr int kLoadNonTemporal = 2;
template <int AUX = 0>
__device__ __forceinline__ void dmab16(__amdgpu_buffer_rsrc_t rsrc, void* lds_base, uint32_t voffset,
                                       uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_ptr)lds_base, 16, voffset, soffset, 0, AUX);
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

// max(a, b, c): the compiler folds the two maxima into one v_max3_f32.  It
// must stay visible to the compiler (no inline assembly): the operands are
// often MFMA results, which a VALU instruction may read only after the wait
// states the compiler inserts for them.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  return __builtin_fmaxf(__builtin_fmaxf(a, b), c);
}

// max(x, x of lane ^ 32) on every lane, through v_permlane32_swap (a VALU
// exchange of the two 32-lane halves; no LDS round trip).  The swap leaves
// each lane holding its own value in one output and its partner's in the
// other, so the maximum of the two outputs is the pair's maximum.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max3f(__uint_as_float(r[0]), __uint_as_float(r[1]), __uint_as_float(r[1]));
}

// x + x of lane ^ 32 on every lane (the same value on both lanes of a pair:
// float addition is commutative).
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): four 32-bit words from
// a 128-bit counter and a 64-bit key.  Each round multiplies counter words 0
// and 2 by the two round constants, swaps the halves of the products into the
// other words under the round key, and bumps the key by the two Weyl constants.
__host__ __device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                        uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(c0, c1, c2, c3);
}

// The same generator for device code on gfx950: each round's two
// three-operand XORs (product half ^ counter word ^ key) are one v_bitop3_b32
// each (truth table 0x96 = a ^ b ^ c).  Bit-identical to philox4x32_10.
__device__ __forceinline__ uint4 philox4x32_10_dev(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                                   uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(c0, c1, c2, c3);
}

// Gumbel part of a perturbed score in the log2 domain: -log2(-log2 u) with
// u = ((x >> 9) + 1/2) * 2^-23 in (0, 1), exact in float32.  Adding it to
// z * log2(e) / T gives log2(e) * (z / T + G) up to a constant, G standard
// Gumbel, so the argmax is the Gumbel-max sample.
__device__ __forceinline__ float gumbel_log2(uint32_t x) {
  const float u = fmaf((float)(x >> 9), 0x1p-23f, 0x1p-24f);  // exact: 2k+1 < 2^24
  return -__builtin_amdgcn_logf(-__builtin_amdgcn_logf(u));
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

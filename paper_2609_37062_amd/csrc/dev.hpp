// Device helpers for gfx950: bf16 conversion, MFMA wrappers, wave reductions.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace vsk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(uint32_t u16) { return __uint_as_float(u16 << 16); }

// float -> bf16 bits, round to nearest even; NaN stays a (quiet) NaN.
// Both results are computed and one is selected: no branch per call.
__device__ __forceinline__ uint32_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t quiet_nan = ((u >> 16) | 0x40u) & 0xffffu;
  return (u & 0x7fffffffu) > 0x7f800000u ? quiet_nan : rounded;
}

__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) { return f2bf(lo) | (f2bf(hi) << 16); }

// double -> bf16 bits, round to nearest even.  Rounds to float first; that
// can only mislead the second rounding when the float lands exactly on a bf16
// midpoint from a double that was not one, which is resolved toward the double.
// (All three candidates are computed and one is selected: no branch.)
__device__ __forceinline__ uint32_t d2bf(double d) {
  const float f = static_cast<float>(d);
  const uint32_t u = __float_as_uint(f);
  const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t quiet_nan = ((u >> 16) | 0x40u) & 0xffffu;
  const bool tie = (u & 0xffffu) == 0x8000u && static_cast<double>(f) != d;
  const uint32_t resolved = ((u >> 16) + (fabs(d) > fabs(static_cast<double>(f)) ? 1u : 0u)) & 0xffffu;
  return (u & 0x7fffffffu) > 0x7f800000u ? quiet_nan : tie ? resolved : rounded;
}

// D(16x16,f32) += A(16x32) * B(32x16), bf16 operands, 8 per lane.
__device__ __forceinline__ f32x4 mfma_16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
// D(16x16,f32) += A(16x16) * B(16x16), bf16 operands, 4 per lane.
__device__ __forceinline__ f32x4 mfma_16x16x16(u32x2 a, u32x2 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4_t, a),
                                                   __builtin_bit_cast(bf16x4_t, b), c, 0, 0, 0);
}

// Write-through stores (sc1): the data goes to memory instead of staying in
// this XCD's L2, so a workgroup on another XCD of the same launch reads it
// once this wave's memory counter has drained.  Plain stores are only made
// visible to other XCDs at the end of the kernel.
__device__ __forceinline__ void store_wt(void* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store_wt(void* p, u32x2 v) {
  asm volatile("global_store_dwordx2 %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store_wt(void* p, uint32_t v) {
  asm volatile("global_store_dword %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store_wt(void* p, double v) { store_wt(p, __builtin_bit_cast(u32x2, v)); }
__device__ __forceinline__ void store_wt16(void* p, uint32_t v) {
  asm volatile("global_store_short %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}

// threadIdx.x through an opaque move: values derived from it inside a
// phase of a persistent kernel are then computed in that phase instead of
// being hoisted out of the surrounding loop and held in registers across
// every other phase.
// 16 bytes per lane from global memory straight into LDS: lane l's bytes land
// at lds + 16 l (the LDS address must be the same for the whole wave).  The
// load counts in the wave's vector-memory counter until its bytes are in LDS.
__device__ __forceinline__ void lds_load16(const u32x4* g, u32x4* lds) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Workgroup barrier without a memory fence, for rings filled by
// global-to-LDS loads.  __syncthreads() also fences, and before the fence the
// compiler waits for every outstanding load into LDS, which would drain the
// loads issued ahead.  Here a loading wave waits explicitly (s_waitcnt
// vmcnt(N)) for exactly the loads that must have landed, and a reading wave
// waits for its own LDS reads (lgkmcnt(0)) before the slot can be refilled.
// The empty asm statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void barrier_after_lds_reads() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void barrier_no_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int opaque_tid() {
  int t;
  asm volatile("v_mov_b32 %0, %1" : "=v"(t) : "v"(static_cast<int>(threadIdx.x)));
  return t;
}

__device__ __forceinline__ float shfl_xor(float v, int m) { return __shfl_xor(v, m, 64); }

// A value combined with lane l ^ 16 (or l ^ 32) through the gfx950 lane
// swaps (v_permlane16_swap / v_permlane32_swap: VALU, no LDS round trip).
// Swapping v with itself leaves each lane the pair {v[l], v[l ^ 16]} (resp.
// l ^ 32) in some order; max and + are symmetric, so both lanes of a pair
// get the same bits, as with a shuffle.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float add_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ int shfl_xor(int v, int m) { return __shfl_xor(v, m, 64); }

// (value, index) candidate for greedy argmax: larger value wins, equal values
// keep the lower index, NaN never wins (it is entered as -inf with index INT_MAX).
__device__ __forceinline__ void am_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

}  // namespace vsk

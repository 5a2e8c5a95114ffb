// Device-side helpers shared by the kernels: 16-bit float conversions, vector types,
// wave-size constants. Everything here is written for gfx950 (wave64, CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "../../include/aqmb.h"

namespace aqmb {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte streaming load (read once: non-temporal hint).
__device__ __forceinline__ uint4 load_stream16(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// 8-byte streaming load (same cache policy as load_stream16).
__device__ __forceinline__ uint2 load_stream8(const void* p) {
  typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
  const u32x2_t v = __builtin_nontemporal_load((const u32x2_t*)p);
  return make_uint2(v.x, v.y);
}

// Direct global->LDS load of 16 bytes per lane: lane l's bytes land at lds_base + 16 l (lds_base
// is an LDS byte address, uniform across the wave). Issued as inline assembly so the compiler
// neither serialises these loads against each other and against later LDS reads (it cannot see
// that the destinations are disjoint) nor waits for them; completion is awaited explicitly with
// wait_vmcnt before the barrier that publishes the data. Loads complete in issue order, so a
// wait for the loads the compiler issues itself is never too short.
__device__ __forceinline__ void load_lds16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(gptr) : "memory", "m0");
}

// s_waitcnt vmcnt(N), the other counters left at their maxima (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// LDS byte address of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// fp16 bits -> fp32 (exact; fp16 subnormals become fp32 normals).
__device__ __forceinline__ float f16_to_f32(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}
__device__ __forceinline__ float f16lo(uint32_t w) { return f16_to_f32(w & 0xFFFFu); }
__device__ __forceinline__ float f16hi(uint32_t w) { return f16_to_f32(w >> 16); }

// bf16 bits -> fp32 (exact).
__device__ __forceinline__ float bf16lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xFFFF0000u); }

// fp32 -> fp16 / bf16 bits, round to nearest even (the default rounding mode).
__device__ __forceinline__ uint16_t f32_to_f16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}
// Two values at once (one v_cvt_pk_bf16_f32 / v_cvt_pk_f16_f32, each half rounded to nearest
// even like the scalar conversions above).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, half2_t));
}

// acc + the fp16 value in the low or high half of w, rounded once to binary32 (an fma with 1.0:
// the product is exact, so the result is the binary32 sum, signed zeros included).
__device__ __forceinline__ float add_f16_lo(uint32_t w, float acc) {
  float d;
  asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel_hi:[1,0,0]" : "=v"(d) : "v"(w), "v"(acc));
  return d;
}
__device__ __forceinline__ float add_f16_hi(uint32_t w, float acc) {
  float d;
  asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(d) : "v"(w), "v"(acc));
  return d;
}

// fp32 dot of two fp16 pairs plus an fp32 addend (products exact in fp32).
__device__ __forceinline__ float dot2_f16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c, false);
}

// Output element store for the three output dtypes.
template <int DT> struct OutT;
template <> struct OutT<AQMB_F16> {
  static __device__ __forceinline__ void store(void* p, size_t i, float v) { ((uint16_t*)p)[i] = f32_to_f16_bits(v); }
};
template <> struct OutT<AQMB_BF16> {
  static __device__ __forceinline__ void store(void* p, size_t i, float v) { ((uint16_t*)p)[i] = f32_to_bf16_bits(v); }
};
template <> struct OutT<AQMB_F32> {
  static __device__ __forceinline__ void store(void* p, size_t i, float v) { ((float*)p)[i] = v; }
};

}  // namespace aqmb

// Device helpers shared by the kernel sources (vector types, buffer
// descriptors, wave-uniform values, bf16 / fp8 conversions).  Each translation
// unit gets its own internal copy.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rlda {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kRescaleLog2 = 8.f;          // lazy-rescale threshold of the online softmax (log2 units)
constexpr uint32_t kRsrcWord3 = 0x00020000u; // raw buffer, 32-bit data format
constexpr int kLoadNT = 2;                   // cache policy: non-temporal (KV is read once)
constexpr int kPastRange = 0x40000000;       // buffer offset beyond any descriptor's records: reads 0

__device__ __forceinline__ float neg_inf() { return -__builtin_huge_valf(); }

// Workgroup barrier for data exchanged through LDS only: this wave's LDS operations
// are complete, then s_barrier.  Unlike __syncthreads it does not wait for this
// wave's global stores to complete.  The memory clobber keeps the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Values equal in every lane, moved to scalar registers so that buffer
// descriptors and loop bounds built from them stay scalar.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int64_t uni64(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, (int)kRsrcWord3);
}

// Descriptor from wave-uniform inputs, kept in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_uni(const void* base, uint32_t bytes) {
  const int64_t a = uni64((int64_t)(uintptr_t)base);
  return make_rsrc((const void*)(uintptr_t)a, (uint32_t)uni((int)bytes));
}

// Two OCP E4M3FN bytes of `w` (bytes 0,1 or, with hi_half, bytes 2,3) as floats.
__device__ __forceinline__ f32x2 fp8x2_to_f32(uint32_t w, bool hi_half) {
  return hi_half ? __builtin_amdgcn_cvt_pk_f32_fp8(w, true) : __builtin_amdgcn_cvt_pk_f32_fp8(w, false);
}

#ifndef RLDA_FP8_DIRECT
#define RLDA_FP8_DIRECT 1
#endif
constexpr bool kFp8Direct = RLDA_FP8_DIRECT;   // fp8 -> bf16 operands in one conversion per pair

// Two e4m3 values (bytes 0, 1, or 2, 3 with hi_half) to a bf16 pair, low half first.
// Every e4m3 value is a bf16 value, and the scale is one, so the conversion is exact.
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w, bool hi_half) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 v = hi_half ? __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true)
                           : __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false);
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

}  // namespace
}  // namespace rlda

// Device-side helpers shared by the gfx950 kernels (kernels.hip, sgemv.hip, gemm.hip):
// vector types, bfloat16 conversion, 16x16x32 bf16 MFMA, reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctx.h"

namespace specdec {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// float -> bfloat16, round to nearest even; NaN stays NaN.  The conversion
// is gfx950's packed v_cvt_pk_bf16_f32 (one instruction for two values).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t f2bf_bits(float f) { return pack2(f, 0.f) & 0xffffu; }
__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)f2bf_bits(f); }

__device__ __forceinline__ u32x4 ld16(const bf16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ u32x2 ld8(const bf16_t* p) { return *reinterpret_cast<const u32x2*>(p); }
// Non-temporal 16-byte load, for weights (read once per pass): streamed with
// the nt hint they do not displace data that is reused.
__device__ __forceinline__ u32x4 ld16_nt(const bf16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}

// Device-coherent accesses for data handed between workgroups of one launch
// (possibly on different XCDs): relaxed agent-scope atomic loads and stores,
// which go to the device's coherence point instead of the XCD's L2.  A writer
// waits for its stores to complete (s_waitcnt) before it signals; a reader
// that saw the signal reads with ld_coh*.  No cache-wide writeback or
// invalidate is involved.
#define SD_GLOBAL __attribute__((address_space(1)))
__device__ __forceinline__ f32x4 ld_coh4(const float* p) {
  const SD_GLOBAL uint64_t* q = (const SD_GLOBAL uint64_t*)(p);
  const uint64_t a = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t b = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return f32x4{__uint_as_float((uint32_t)a), __uint_as_float((uint32_t)(a >> 32)), __uint_as_float((uint32_t)b),
               __uint_as_float((uint32_t)(b >> 32))};
}
__device__ __forceinline__ float2 ld_coh2(const float* p) {
  const uint64_t a =
      __hip_atomic_load((const SD_GLOBAL uint64_t*)(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)a), __uint_as_float((uint32_t)(a >> 32)));
}
__device__ __forceinline__ void st_coh4(float* p, f32x4 v) {
  SD_GLOBAL uint64_t* q = (SD_GLOBAL uint64_t*)(p);
  __hip_atomic_store(q, (uint64_t)__float_as_uint(v.x) | ((uint64_t)__float_as_uint(v.y) << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, (uint64_t)__float_as_uint(v.z) | ((uint64_t)__float_as_uint(v.w) << 32),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh2(float* p, float x, float y) {
  __hip_atomic_store((SD_GLOBAL uint64_t*)(p), (uint64_t)__float_as_uint(x) | ((uint64_t)__float_as_uint(y) << 32),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh_u32(void* p, uint32_t v) {
  __hip_atomic_store((SD_GLOBAL uint32_t*)(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_coh_u32(const void* p) {
  return __hip_atomic_load((const SD_GLOBAL uint32_t*)(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waits until every vector memory access of the wave has completed.
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Block-wide sum of one float per thread (blockDim.x a multiple of 64, <= 1024),
// in a fixed order.
__device__ float block_sum(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, nw = blockDim.x >> 6;
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += sh[i];
  __syncthreads();
  return t;
}

// Argmax pair reduction: larger value wins, equal values go to the lower index.
__device__ __forceinline__ void amax_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

}  // namespace specdec

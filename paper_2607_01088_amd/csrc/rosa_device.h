// Device-side helpers for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rosa {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;    // MFMA bf16 operand (8 per lane)
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;    // 32x32 MFMA accumulator
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) short i16x4;

// One 1 KB global -> LDS copy (lane i: 16 bytes from its own source to
// lds + 16 i), written as inline assembly so the compiler does not track it:
// its model of this copy makes it wait for every outstanding LDS read before
// the next MFMA, which would cap the LDS reads in flight at one.  The kernels
// wait for the copies themselves (vmcnt) and set M0, which nothing else in
// them uses; the s_nop is the wait state the M0 write needs before the copy.
// dma_1k_s takes a wave-uniform 64-bit base (SGPRs) plus a 32-bit per-lane
// byte offset; dma_1k a full per-lane address.
__device__ __forceinline__ void dma_1k(const void *src, uint32_t lds) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
#pragma clang diagnostic pop
}
__device__ __forceinline__ void dma_1k_s(const void *base, uint32_t off, uint32_t lds) {
  // The base is wave-uniform by construction; reading it through readfirstlane
  // keeps it in SGPRs even where the compiler cannot prove that.
  const uint64_t b64 = (uint64_t)(size_t)base;
  const uint64_t ub = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(b64 >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b64);
  const void *bs = (const void *)(size_t)ub;
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(bs), "s"(lds)
               : "memory", "m0");
#pragma clang diagnostic pop
}
__device__ __forceinline__ uint32_t lds_u32(const uint8_t *p) {
  return (uint32_t)(size_t)(__attribute__((address_space(3))) void *)(p);
}

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }  // RNE

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + expf(-x)); }

// tanh-approximate GELU: 0.5 x (1 + tanh(z)), z = sqrt(2/pi) (x + 0.044715 x^3),
// evaluated through the identity 0.5 (1 + tanh(z)) = 1 / (1 + e^(-2z)): one
// exponential and one reciprocal instead of a tanh.  For large |x| the
// exponential saturates to 0 or +inf, giving x or -0 exactly.
__device__ __forceinline__ float gelu_tanh_f(float x) {
  // x / (1 + 2^(k2 (x + 0.044715 x^3))); the hardware exp2 flushes results
  // below 2^-126 to 0, where 1 + e is 1 in fp32 anyway.
  const float k2 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float u = fmaf(x * x, k2 * 0.044715f, k2);
  const float e = __builtin_amdgcn_exp2f(x * u);
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

}  // namespace rosa

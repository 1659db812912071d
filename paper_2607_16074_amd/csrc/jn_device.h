// Device-side helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace jnx {

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round-to-nearest-even fp32 -> bf16 (hardware v_cvt on gfx950).
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
}

// ds_read_b64_tr_b16 at LDS address p + OFF bytes (in each 16-lane group,
// lane i receives element i % 4 of the 8-byte chunks that lanes 4e + i / 4
// address, e = 0..3), issued as inline assembly.  The compiler's wait
// insertion treats the builtin form as a read that may alias any LDS DMA in
// flight and puts a vmcnt(0) before it, which drains every prefetch that is
// in flight; the asm is invisible to that pass, so the caller waits
// (lgkmcnt) before it uses the result.
template <int OFF>
__device__ __forceinline__ uint64_t lds_read_tr_b16(const void* p) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
  uint64_t r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
  return r;
}

// v together with the value lane l ^ 16 (v_permlane16_swap) or l ^ 32
// (v_permlane32_swap) holds, without an LDS round trip.  The two come back
// in an order that differs between the lanes of a pair, so only commutative
// combinations (max, sum) of .x and .y are the same in both lanes.
__device__ __forceinline__ float2 lane_pair16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float2 lane_pair32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float max_xor16(float v) {
  const float2 p = lane_pair16(v);
  return fmaxf(p.x, p.y);
}

__device__ __forceinline__ float max_xor32(float v) {
  const float2 p = lane_pair32(v);
  return fmaxf(p.x, p.y);
}

__device__ __forceinline__ float sum_xor16(float v) {
  const float2 p = lane_pair16(v);
  return p.x + p.y;
}

__device__ __forceinline__ float sum_xor32(float v) {
  const float2 p = lane_pair32(v);
  return p.x + p.y;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// tanh-form GELU and its derivative, fp32.
__device__ __forceinline__ float gelu_f(float u) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * u * (1.0f + tanhf(c * (u + 0.044715f * u * u * u)));
}

// The same tanh-form GELU written as u / (1 + 2^(y)), y = -log2(e) * 2 sqrt(2/pi)
// * (u + 0.044715 u^3), with the log2(e) factor folded into the polynomial and
// the hardware exp2 / reciprocal (relative error ~1e-6, far below the bf16
// rounding of the values it produces).  Used in GEMM epilogues.
__device__ __forceinline__ float gelu_fast_f(float u) {
  const float y = u * (-2.302208198144325f - 0.1029432395800235f * u * u);
  return u * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(y));
}

__device__ __forceinline__ float gelu_grad_f(float u) {
  const float c = 0.7978845608028654f;
  float t = tanhf(c * (u + 0.044715f * u * u * u));
  return 0.5f * (1.0f + t) + 0.5f * u * (1.0f - t * t) * c * (1.0f + 3.0f * 0.044715f * u * u);
}

}  // namespace jnx

// RMSNorm over rows of the packed batch: one wavefront per row, the row held
// in registers between the sum-of-squares pass and the scaling pass, a
// butterfly wave reduction (deterministic order), fp32 math, bf16 output.
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

constexpr int kNormRowsPerBlock = 4;  // 4 waves, one row each

// Load VEC bf16 values starting at element `e` of a bf16 row.
template <int VEC>
__device__ __forceinline__ void load_bf(const uint16_t* row, int e, float* v) {
  if constexpr (VEC == 8) {
    uint4 q = *reinterpret_cast<const uint4*>(row + e);
    uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[2 * k] = __uint_as_float(w[k] << 16);
      v[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
    }
  } else if constexpr (VEC == 4) {
    uint2 q = *reinterpret_cast<const uint2*>(row + e);
    v[0] = __uint_as_float(q.x << 16);
    v[1] = __uint_as_float(q.x & 0xffff0000u);
    v[2] = __uint_as_float(q.y << 16);
    v[3] = __uint_as_float(q.y & 0xffff0000u);
  } else {
    uint32_t q = *reinterpret_cast<const uint32_t*>(row + e);
    v[0] = __uint_as_float(q << 16);
    v[1] = __uint_as_float(q & 0xffff0000u);
  }
}

template <int VEC>
__device__ __forceinline__ void load_f32(const float* row, int e, float* v) {
#pragma unroll
  for (int k = 0; k < VEC; k += 2) {
    float2 q = *reinterpret_cast<const float2*>(row + e + k);
    v[k] = q.x;
    v[k + 1] = q.y;
  }
}

template <int VEC>
__device__ __forceinline__ void store_f32(float* row, int e, const float* v) {
#pragma unroll
  for (int k = 0; k < VEC; k += 2) *reinterpret_cast<float2*>(row + e + k) = make_float2(v[k], v[k + 1]);
}

template <int VEC>
__device__ __forceinline__ void store_bf(uint16_t* row, int e, const float* v) {
  if constexpr (VEC == 8) {
    *reinterpret_cast<uint4*>(row + e) =
        make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
  } else if constexpr (VEC == 4) {
    *reinterpret_cast<uint2*>(row + e) = make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
  } else {
    *reinterpret_cast<uint32_t*>(row + e) = pack_bf2(v[0], v[1]);
  }
}

// IN_BF16: x is bf16 (the packed tokens); its fp32 widening is also written to
// x_out (the residual stream).  Otherwise x is the fp32 residual stream.
// Each lane owns elements (c*64 + lane)*VEC .. +VEC for c < NC.
template <int VEC, int NC, bool IN_BF16>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const void* __restrict__ xin, float* __restrict__ x_out,
                                                      const uint16_t* __restrict__ g, uint16_t* __restrict__ h,
                                                      int32_t rows, int32_t d, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kNormRowsPerBlock + (threadIdx.x >> 6);
  if (row >= rows) return;
  float v[NC][VEC];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int e = (c * 64 + lane) * VEC;
    if constexpr (IN_BF16)
      load_bf<VEC>(reinterpret_cast<const uint16_t*>(xin) + row * d, e, v[c]);
    else
      load_f32<VEC>(reinterpret_cast<const float*>(xin) + row * d, e, v[c]);
#pragma unroll
    for (int k = 0; k < VEC; ++k) ss += v[c][k] * v[c][k];
  }
  ss = wave_sum(ss);
  const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int e = (c * 64 + lane) * VEC;
    if constexpr (IN_BF16) store_f32<VEC>(x_out + row * d, e, v[c]);
    float gv[VEC], o[VEC];
    load_bf<VEC>(g, e, gv);
#pragma unroll
    for (int k = 0; k < VEC; ++k) o[k] = v[c][k] * r * gv[k];
    store_bf<VEC>(h + row * d, e, o);
  }
}

template <bool IN_BF16>
static hipError_t launch_rms(hipStream_t s, const void* x, float* x_out, const void* g, void* h, int32_t rows,
                             int32_t d, float eps) {
  dim3 grid((rows + kNormRowsPerBlock - 1) / kNormRowsPerBlock);
  auto G = reinterpret_cast<const uint16_t*>(g);
  auto H = reinterpret_cast<uint16_t*>(h);
#define JN_RMS(VEC, NC)                                                                     \
  if (d == 64 * (VEC) * (NC)) {                                                             \
    rmsnorm_kernel<VEC, NC, IN_BF16><<<grid, 256, 0, s>>>(x, x_out, G, H, rows, d, eps);    \
    return hipGetLastError();                                                               \
  }
  JN_RMS(2, 1)   // 128
  JN_RMS(4, 1)   // 256
  JN_RMS(4, 2)   // 512
  JN_RMS(4, 3)   // 768
  JN_RMS(8, 2)   // 1024
  JN_RMS(8, 3)   // 1536
  JN_RMS(8, 4)   // 2048
  JN_RMS(8, 5)   // 2560
  JN_RMS(8, 6)   // 3072
  JN_RMS(8, 8)   // 4096
  // any other multiple of 128 up to 4096: two elements per lane per chunk
#define JN_RMS2(NC) JN_RMS(2, NC)
  JN_RMS2(3) JN_RMS2(5) JN_RMS2(7) JN_RMS2(9) JN_RMS2(10) JN_RMS2(11) JN_RMS2(13) JN_RMS2(14) JN_RMS2(15)
  JN_RMS2(17) JN_RMS2(18) JN_RMS2(19) JN_RMS2(20) JN_RMS2(21) JN_RMS2(22) JN_RMS2(23) JN_RMS2(25)
  JN_RMS2(26) JN_RMS2(27) JN_RMS2(28) JN_RMS2(29) JN_RMS2(30) JN_RMS2(31)
#undef JN_RMS2
#undef JN_RMS
  return hipErrorInvalidValue;
}

hipError_t launch_rmsnorm_bf16in(hipStream_t s, const void* x_bf16, float* x_out, const void* g, void* h,
                                 int32_t rows, int32_t d, float eps) {
  return launch_rms<true>(s, x_bf16, x_out, g, h, rows, d, eps);
}

hipError_t launch_rmsnorm_f32in(hipStream_t s, const float* x, const void* g, void* h, int32_t rows, int32_t d,
                                float eps) {
  return launch_rms<false>(s, x, nullptr, g, h, rows, d, eps);
}

}  // namespace jnx

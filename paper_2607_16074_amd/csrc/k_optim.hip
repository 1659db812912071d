// Per-tenant AdamW step over every tensor of every tenant in one launch.
// Block b updates elements [4096 (b - block_start), +4096) of the tensor whose
// block range holds b; each thread handles 16 elements as four 16-byte
// accesses per operand (the tail of a tensor element by element).  HBM-bound:
// 16 bytes read and 12 written per element (+2 for a bf16 copy).
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

__device__ __forceinline__ void adamw_elem(const AdamwTenant& h, float& p, float g, float& m, float& v) {
  m = h.b1 * m + (1.f - h.b1) * g;
  v = h.b2 * v + (1.f - h.b2) * g * g;
  const float den = sqrtf(v) * h.inv_sqrt_bc2 + h.eps;
  p = p * h.decay - h.step_size * (m / den);
}

__global__ __launch_bounds__(256) void adamw_kernel(const AdamwTensor* __restrict__ ts, int32_t n,
                                                    const AdamwTenant* __restrict__ tens) {
  // the last tensor whose block range starts at or before this block (binary search)
  const int32_t b = blockIdx.x;
  int32_t lo = 0, hi = n - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (ts[mid].block_start <= b) lo = mid; else hi = mid - 1;
  }
  const int32_t i = lo;
  const AdamwTensor T = ts[i];
  const AdamwTenant H = tens[T.tenant];
  const int64_t e0 = (int64_t)(b - T.block_start) * kAdamwBlockElems;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t e = e0 + ((int64_t)k * 256 + threadIdx.x) * 4;
    if (e >= T.numel) break;
    if (e + 4 <= T.numel) {
      float4 p = *reinterpret_cast<const float4*>(T.p + e);
      const float4 g = *reinterpret_cast<const float4*>(T.g + e);
      float4 m = *reinterpret_cast<const float4*>(T.m + e);
      float4 v = *reinterpret_cast<const float4*>(T.v + e);
      adamw_elem(H, p.x, g.x, m.x, v.x);
      adamw_elem(H, p.y, g.y, m.y, v.y);
      adamw_elem(H, p.z, g.z, m.z, v.z);
      adamw_elem(H, p.w, g.w, m.w, v.w);
      *reinterpret_cast<float4*>(T.p + e) = p;
      *reinterpret_cast<float4*>(T.m + e) = m;
      *reinterpret_cast<float4*>(T.v + e) = v;
      if (T.b16) *reinterpret_cast<uint2*>(T.b16 + e) = make_uint2(pack_bf2(p.x, p.y), pack_bf2(p.z, p.w));
    } else {
      for (int64_t j = e; j < T.numel; ++j) {
        float p = T.p[j], m = T.m[j], v = T.v[j];
        adamw_elem(H, p, T.g[j], m, v);
        T.p[j] = p;
        T.m[j] = m;
        T.v[j] = v;
        if (T.b16) T.b16[j] = f2bf(p);
      }
    }
  }
}

int32_t adamw_prepare(AdamwTensor* t, int32_t n) {
  int32_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    t[i].block_start = total;
    total += (int32_t)((t[i].numel + kAdamwBlockElems - 1) / kAdamwBlockElems);
  }
  return total;
}

hipError_t launch_adamw(hipStream_t s, const AdamwTensor* t, int32_t n, const AdamwTenant* ten, int32_t blocks) {
  if (blocks <= 0) return hipSuccess;
  adamw_kernel<<<blocks, 256, 0, s>>>(t, n, ten);
  return hipGetLastError();
}

}  // namespace jnx

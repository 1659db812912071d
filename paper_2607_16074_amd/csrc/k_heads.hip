// Tenant split and tenant-private action heads (fp32):
//   pool       mean of each sample's valid rows of the shared feature, written
//              in tenant order (the split of the shared features by slices)
//   head_gemm  one launch per head layer for all tenants: forward (bias +
//              GELU fused), weight gradient (bias gradient fused) and data
//              gradient (GELU derivative fused); tenant row ranges are read
//              from the device maps, so the host needs no per-tenant counts
//   mse        per-tenant mean squared error and its gradient
// Every reduction runs in a fixed order: results are bitwise reproducible.
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

// ------------------------------------------------------------------ pool ---

template <int CPT>  // column pairs per thread
__global__ __launch_bounds__(256) void pool_kernel(const uint16_t* __restrict__ hidden,
                                                   const int32_t* __restrict__ seqlens,
                                                   const int32_t* __restrict__ cu_seqlens,
                                                   const int32_t* __restrict__ rank, int32_t d,
                                                   float* __restrict__ pooled) {
  const int32_t i = blockIdx.x;
  const int32_t L = seqlens[i];
  const uint32_t* base = reinterpret_cast<const uint32_t*>(hidden + (int64_t)cu_seqlens[i] * d);
  const int32_t pairs = d / 2;
  float acc[CPT][2];
#pragma unroll
  for (int c = 0; c < CPT; ++c) acc[c][0] = acc[c][1] = 0.f;
  for (int32_t j = 0; j < L; ++j) {
    const uint32_t* row = base + (int64_t)j * pairs;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int32_t p = threadIdx.x + c * 256;
      if (p < pairs) {
        uint32_t w = row[p];
        acc[c][0] += __uint_as_float(w << 16);
        acc[c][1] += __uint_as_float(w & 0xffff0000u);
      }
    }
  }
  const float inv = 1.0f / (float)L;
  float* out = pooled + (int64_t)rank[i] * d;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int32_t p = threadIdx.x + c * 256;
    if (p < pairs) *reinterpret_cast<float2*>(out + 2 * p) = make_float2(acc[c][0] * inv, acc[c][1] * inv);
  }
}

hipError_t launch_pool(hipStream_t s, const void* hidden, const int32_t* seqlens, const int32_t* cu_seqlens,
                       const int32_t* rank, int32_t N, int32_t d, float* pooled) {
  auto H = reinterpret_cast<const uint16_t*>(hidden);
  const int cpt = (d / 2 + 255) / 256;
  if (cpt <= 1)
    pool_kernel<1><<<N, 256, 0, s>>>(H, seqlens, cu_seqlens, rank, d, pooled);
  else if (cpt <= 2)
    pool_kernel<2><<<N, 256, 0, s>>>(H, seqlens, cu_seqlens, rank, d, pooled);
  else if (cpt <= 4)
    pool_kernel<4><<<N, 256, 0, s>>>(H, seqlens, cu_seqlens, rank, d, pooled);
  else if (cpt <= 8)
    pool_kernel<8><<<N, 256, 0, s>>>(H, seqlens, cu_seqlens, rank, d, pooled);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ------------------------------------------------------------- head gemm ---

constexpr int HT = 64;   // tile edge
constexpr int HK = 16;   // k step

__global__ __launch_bounds__(256) void head_gemm_kernel(const HeadGemm* __restrict__ descs,
                                                        const HeadTile* __restrict__ tiles,
                                                        const int32_t* __restrict__ tso) {
  __shared__ float As[HK][HT + 4];
  __shared__ float Bs[HK][HT + 4];
  const HeadTile tile = tiles[blockIdx.x];
  const HeadGemm D = descs[tile.desc];
  const int32_t off = tso[D.tenant];
  const int32_t ng = tso[D.tenant + 1] - off;
  const int32_t M = D.M < 0 ? ng : D.M;
  const int32_t N = D.N;
  const int32_t K = D.K < 0 ? ng : D.K;
  const int32_t m0 = tile.tm * HT, n0 = tile.tn * HT;
  if (m0 >= M) return;  // tiles past a tenant's row count (upper-bound grid)
  const float* A = D.A + (int64_t)off * D.bumpA;
  const float* B = D.B + (int64_t)off * D.bumpB;
  const int tid = threadIdx.x;
  const int ty = tid / 16, tx = tid % 16;
  float acc[4][4] = {};
  const bool a_k_fast = D.sak == 1;
  const bool b_k_fast = D.sbk == 1;
  for (int32_t k0 = 0; k0 < K; k0 += HK) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = tid + 256 * q;
      int mm, kk;
      if (a_k_fast) { kk = e % HK; mm = e / HK; } else { mm = e % HT; kk = e / HT; }
      const int32_t m = m0 + mm, k = k0 + kk;
      As[kk][mm] = (m < M && k < K) ? A[(int64_t)m * D.sam + (int64_t)k * D.sak] : 0.f;
      int nn;
      if (b_k_fast) { kk = e % HK; nn = e / HK; } else { nn = e % HT; kk = e / HT; }
      const int32_t n = n0 + nn, k2 = k0 + kk;
      Bs[kk][nn] = (n < N && k2 < K) ? B[(int64_t)k2 * D.sbk + (int64_t)n * D.sbn] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < HK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  float* C = D.C + (int64_t)off * D.bumpC;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int32_t m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int32_t n = n0 + tx * 4 + j;
      if (n >= N) continue;
      float v = acc[i][j];
      const int64_t ci = (int64_t)m * D.ldc + n;
      if (D.bias) v += D.bias[n];
      if (D.Zg) v *= gelu_grad_f((D.Zg + (int64_t)off * D.bumpC)[ci]);
      C[ci] = v;
      if (D.Cact) (D.Cact + (int64_t)off * D.bumpC)[ci] = gelu_f(v);
    }
  }
  if (D.db && tile.tn == 0 && tid < HT) {
    const int32_t m = m0 + tid;
    if (m < M) {
      float sacc = 0.f;
      for (int32_t k = 0; k < K; ++k) sacc += A[(int64_t)m * D.sam + (int64_t)k * D.sak];
      D.db[m] = sacc;
    }
  }
}

hipError_t launch_head_gemm(hipStream_t s, const HeadGemm* descs, const HeadTile* tiles, int32_t n_tiles,
                            const int32_t* tso) {
  head_gemm_kernel<<<n_tiles, 256, 0, s>>>(descs, tiles, tso);
  return hipGetLastError();
}

// ------------------------------------------------------------------- mse ---

__global__ __launch_bounds__(256) void mse_kernel(const LossDesc* __restrict__ descs,
                                                  const int32_t* __restrict__ tso) {
  __shared__ float red[256];
  const LossDesc D = descs[blockIdx.x];
  const int32_t off = tso[D.tenant];
  const int32_t ng = tso[D.tenant + 1] - off;
  const int64_t cnt = (int64_t)ng * D.out;
  const float scale = 2.0f / (float)cnt;
  const float* y = D.y + (int64_t)off * D.ld;
  float* dy = D.dy + (int64_t)off * D.ld;
  float ss = 0.f;
  for (int64_t e = threadIdx.x; e < cnt; e += 256) {
    const int64_t m = e / D.out, n = e % D.out;
    const float yv = y[m * D.ld + n];
    const float diff = yv - D.target[e];
    D.actions[e] = yv;
    dy[m * D.ld + n] = scale * diff;
    ss += diff * diff;
  }
  red[threadIdx.x] = ss;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) D.loss[0] = red[0] / (float)cnt;
}

hipError_t launch_mse(hipStream_t s, const LossDesc* descs, int32_t G, const int32_t* tso) {
  mse_kernel<<<G, 256, 0, s>>>(descs, tso);
  return hipGetLastError();
}

}  // namespace jnx

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

// Block = (sample, 512-column chunk); 256 threads = 4 wavefronts, lane l
// owning columns 8 l .. 8 l + 7 (one 16-byte load covers 1 KB of a row per
// wave).  Wave w sums rows w, w+4, w+8, ... of the sample in that order, four
// loads in flight per lane; the four wave sums are combined as
// (s0 + s1) + (s2 + s3).  The order depends only on the sample's own length,
// so a sample pools to the same bits in any batch.
constexpr int kPoolCols = 512;
constexpr int kPoolWaves = 4;

__global__ __launch_bounds__(256) void pool_kernel(const uint16_t* __restrict__ hidden,
                                                   const int32_t* __restrict__ seqlens,
                                                   const int32_t* __restrict__ cu_seqlens,
                                                   const int32_t* __restrict__ rank, int32_t d,
                                                   float* __restrict__ pooled) {
  __shared__ float red[kPoolWaves][kPoolCols];
  const int32_t chunks = (d + kPoolCols - 1) / kPoolCols;
  const int32_t i = blockIdx.x / chunks;
  const int32_t c0 = (blockIdx.x % chunks) * kPoolCols;
  const int32_t L = seqlens[i];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int32_t col = c0 + lane * 8;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  if (col < d) {
    const uint16_t* base = hidden + (int64_t)cu_seqlens[i] * d + col;
    auto add = [&](const uint4& q) {
      const uint32_t v[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += __uint_as_float(v[e] << 16);
        acc[2 * e + 1] += __uint_as_float(v[e] & 0xffff0000u);
      }
    };
    int32_t j = w;
    for (; j + 3 * kPoolWaves < L; j += 4 * kPoolWaves) {
      uint4 q[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) q[k] = *reinterpret_cast<const uint4*>(base + (int64_t)(j + k * kPoolWaves) * d);
#pragma unroll
      for (int k = 0; k < 4; ++k) add(q[k]);
    }
    for (; j < L; j += kPoolWaves) add(*reinterpret_cast<const uint4*>(base + (int64_t)j * d));
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[w][lane * 8 + e] = acc[e];
  __syncthreads();
  const float inv = 1.0f / (float)L;
  for (int t = threadIdx.x; t < kPoolCols; t += 256) {
    if (c0 + t < d)
      pooled[(int64_t)rank[i] * d + c0 + t] = ((red[0][t] + red[1][t]) + (red[2][t] + red[3][t])) * inv;
  }
}

hipError_t launch_pool(hipStream_t s, const void* hidden, const int32_t* seqlens, const int32_t* cu_seqlens,
                       const int32_t* rank, int32_t N, int32_t d, float* pooled) {
  const int64_t blocks = (int64_t)((d + kPoolCols - 1) / kPoolCols) * N;
  if (d % 8 != 0 || N < 1 || blocks > 0x7fffffff) return hipErrorInvalidValue;
  dim3 grid((unsigned)blocks);
  pool_kernel<<<grid, 256, 0, s>>>(reinterpret_cast<const uint16_t*>(hidden), seqlens, cu_seqlens, rank, d, pooled);
  return hipGetLastError();
}

// ------------------------------------------------------------- head gemm ---

constexpr int HT = 64;   // tile edge
constexpr int HK = 64;   // k step; the next step's operands are loaded into
                         // registers while the current step is computed

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
  constexpr int Q = HT * HK / 256;  // operand elements per thread per step
  float ra[Q], rb[Q];
  auto load = [&](int32_t k0) {
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int e = tid + 256 * q;
      int mm, kk;
      if (a_k_fast) { kk = e % HK; mm = e / HK; } else { mm = e % HT; kk = e / HT; }
      const int32_t m = m0 + mm, k = k0 + kk;
      ra[q] = (m < M && k < K) ? A[(int64_t)m * D.sam + (int64_t)k * D.sak] : 0.f;
      int nn;
      if (b_k_fast) { kk = e % HK; nn = e / HK; } else { nn = e % HT; kk = e / HT; }
      const int32_t n = n0 + nn, k2 = k0 + kk;
      rb[q] = (n < N && k2 < K) ? B[(int64_t)k2 * D.sbk + (int64_t)n * D.sbn] : 0.f;
    }
  };
  load(0);
  for (int32_t k0 = 0; k0 < K; k0 += HK) {
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int e = tid + 256 * q;
      if (a_k_fast) As[e % HK][e / HK] = ra[q]; else As[e / HT][e % HT] = ra[q];
      if (b_k_fast) Bs[e % HK][e / HK] = rb[q]; else Bs[e / HT][e % HT] = rb[q];
    }
    __syncthreads();
    if (k0 + HK < K) load(k0 + HK);
#pragma unroll 8
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

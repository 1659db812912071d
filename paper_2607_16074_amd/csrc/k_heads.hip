// Tenant split and tenant-private action heads (fp32):
//   pool       mean of each sample's valid rows of the shared feature, written
//              in tenant order (the split of the shared features by slices)
//   head_gemm  one launch per head layer for all tenants, fp32 matrix-core
//              tiles: forward (bias + GELU fused), weight gradient (bias
//              gradient fused) and data gradient (GELU derivative fused);
//              tenant row ranges are read from the device maps, so the host
//              needs no per-tenant counts
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

// fp32 matrix-core tiles (v_mfma_f32_16x16x4_f32, the heads' precision): a
// workgroup computes a 32 x 64 tile of C with 4 wavefronts, wave w owning
// rows 16 (w >> 1) .. +15 and columns 32 (w & 1) .. +31 (two 16 x 16 MFMA
// blocks).  32 rows fit the local batch of a tenant in one row tile.  Operands
// go through LDS in K chunks of 32, stored K-major (As[k][m], Bs[k][n], row
// stride padded by one float); the next chunk is loaded into registers while
// the current one is multiplied; steps past the end of a short K (a weight
// gradient's K is the tenant's row count) are skipped.  Measured on the
// 2B-shaped workload's heads: chunks of 128 (4x the loads in flight) left the
// forward launches unchanged and made the weight-gradient launches, whose
// K is 32, 3x slower (more LDS per workgroup, zero-filled chunk work).  MFMA operand layout (16x16x4): lane l holds
// A(m = l & 15, k = l >> 4) and B(k = l >> 4, n = l & 15); the result block
// gives lane l rows 4 (l >> 4) .. +3 of column l & 15.  The K order of every
// output element is fixed (chunks in order, four k per MFMA), and the bias
// gradient of a weight-gradient tile is the row sum of its A operand taken
// from LDS chunk by chunk in k order, so results are bitwise reproducible and
// independent of the other tenants of the launch.
constexpr int HM = 32;   // tile rows
constexpr int HN = 64;   // tile columns
constexpr int HKC = 32;   // K chunk

typedef float f32x4h __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void head_gemm_kernel(const HeadGemm* __restrict__ descs,
                                                        const HeadTile* __restrict__ tiles,
                                                        const int32_t* __restrict__ tso) {
  __shared__ float As[HKC][HM + 1];
  __shared__ float Bs[HKC][HN + 1];
  const HeadTile tile = tiles[blockIdx.x];
  const HeadGemm D = descs[tile.desc];
  const int32_t off = tso[D.tenant];
  const int32_t ng = tso[D.tenant + 1] - off;
  const int32_t M = D.M < 0 ? ng : D.M;
  const int32_t N = D.N;
  const int32_t K = D.K < 0 ? ng : D.K;
  const int32_t m0 = tile.tm * HM, n0 = tile.tn * HN;
  if (m0 >= M) return;  // tiles past a tenant's row count (upper-bound grid)
  // K range of this tile: all of K, or range tk of ksplit (chunk-aligned)
  int32_t kb = 0, ke = K;
  if (D.ksplit > 1) {
    const int32_t kc = ((K + D.ksplit - 1) / D.ksplit + HKC - 1) / HKC * HKC;
    kb = min(K, tile.tk * kc);
    ke = min(K, kb + kc);
  }
  const float* A = D.A + (int64_t)off * D.bumpA;
  const float* B = D.B + (int64_t)off * D.bumpB;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const bool a_k_fast = D.sak == 1;
  const bool b_k_fast = D.sbk == 1;
  const bool want_db = D.db != nullptr && tile.tn == 0;

  constexpr int QA = HM * HKC / 256;  // A elements per thread per chunk (4)
  constexpr int QB = HN * HKC / 256;  // B elements per thread per chunk (8)
  float ra[QA], rb[QB];
  auto load = [&](int32_t k0) {
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int e = tid + 256 * q;
      int mm, kk;
      if (a_k_fast) { kk = e % HKC; mm = e / HKC; } else { mm = e % HM; kk = e / HM; }
      const int32_t m = m0 + mm, k = k0 + kk;
      ra[q] = (m < M && k < ke) ? A[(int64_t)m * D.sam + (int64_t)k * D.sak] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const int e = tid + 256 * q;
      int nn, kk;
      if (b_k_fast) { kk = e % HKC; nn = e / HKC; } else { nn = e % HN; kk = e / HN; }
      const int32_t n = n0 + nn, k = k0 + kk;
      rb[q] = (n < N && k < ke) ? B[(int64_t)k * D.sbk + (int64_t)n * D.sbn] : 0.f;
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int e = tid + 256 * q;
      if (a_k_fast) As[e % HKC][e / HKC] = ra[q]; else As[e / HM][e % HM] = ra[q];
    }
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const int e = tid + 256 * q;
      if (b_k_fast) Bs[e % HKC][e / HKC] = rb[q]; else Bs[e / HN][e % HN] = rb[q];
    }
  };

  f32x4h acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  float dbs = 0.f;  // bias gradient of row m0 + tid (tid < HM), k in order
  const int am = wm * 16 + (lane & 15), kq = lane >> 4;
  const int bn0 = wn * 32 + (lane & 15);
  load(kb);
  for (int32_t k0 = kb; k0 < ke; k0 += HKC) {
    store();
    __syncthreads();
    if (k0 + HKC < ke) load(k0 + HKC);
    const int kend = min(HKC, ke - k0);  // zero-filled beyond the range
#pragma unroll 8
    for (int kk = 0; kk < kend; kk += 4) {
      const float a = As[kk + kq][am];
      acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Bs[kk + kq][bn0], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a, Bs[kk + kq][bn0 + 16], acc1, 0, 0, 0);
    }
    if (want_db && tid < HM) {
#pragma unroll 8
      for (int kk = 0; kk < kend; ++kk) dbs += As[kk][tid];
    }
    __syncthreads();
  }

  if (D.ksplit > 1) {  // raw sum of this K range; the reduce launch finishes the tile
    float* Pt = D.part + tile.tk * D.part_plane + (int64_t)off * D.bumpC;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int32_t n = n0 + wn * 32 + j * 16 + (lane & 15);
      if (n >= N) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int32_t m = m0 + wm * 16 + 4 * (lane >> 4) + e;
        if (m < M) Pt[(int64_t)m * D.ldc + n] = j == 0 ? acc0[e] : acc1[e];
      }
    }
    return;
  }
  float* C = D.C + (int64_t)off * D.bumpC;
  const float* Zg = D.Zg ? D.Zg + (int64_t)off * D.bumpC : nullptr;
  float* Cact = D.Cact ? D.Cact + (int64_t)off * D.bumpC : nullptr;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int32_t n = n0 + wn * 32 + j * 16 + (lane & 15);
    if (n >= N) continue;
    const float bias = D.bias ? D.bias[n] : 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int32_t m = m0 + wm * 16 + 4 * (lane >> 4) + e;
      if (m >= M) continue;
      float v = (j == 0 ? acc0[e] : acc1[e]) + bias;
      const int64_t ci = (int64_t)m * D.ldc + n;
      if (Zg) v *= gelu_grad_f(Zg[ci]);
      C[ci] = v;
      if (Cact) Cact[ci] = gelu_f(v);
    }
  }
  if (want_db && tid < HM && m0 + tid < M) D.db[m0 + tid] = dbs;
}

hipError_t launch_head_gemm(hipStream_t s, const HeadGemm* descs, const HeadTile* tiles, int32_t n_tiles,
                            const int32_t* tso) {
  head_gemm_kernel<<<n_tiles, 256, 0, s>>>(descs, tiles, tso);
  return hipGetLastError();
}

// A long contraction (K >= 512) split into ksplit ranges keeps ~8x more
// workgroups busy: the 2048-wide first layer of the 2B-shaped workload's
// heads is 64 sequential K chunks per tile otherwise, each waiting for its
// loads.  This launch finishes such tiles: thread t owns column n0 + t % 64
// of rows m0 + t / 64 + 4 i; ranges are added in order, then the epilogue.
__global__ __launch_bounds__(256) void head_reduce_kernel(const HeadGemm* __restrict__ descs,
                                                          const HeadTile* __restrict__ tiles,
                                                          const int32_t* __restrict__ tso) {
  const HeadTile tile = tiles[blockIdx.x];
  const HeadGemm D = descs[tile.desc];
  const int32_t off = tso[D.tenant];
  const int32_t ng = tso[D.tenant + 1] - off;
  const int32_t M = D.M < 0 ? ng : D.M;
  const int32_t m0 = tile.tm * HM;
  const int32_t n = tile.tn * HN + (threadIdx.x & 63);
  if (m0 >= M || n >= D.N) return;
  const float* Pt = D.part + (int64_t)off * D.bumpC;
  float* C = D.C + (int64_t)off * D.bumpC;
  const float* Zg = D.Zg ? D.Zg + (int64_t)off * D.bumpC : nullptr;
  float* Cact = D.Cact ? D.Cact + (int64_t)off * D.bumpC : nullptr;
  const float bias = D.bias ? D.bias[n] : 0.f;
#pragma unroll
  for (int i = 0; i < HM / 4; ++i) {
    const int32_t m = m0 + (threadIdx.x >> 6) + 4 * i;
    if (m >= M) break;
    const int64_t ci = (int64_t)m * D.ldc + n;
    float v = Pt[ci];
    for (int32_t t = 1; t < D.ksplit; ++t) v += Pt[t * D.part_plane + ci];
    v += bias;
    if (Zg) v *= gelu_grad_f(Zg[ci]);
    C[ci] = v;
    if (Cact) Cact[ci] = gelu_f(v);
  }
}

hipError_t launch_head_reduce(hipStream_t s, const HeadGemm* descs, const HeadTile* tiles, int32_t n_tiles,
                              const int32_t* tso) {
  head_reduce_kernel<<<n_tiles, 256, 0, s>>>(descs, tiles, tso);
  return hipGetLastError();
}

// ------------------------------------------------------------------- mse ---

// Block (tenant g, part b) of kMseParts takes elements [b c, (b + 1) c) of
// the tenant's row-major [n_g][out] block (c = ceil(count / kMseParts)),
// thread t every 256th of them in order; the block's partial sum of squared
// errors goes to part[g kMseParts + b] (fixed-order tree), and a second
// launch adds a tenant's parts in order.  One block per tenant measured
// ~0.1 ms on the 2B-shaped workload (eight CUs waiting on their loads).
constexpr int kMseParts = 16;

__global__ __launch_bounds__(256) void mse_kernel(const LossDesc* __restrict__ descs,
                                                  const int32_t* __restrict__ tso, float* __restrict__ part) {
  __shared__ float red[256];
  const int32_t g = blockIdx.x / kMseParts, b = blockIdx.x % kMseParts;
  const LossDesc D = descs[g];
  const int32_t off = tso[D.tenant];
  const int32_t ng = tso[D.tenant + 1] - off;
  const int32_t cnt = ng * D.out;
  const float scale = 2.0f / (float)cnt;
  const float* y = D.y + (int64_t)off * D.ld;
  float* dy = D.dy + (int64_t)off * D.ld;
  const int32_t c = (cnt + kMseParts - 1) / kMseParts;
  const int32_t e1 = min(cnt, (b + 1) * c);
  float ss = 0.f;
#pragma unroll 4
  for (int32_t e = b * c + (int32_t)threadIdx.x; e < e1; e += 256) {
    const int32_t m = e / D.out, n = e - m * D.out;
    const float yv = y[(int64_t)m * D.ld + n];
    const float diff = yv - D.target[e];
    D.actions[e] = yv;
    dy[(int64_t)m * D.ld + n] = scale * diff;
    ss = fmaf(diff, diff, ss);
  }
  red[threadIdx.x] = ss;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(64) void mse_final_kernel(const LossDesc* __restrict__ descs,
                                                       const int32_t* __restrict__ tso, const float* __restrict__ part,
                                                       int32_t G) {
  const int32_t g = blockIdx.x * 64 + threadIdx.x;
  if (g >= G) return;
  const LossDesc D = descs[g];
  const int32_t cnt = (tso[D.tenant + 1] - tso[D.tenant]) * D.out;
  float ss = 0.f;
  for (int b = 0; b < kMseParts; ++b) ss += part[g * kMseParts + b];
  D.loss[0] = ss / (float)cnt;
}

hipError_t launch_mse(hipStream_t s, const LossDesc* descs, int32_t G, const int32_t* tso, float* part) {
  mse_kernel<<<G * kMseParts, 256, 0, s>>>(descs, tso, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  mse_final_kernel<<<(G + 63) / 64, 64, 0, s>>>(descs, tso, part, G);
  return hipGetLastError();
}

}  // namespace jnx

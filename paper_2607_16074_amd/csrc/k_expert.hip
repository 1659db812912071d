// Kernels of the tenant-private action expert (forward, loss, weight
// gradients).  GEMMs go through the grouped bf16 GEMM (k_gemm.hip); this file
// holds the rest:
//   copy2d       grouped strided 2-D copy with zero padding and fp32 <-> bf16
//                conversion (operand padding, bf16 rounding points, saves)
//   ksum         ordered sum of the K-range partials of a split weight gradient
//   transpose    grouped bf16 transpose with zero-padded columns (operands of
//                the data- and weight-gradient GEMMs where they cannot be read
//                transposed in place)
//   prefix       tenant-ordered copy of every sample's valid backbone rows
//   rmsnorm      per-tenant-gain RMSNorm forward (fp32 -> bf16) and backward
//                (fp32), gain gradients by fixed-order column sums
//   attention    self- / cross-attention forward and backward on the bf16
//                matrix cores, per (sample, head); a sample's queries never
//                see another sample's keys
//   loss         per-tenant mean squared error and its gradient
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

// ---------------------------------------------------------------- copy2d ---
// Each block covers 2048 elements of one descriptor (row-major over rows x
// cols).  Descriptors whose columns, leading dimensions and source width are
// multiples of 4 move 4 elements per thread step (16-byte fp32 / 8-byte bf16
// accesses); the rest go element by element.

__device__ __forceinline__ void copy4_load(const CopyDesc& D, int64_t r, int64_t c, float (&v)[4]) {
  if (r < D.src_rows && c < D.src_cols) {
    const int64_t si = r * D.src_ld + c;
    if (D.src_bf16) {
      const uint2 u = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(D.src) + si);
      v[0] = __uint_as_float(u.x << 16);
      v[1] = __uint_as_float(u.x & 0xffff0000u);
      v[2] = __uint_as_float(u.y << 16);
      v[3] = __uint_as_float(u.y & 0xffff0000u);
    } else {
      const float4 f = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(D.src) + si);
      v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    }
  } else {
    v[0] = v[1] = v[2] = v[3] = 0.f;
  }
}

__global__ __launch_bounds__(256) void copy2d_kernel(const CopyDesc* __restrict__ descs, int32_t ndesc) {
  int32_t p = 0;
  const int32_t b = blockIdx.x;
  while (p + 1 < ndesc && descs[p + 1].block_start <= b) ++p;
  const CopyDesc D = descs[p];
  const int64_t total = (int64_t)D.rows * D.cols;
  const int64_t base = (int64_t)(b - D.block_start) * 256 * 8;
  const bool vec = D.vec != 0;
  if (vec) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int64_t e = base + ((int64_t)k * 256 + threadIdx.x) * 4;
      if (e >= total) break;
      const int64_t r = e / D.cols, c = e % D.cols;
      float v[4];
      copy4_load(D, r, c, v);
      const int64_t di = r * D.dst_ld + c;
      if (D.dst_bf16)
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(D.dst) + di) =
            make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
      else
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(D.dst) + di) = make_float4(v[0], v[1], v[2], v[3]);
    }
    return;
  }
  for (int k = 0; k < 8; ++k) {
    const int64_t e = base + (int64_t)k * 256 + threadIdx.x;
    if (e >= total) break;
    const int64_t r = e / D.cols, c = e % D.cols;
    float v = 0.f;
    if (r < D.src_rows && c < D.src_cols) {
      const int64_t si = r * D.src_ld + c;
      v = D.src_bf16 ? bf2f(reinterpret_cast<const uint16_t*>(D.src)[si]) : reinterpret_cast<const float*>(D.src)[si];
    }
    const int64_t di = r * D.dst_ld + c;
    if (D.dst_bf16)
      reinterpret_cast<uint16_t*>(D.dst)[di] = f2bf(v);
    else
      reinterpret_cast<float*>(D.dst)[di] = v;
  }
}

int32_t copy2d_prepare(CopyDesc* d, int32_t n) {
  int32_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    const CopyDesc& D = d[i];
    const bool vec = D.cols % 4 == 0 && D.src_ld % 4 == 0 && D.dst_ld % 4 == 0 &&
                     (D.src_cols % 4 == 0 || D.src_cols >= D.cols) &&
                     (D.src == nullptr || reinterpret_cast<uintptr_t>(D.src) % 16 == 0) &&
                     reinterpret_cast<uintptr_t>(D.dst) % 16 == 0;
    d[i].vec = vec ? 1 : 0;
    d[i].block_start = total;
    // vector descriptors: 2048 elements per block as 512 threads-steps of 4
    total += (int32_t)(((int64_t)D.rows * D.cols + 2047) / 2048);
  }
  return total;
}

hipError_t launch_copy2d(hipStream_t s, const CopyDesc* d, int32_t n, int32_t blocks) {
  if (blocks <= 0) return hipSuccess;
  copy2d_kernel<<<blocks, 256, 0, s>>>(d, n);
  return hipGetLastError();
}

// ------------------------------------------------------------------ ksum ---
// One block per 4096 elements of a descriptor (a thread sums 4 x 4 columns).
__global__ __launch_bounds__(256) void ksum_kernel(const KSumDesc* __restrict__ descs, int32_t ndesc) {
  const int32_t b = blockIdx.x;
  int32_t i = 0;
  while (i + 1 < ndesc && descs[i + 1].block_start <= b) ++i;
  const KSumDesc D = descs[i];
  const int64_t base = (int64_t)(b - D.block_start) * 4096;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t e = base + ((int64_t)k * 256 + threadIdx.x) * 4;
    if (e >= D.n) break;
    float4 acc = *reinterpret_cast<const float4*>(D.src + e);
    for (int32_t r = 1; r < D.S; ++r) {
      const float4 v = *reinterpret_cast<const float4*>(D.src + r * D.n + e);
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    *reinterpret_cast<float4*>(D.dst + e) = acc;
  }
}

int32_t ksum_prepare(KSumDesc* d, int32_t n) {
  int32_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (d[i].n <= 0 || d[i].n % 4 != 0 || d[i].S < 1 || reinterpret_cast<uintptr_t>(d[i].src) % 16 != 0 ||
        reinterpret_cast<uintptr_t>(d[i].dst) % 16 != 0)
      return -1;
    d[i].block_start = total;
    total += (int32_t)((d[i].n + 4095) / 4096);
  }
  return total;
}

hipError_t launch_ksum(hipStream_t s, const KSumDesc* d, int32_t n, int32_t blocks) {
  if (blocks <= 0 || n <= 0) return hipSuccess;
  ksum_kernel<<<blocks, 256, 0, s>>>(d, n);
  return hipGetLastError();
}

// ------------------------------------------------------------- transpose ---
// dst[c][r] = src[r][c] for r < rows, 0 for rows <= r < rows_pad; 64x64 tiles.
// Tiles that lie wholly inside the source (and whose leading dimensions are
// multiples of 8) move 16 bytes per thread access; edge tiles go element by
// element.

__global__ __launch_bounds__(256) void transpose_kernel(const TransDesc* __restrict__ descs, int32_t ndesc) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[64][72];
  int32_t p = 0;
  const int32_t b = blockIdx.x;
  while (p + 1 < ndesc && descs[p + 1].block_start <= b) ++p;
  const TransDesc D = descs[p];
  const int32_t tcols = (D.cols + 63) / 64;
  const int32_t local = b - D.block_start;
  const int32_t r0 = (local / tcols) * 64, c0 = (local % tcols) * 64;
  const bool full = r0 + 64 <= D.rows && c0 + 64 <= D.cols && D.src_ld % 8 == 0 && D.dst_ld % 8 == 0 &&
                    r0 + 64 <= D.rows_pad && reinterpret_cast<uintptr_t>(D.src) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(D.dst) % 16 == 0;
  if (full) {
    // load: thread t takes row t >> 2, columns 16*(t & 3) .. +15
    const int rr = threadIdx.x >> 2, cc = 16 * (threadIdx.x & 3);
    const uint4* sp = reinterpret_cast<const uint4*>(D.src + (int64_t)(r0 + rr) * D.src_ld + c0 + cc);
    *reinterpret_cast<uint4*>(&tile[rr][cc]) = sp[0];
    *reinterpret_cast<uint4*>(&tile[rr][cc + 8]) = sp[1];
    __syncthreads();
    // store: thread t writes output row (input column) t >> 2, outputs 16*(t & 3) .. +15
    uint32_t o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = (uint32_t)tile[cc + 2 * i][rr] | ((uint32_t)tile[cc + 2 * i + 1][rr] << 16);
    uint4* dp = reinterpret_cast<uint4*>(D.dst + (int64_t)(c0 + rr) * D.dst_ld + r0 + cc);
    dp[0] = make_uint4(o[0], o[1], o[2], o[3]);
    dp[1] = make_uint4(o[4], o[5], o[6], o[7]);
    return;
  }
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int32_t r = r0 + i, c = c0 + tx;
    uint16_t v = 0;
    if (r < D.rows && c < D.cols) v = D.src[(int64_t)r * D.src_ld + c];
    tile[i][tx] = v;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int32_t c = c0 + i, r = r0 + tx;
    if (c < D.cols && r < D.rows_pad) D.dst[(int64_t)c * D.dst_ld + r] = tile[tx][i];
  }
}

int32_t transpose_prepare(TransDesc* d, int32_t n) {
  int32_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    d[i].block_start = total;
    total += ((d[i].rows_pad + 63) / 64) * ((d[i].cols + 63) / 64);
  }
  return total;
}

hipError_t launch_transpose(hipStream_t s, const TransDesc* d, int32_t n, int32_t blocks) {
  if (blocks <= 0) return hipSuccess;
  transpose_kernel<<<blocks, 256, 0, s>>>(d, n);
  return hipGetLastError();
}

// ----------------------------------------------------------------- prefix ---
// zoff[k] (k in tenant order) = row of the tenant-ordered prefix buffer where
// sample tenant_perm[k]'s valid backbone rows start; zoff[N] = total rows.

__global__ __launch_bounds__(256) void prefix_offsets_kernel(const int32_t* __restrict__ tenant_perm,
                                                            const int32_t* __restrict__ seqlens, int32_t N,
                                                            int32_t* __restrict__ zoff) {
  __shared__ int32_t part[256];
  const int per = (N + 255) / 256;
  const int k0 = threadIdx.x * per;
  int32_t s = 0;
  for (int k = k0; k < min(N, k0 + per); ++k) s += seqlens[tenant_perm[k]];
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t run = 0;
    for (int t = 0; t < 256; ++t) {
      const int32_t v = part[t];
      part[t] = run;
      run += v;
    }
  }
  __syncthreads();
  int32_t run = part[threadIdx.x];
  for (int k = k0; k < min(N, k0 + per); ++k) {
    zoff[k] = run;
    run += seqlens[tenant_perm[k]];
  }
  if (threadIdx.x == 255) zoff[N] = run;
}

// Copy rows of each sample (grid: tenant-order sample x 16-row slab); rows
// past `cap` are dropped so an inconsistent caller row count cannot overflow.
__global__ __launch_bounds__(256) void prefix_gather_kernel(const uint16_t* __restrict__ hidden,
                                                           const int32_t* __restrict__ tenant_perm,
                                                           const int32_t* __restrict__ seqlens,
                                                           const int32_t* __restrict__ cu_seqlens,
                                                           const int32_t* __restrict__ zoff, int32_t d, int64_t cap,
                                                           uint16_t* __restrict__ z) {
  const int32_t k = blockIdx.x;
  const int32_t i = tenant_perm[k];
  const int32_t L = seqlens[i];
  const int32_t j0 = blockIdx.y * 16;
  if (j0 >= L) return;
  const int32_t nr = min(16, L - j0);
  const int32_t chunks = d / 8;
  const uint4* src = reinterpret_cast<const uint4*>(hidden + (int64_t)(cu_seqlens[i] + j0) * d);
  for (int32_t e = threadIdx.x; e < nr * chunks; e += 256) {
    const int64_t row = (int64_t)zoff[k] + j0 + e / chunks;
    if (row >= cap) continue;
    reinterpret_cast<uint4*>(z + row * d)[e % chunks] = src[e];
  }
}

hipError_t launch_prefix(hipStream_t s, const void* hidden, const int32_t* tenant_perm, const int32_t* seqlens,
                         const int32_t* cu_seqlens, int32_t N, int32_t max_seqlen, int32_t d, int64_t cap,
                         int32_t* zoff, void* z) {
  prefix_offsets_kernel<<<1, 256, 0, s>>>(tenant_perm, seqlens, N, zoff);
  dim3 grid(N, (max_seqlen + 15) / 16);
  prefix_gather_kernel<<<grid, 256, 0, s>>>(reinterpret_cast<const uint16_t*>(hidden), tenant_perm, seqlens,
                                            cu_seqlens, zoff, d, cap, reinterpret_cast<uint16_t*>(z));
  return hipGetLastError();
}

// ---------------------------------------------------------------- rmsnorm ---
// Rows are tenant-contiguous: tenant t owns rows [roff[t], roff[t+1]) and its
// gain is gains[t] (bf16 [d]).  One wavefront per row, d = 64 * 4 * NC.

__device__ __forceinline__ int32_t row_tenant(const int32_t* roff, int32_t G, int32_t row) {
  int32_t t = 0;
  while (t + 1 < G && roff[t + 1] <= row) ++t;
  return t;
}

template <int NC>
__global__ __launch_bounds__(256) void xrms_fwd_kernel(const float* __restrict__ x, const uint16_t* const* __restrict__ gains,
                                                      const int32_t* __restrict__ roff, int32_t G, int32_t rows,
                                                      int32_t d, float eps, uint16_t* __restrict__ h) {
  const int lane = threadIdx.x & 63;
  const int32_t row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint16_t* g = gains[row_tenant(roff, G, row)];
  float v[NC][4];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const float4 q = *reinterpret_cast<const float4*>(x + (int64_t)row * d + (c * 64 + lane) * 4);
    v[c][0] = q.x; v[c][1] = q.y; v[c][2] = q.z; v[c][3] = q.w;
#pragma unroll
    for (int k = 0; k < 4; ++k) ss += v[c][k] * v[c][k];
  }
  ss = wave_sum(ss);
  const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int e = (c * 64 + lane) * 4;
    const uint2 gq = *reinterpret_cast<const uint2*>(g + e);
    const float g0 = __uint_as_float(gq.x << 16), g1 = __uint_as_float(gq.x & 0xffff0000u);
    const float g2 = __uint_as_float(gq.y << 16), g3 = __uint_as_float(gq.y & 0xffff0000u);
    *reinterpret_cast<uint2*>(h + (int64_t)row * d + e) =
        make_uint2(pack_bf2(v[c][0] * r * g0, v[c][1] * r * g1), pack_bf2(v[c][2] * r * g2, v[c][3] * r * g3));
  }
}

// dx += r g dh - x r^3 (sum_j g_j dh_j x_j) / d ;  gx[row][j] = dh_j x_j r
template <int NC>
__global__ __launch_bounds__(256) void xrms_bwd_kernel(const float* __restrict__ x, const uint16_t* const* __restrict__ gains,
                                                      const int32_t* __restrict__ roff, int32_t G, int32_t rows,
                                                      int32_t d, float eps, const float* __restrict__ dh,
                                                      float* __restrict__ dx, float* __restrict__ gx) {
  const int lane = threadIdx.x & 63;
  const int32_t row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint16_t* g = gains[row_tenant(roff, G, row)];
  float xv[NC][4], gd[NC][4], dv[NC][4];
  float ss = 0.f, dot = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int e = (c * 64 + lane) * 4;
    const float4 q = *reinterpret_cast<const float4*>(x + (int64_t)row * d + e);
    const float4 t = *reinterpret_cast<const float4*>(dh + (int64_t)row * d + e);
    const uint2 gq = *reinterpret_cast<const uint2*>(g + e);
    const float gg[4] = {__uint_as_float(gq.x << 16), __uint_as_float(gq.x & 0xffff0000u),
                         __uint_as_float(gq.y << 16), __uint_as_float(gq.y & 0xffff0000u)};
    xv[c][0] = q.x; xv[c][1] = q.y; xv[c][2] = q.z; xv[c][3] = q.w;
    dv[c][0] = t.x; dv[c][1] = t.y; dv[c][2] = t.z; dv[c][3] = t.w;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      gd[c][k] = gg[k] * dv[c][k];
      ss += xv[c][k] * xv[c][k];
      dot += gd[c][k] * xv[c][k];
    }
  }
  ss = wave_sum(ss);
  dot = wave_sum(dot);
  const float r = rsqrtf(ss / (float)d + eps);
  const float coef = r * r * r * dot / (float)d;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int e = (c * 64 + lane) * 4;
    float4* px = reinterpret_cast<float4*>(dx + (int64_t)row * d + e);
    float4 o = *px;
    o.x += r * gd[c][0] - xv[c][0] * coef;
    o.y += r * gd[c][1] - xv[c][1] * coef;
    o.z += r * gd[c][2] - xv[c][2] * coef;
    o.w += r * gd[c][3] - xv[c][3] * coef;
    *px = o;
    *reinterpret_cast<float4*>(gx + (int64_t)row * d + e) =
        make_float4(dv[c][0] * xv[c][0] * r, dv[c][1] * xv[c][1] * r, dv[c][2] * xv[c][2] * r, dv[c][3] * xv[c][3] * r);
  }
}

// dg_t[j] = sum over tenant t's rows of gx[row][j], in two fixed-order stages:
// partial sums over kColSeg row segments, then the sum of the segments.
constexpr int kColSeg = 16;

__global__ __launch_bounds__(256) void colsum_part_kernel(const float* __restrict__ gx, const int32_t* __restrict__ roff,
                                                          float* __restrict__ part, int32_t d) {
  const int32_t t = blockIdx.x, seg = blockIdx.z;
  const int32_t j = blockIdx.y * 256 + threadIdx.x;
  if (j >= d) return;
  const int32_t r0 = roff[t], n = roff[t + 1] - r0;
  const int32_t per = (n + kColSeg - 1) / kColSeg;
  const int32_t a = r0 + min(n, seg * per), b = r0 + min(n, (seg + 1) * per);
  float s = 0.f;
  for (int32_t r = a; r < b; ++r) s += gx[(int64_t)r * d + j];
  part[((int64_t)t * kColSeg + seg) * d + j] = s;
}

__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ part, float* const* __restrict__ out,
                                                           int32_t d) {
  const int32_t t = blockIdx.x;
  const int32_t j = blockIdx.y * 256 + threadIdx.x;
  if (j >= d) return;
  float s = 0.f;
#pragma unroll
  for (int seg = 0; seg < kColSeg; ++seg) s += part[((int64_t)t * kColSeg + seg) * d + j];
  out[t][j] = s;
}

hipError_t launch_xrms_fwd(hipStream_t s, const float* x, const void* const* gains, const int32_t* roff, int32_t G,
                           int32_t rows, int32_t d, float eps, void* h) {
  dim3 grid((rows + 3) / 4);
  auto gp = reinterpret_cast<const uint16_t* const*>(gains);
  auto hp = reinterpret_cast<uint16_t*>(h);
  switch (d) {
    case 256: xrms_fwd_kernel<1><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, hp); break;
    case 512: xrms_fwd_kernel<2><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, hp); break;
    case 1024: xrms_fwd_kernel<4><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, hp); break;
    case 2048: xrms_fwd_kernel<8><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, hp); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_xrms_bwd(hipStream_t s, const float* x, const void* const* gains, const int32_t* roff, int32_t G,
                           int32_t rows, int32_t d, float eps, const float* dh, float* dx, float* gx, float* part,
                           float* const* dg) {
  dim3 grid((rows + 3) / 4);
  auto gp = reinterpret_cast<const uint16_t* const*>(gains);
  switch (d) {
    case 256: xrms_bwd_kernel<1><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, dh, dx, gx); break;
    case 512: xrms_bwd_kernel<2><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, dh, dx, gx); break;
    case 1024: xrms_bwd_kernel<4><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, dh, dx, gx); break;
    case 2048: xrms_bwd_kernel<8><<<grid, 256, 0, s>>>(x, gp, roff, G, rows, d, eps, dh, dx, gx); break;
    default: return hipErrorInvalidValue;
  }
  dim3 g2(G, (d + 255) / 256, kColSeg), g3(G, (d + 255) / 256);
  colsum_part_kernel<<<g2, 256, 0, s>>>(gx, roff, part, d);
  colsum_final_kernel<<<g3, 256, 0, s>>>(part, dg, d);
  return hipGetLastError();
}

// -------------------------------------------------------------- attention ---
// Self- / cross-attention of the expert on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation and softmax statistics).
// Queries: rows q_row0 + 0..Lq-1 of Q (Lq <= 64: four 16-row blocks, one per
// wave); keys / values: rows kv_row0 .. + Lk - 1 of K / V.  Self attention:
// the sample's own action rows; cross attention: the sample's rows of the
// tenant-ordered prefix (zoff), so a query never sees another sample's keys.
// Q, K, V are bf16 (their projections store them so); the probabilities are
// rounded to bf16 before they meet V, and in the backward the incoming output
// gradient, the recomputed probabilities and the score gradient before they
// meet their products.  The softmax runs in the log2 domain: lse holds
// m + log2(l) of the scaled scores.
//
// MFMA layouts (16x16x32): A (16 x 32) -- lane l supplies row l & 15,
// k-slots 8 (l >> 4) .. +7; B (32 x 16) -- column l & 15, the same k-slots;
// D -- lane l holds rows 4 (l >> 4) .. +3 of column l & 15.  Scores are
// formed transposed where the lane should own a query (S^T = K Q^T: lane =
// query, registers = 4 keys of each 16-key block), so a query's row
// statistics need only exchanges with lanes l ^ 16 and l ^ 32.  Products
// whose contraction runs over the rows of a row-major LDS tile (V^T P^T,
// K^T dS^T, dO^T P, Q^T dS) read their A operand with ds_read_b64_tr_b16:
// lane (g, j) of 16-lane group g addresses row 32 c + 4 g + j / 4 (and +16)
// at column 16 t + 4 (j % 4) and receives column 16 t + j of rows
// 32 c + 4 g .. +3 and 32 c + 16 + 4 g .. +3, so k-slot s of lane (g, j)
// is row 32 c + 4 g + (s & 3) + 16 (s >> 2) -- the order in which the lane
// already holds the matching B values (register e of blocks 2c and 2c+1).
// Every LDS tile row is a permutation of its 16-byte chunks (chunk c at
// c ^ swz(row)) so that both the 16-byte fragment reads and the transposed
// reads touch each bank once per 256 bytes.

typedef __bf16 xbf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 xbf16x4 __attribute__((ext_vector_type(4)));
typedef float xf32x4 __attribute__((ext_vector_type(4)));

#define XA_GPTR(p) ((__attribute__((address_space(1))) void*)(p))
#define XA_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

template <int HD>
__device__ __forceinline__ int xa_swz(int r) {
  if constexpr (HD == 64) {
    const int x = (r >> 1) & 7;  // 2 rows per 256-byte bank row: bit-reversed row pair
    return ((x & 1) << 2) | (x & 2) | (x >> 2);
  } else {
    // one row per bank row; rows r and r ^ 8 share a bank slot pair, so the
    // transposed reads of 16-lane groups q and q ^ 1, which the hardware
    // serves together, stay on 16 distinct slots (a fragment read's 16 rows
    // as well).  The backbone attention's head-width-256 rule, which also
    // avoids the q / q ^ 2 pairing, measured 1% slower here.
    return ((r & 7) << 1) | ((r >> 3) & 1);
  }
}

// 16-byte fragment: logical chunk c (8 elements) of row r of an LDS tile
template <int HD>
__device__ __forceinline__ xbf16x8 xa_frag(const uint16_t* t, int r, int c) {
  return *reinterpret_cast<const xbf16x8*>(t + r * HD + ((c ^ xa_swz<HD>(r)) * 8));
}

// transposed A operand: rows 32 c + 4 g + {0..3, 16..19} of column 16 t + j
// (lane (g, j)); swz = xa_swz(4 g + j / 4), shared by those rows
template <int HD>
__device__ __forceinline__ xbf16x8 xa_tr(const uint16_t* t, int c, int ct, int quad, int j16, int swz) {
  const int col = ct * 16 + 4 * (j16 & 3);
  const int pos = (((col >> 3) ^ swz) * 8) + (col & 7);
  const int r0 = c * 32 + 4 * quad + (j16 >> 2);
  const xbf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) xbf16x4*)(t + r0 * HD + pos));
  const xbf16x4 hi =
      __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) xbf16x4*)(t + (r0 + 16) * HD + pos));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

__device__ __forceinline__ xf32x4 xa_mfma(xbf16x8 a, xbf16x8 b, xf32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 8 fp32 values -> bf16 operand (round to nearest even)
__device__ __forceinline__ xbf16x8 xa_pack8(const float* v) {
  xbf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)v[e];
  return r;
}

__device__ __forceinline__ void attn_rows(const AttnArgs& A, int32_t k, int32_t& q0, int32_t& Lq, int64_t& kv0,
                                          int32_t& Lk) {
  q0 = k * A.Lq;
  Lq = A.Lq;
  if (A.zoff) {
    kv0 = A.zoff[k];
    const int64_t kv1 = min((int64_t)A.zoff[k + 1], A.kv_cap);
    Lk = (int32_t)max((int64_t)0, kv1 - kv0);
  } else {
    kv0 = (int64_t)k * A.Lq;
    Lk = A.Lq;
  }
}

// K and V tiles of 64 keys ([64][HD] bf16 each, swizzled), double buffered,
// moved by direct DMA: 1 KB instructions, lane -> (row RPI v + lane / CPR,
// chunk (lane % CPR) ^ swz(row)); rows past the sample repeat its last row.
template <int HD>
struct XaTiles {
  static constexpr int CPR = HD / 8, RPI = 512 / HD, TILE = 64 * HD, NDMA = 2 * TILE / 512, DPW = NDMA / 4;
  __device__ __forceinline__ static void issue(uint16_t* stage, const uint16_t* Kb, const uint16_t* Vb, int64_t ld,
                                               int64_t kv0, int32_t Lk, int32_t j0, int wave, int lane) {
#pragma unroll
    for (int k = 0; k < DPW; ++k) {
      const int u = wave * DPW + k;
      const bool isv = u >= NDMA / 2;
      const int v = isv ? u - NDMA / 2 : u;
      const int r = v * RPI + lane / CPR;
      const int c = (lane % CPR) ^ xa_swz<HD>(r);
      const int64_t key = kv0 + min(j0 + r, Lk - 1);
      const uint16_t* src = (isv ? Vb : Kb) + key * ld + c * 8;
      __builtin_amdgcn_global_load_lds(XA_GPTR(src), XA_LPTR(stage + u * 512), 16, 0, 0);
    }
  }
};

// Forward: one workgroup per (sample, head), wave w = queries 16 w ..;
// O = softmax(Q K^T scale) V in fp32 (and a bf16 copy), lse per query.
template <int HD>
__global__ __launch_bounds__(256, 2) void xattn_fwd_kernel(AttnArgs A) {
  using T = XaTiles<HD>;
  constexpr int NQC = HD / 32, NOT = HD / 16;
  __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2 * T::TILE];
  const int k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  if (Lk <= 0) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j16 = lane & 15, quad = lane >> 4;
  const int qi = wave * 16 + j16;  // this lane's query
  const int64_t qrow = q0 + min(qi, Lq - 1);
  const float sl2 = A.scale * 1.4426950408889634f;
  xbf16x8 qf[NQC];
#pragma unroll
  for (int c = 0; c < NQC; ++c) qf[c] = *reinterpret_cast<const xbf16x8*>(A.Q + qrow * A.ldq + h * HD + c * 32 + quad * 8);
  const uint16_t* Kb = A.K + A.kcol + h * HD;
  const uint16_t* Vb = A.V + A.vcol + h * HD;
  const int vswz = xa_swz<HD>(4 * quad + (j16 >> 2));

  xf32x4 o[NOT];
#pragma unroll
  for (int t = 0; t < NOT; ++t) o[t] = xf32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  const int32_t ntiles = (Lk + 63) / 64;
  T::issue(&lds[0][0], Kb, Vb, A.ldkv, kv0, Lk, 0, wave, lane);
  for (int32_t jt = 0; jt < ntiles; ++jt) {
    const int32_t j0 = jt * 64;
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();  // tile jt landed; tile jt-1's buffer is free
    T::issue(&lds[(jt + 1) & 1][0], Kb, Vb, A.ldkv, kv0, Lk, min(j0 + 64, (ntiles - 1) * 64), wave, lane);
    const uint16_t* Ks = &lds[jt & 1][0];
    const uint16_t* Vs = Ks + T::TILE;
    xf32x4 s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) s[kb] = xf32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NQC; ++c)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) s[kb] = xa_mfma(xa_frag<HD>(Ks, kb * 16 + j16, 4 * c + quad), qf[c], s[kb]);
    if (j0 + 64 > Lk) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (j0 + kb * 16 + quad * 4 + e >= Lk) s[kb][e] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, s[kb][e]);
    const float m_new = fmaxf(m, max_xor32(max_xor16(mx)) * sl2);
    const float alpha = exp2f(m - m_new);
    l *= alpha;
#pragma unroll
    for (int t = 0; t < NOT; ++t) o[t] *= alpha;
    m = m_new;
    float lsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[kb][e] = exp2f(fmaf(s[kb][e], sl2, -m));
        lsum += s[kb][e];
      }
    l += sum_xor32(sum_xor16(lsum));
    xbf16x8 pf[2];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pf[c][e] = (__bf16)s[2 * c][e];
        pf[c][4 + e] = (__bf16)s[2 * c + 1][e];
      }
#pragma unroll
    for (int t = 0; t < NOT; ++t)
#pragma unroll
      for (int c = 0; c < 2; ++c) o[t] = xa_mfma(xa_tr<HD>(Vs, c, t, quad, j16, vswz), pf[c], o[t]);
  }
  __builtin_amdgcn_s_waitcnt(0);  // the repeated last tile's DMA lands before the LDS is released
  if (qi >= Lq) return;
  const float inv = 1.f / l;
  const int64_t row = q0 + qi;
  float* orow = A.O + row * A.ldo + h * HD + quad * 4;
  uint16_t* brow = A.Ob + row * A.ldo + h * HD + quad * 4;
#pragma unroll
  for (int t = 0; t < NOT; ++t) {
    const float v0 = o[t][0] * inv, v1 = o[t][1] * inv, v2 = o[t][2] * inv, v3 = o[t][3] * inv;
    *reinterpret_cast<float4*>(orow + t * 16) = make_float4(v0, v1, v2, v3);
    *reinterpret_cast<uint2*>(brow + t * 16) = make_uint2(pack_bf2(v0, v1), pack_bf2(v2, v3));
  }
  if (quad == 0) A.lse[row * A.nheads + h] = m + __log2f(l);
}

// Backward, query side: dQ = scale dS K, dS = P (dP - D), P from the saved
// lse, dP^T = V dO^T, D = sum(dO * O) per query (also written to dsum for
// the key side).  Same layout as the forward.
template <int HD>
__global__ __launch_bounds__(256, 2) void xattn_bwd_dq_kernel(AttnArgs A) {
  using T = XaTiles<HD>;
  constexpr int NQC = HD / 32, NOT = HD / 16;
  __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2 * T::TILE];
  const int k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  if (Lk <= 0) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j16 = lane & 15, quad = lane >> 4;
  const int qi = wave * 16 + j16;
  const int64_t qrow = q0 + min(qi, Lq - 1);
  const float sl2 = A.scale * 1.4426950408889634f;
  xbf16x8 qf[NQC], df[NQC];
  float Dq = 0.f;
  {
    const float* drow = A.dO + qrow * A.ldo + h * HD;
    const float* orow = A.O + qrow * A.ldo + h * HD;
#pragma unroll
    for (int c = 0; c < NQC; ++c) {
      qf[c] = *reinterpret_cast<const xbf16x8*>(A.Q + qrow * A.ldq + h * HD + c * 32 + quad * 8);
      float v[8];
      const float4 d0 = *reinterpret_cast<const float4*>(drow + c * 32 + quad * 8);
      const float4 d1 = *reinterpret_cast<const float4*>(drow + c * 32 + quad * 8 + 4);
      const float4 o0 = *reinterpret_cast<const float4*>(orow + c * 32 + quad * 8);
      const float4 o1 = *reinterpret_cast<const float4*>(orow + c * 32 + quad * 8 + 4);
      v[0] = d0.x; v[1] = d0.y; v[2] = d0.z; v[3] = d0.w; v[4] = d1.x; v[5] = d1.y; v[6] = d1.z; v[7] = d1.w;
      df[c] = xa_pack8(v);
      Dq = fmaf(d0.x, o0.x, Dq); Dq = fmaf(d0.y, o0.y, Dq); Dq = fmaf(d0.z, o0.z, Dq); Dq = fmaf(d0.w, o0.w, Dq);
      Dq = fmaf(d1.x, o1.x, Dq); Dq = fmaf(d1.y, o1.y, Dq); Dq = fmaf(d1.z, o1.z, Dq); Dq = fmaf(d1.w, o1.w, Dq);
    }
    Dq = sum_xor32(sum_xor16(Dq));
  }
  const float lse = A.lse[qrow * A.nheads + h];
  if (qi < Lq && quad == 0) A.dsum[(q0 + qi) * A.nheads + h] = Dq;
  const uint16_t* Kb = A.K + A.kcol + h * HD;
  const uint16_t* Vb = A.V + A.vcol + h * HD;
  const int tswz = xa_swz<HD>(4 * quad + (j16 >> 2));

  xf32x4 dq[NOT];
#pragma unroll
  for (int t = 0; t < NOT; ++t) dq[t] = xf32x4{0.f, 0.f, 0.f, 0.f};
  const int32_t ntiles = (Lk + 63) / 64;
  T::issue(&lds[0][0], Kb, Vb, A.ldkv, kv0, Lk, 0, wave, lane);
  for (int32_t jt = 0; jt < ntiles; ++jt) {
    const int32_t j0 = jt * 64;
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    T::issue(&lds[(jt + 1) & 1][0], Kb, Vb, A.ldkv, kv0, Lk, min(j0 + 64, (ntiles - 1) * 64), wave, lane);
    const uint16_t* Ks = &lds[jt & 1][0];
    const uint16_t* Vs = Ks + T::TILE;
    xf32x4 s[4], dp[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) s[kb] = dp[kb] = xf32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NQC; ++c)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        s[kb] = xa_mfma(xa_frag<HD>(Ks, kb * 16 + j16, 4 * c + quad), qf[c], s[kb]);
        dp[kb] = xa_mfma(xa_frag<HD>(Vs, kb * 16 + j16, 4 * c + quad), df[c], dp[kb]);
      }
    xbf16x8 dsf[2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool live = j0 + kb * 16 + quad * 4 + e < Lk;
        const float pv = live ? exp2f(fmaf(s[kb][e], sl2, -lse)) : 0.f;
        dsf[kb >> 1][(kb & 1) * 4 + e] = (__bf16)(pv * (dp[kb][e] - Dq));
      }
#pragma unroll
    for (int t = 0; t < NOT; ++t)
#pragma unroll
      for (int c = 0; c < 2; ++c) dq[t] = xa_mfma(xa_tr<HD>(Ks, c, t, quad, j16, tswz), dsf[c], dq[t]);
  }
  __builtin_amdgcn_s_waitcnt(0);
  if (qi >= Lq) return;
  uint16_t* out = A.dQ + (q0 + qi) * A.lddq + h * HD + quad * 4;
#pragma unroll
  for (int t = 0; t < NOT; ++t)
    *reinterpret_cast<uint2*>(out + t * 16) = make_uint2(pack_bf2(dq[t][0] * A.scale, dq[t][1] * A.scale),
                                                         pack_bf2(dq[t][2] * A.scale, dq[t][3] * A.scale));
}

// Backward, key side: one workgroup per (sample, head, 64-key tile), wave w =
// keys 16 w ..; the sample's queries (<= 64, zero rows past Lq) and its
// bf16-rounded output gradients sit in LDS.  Scores untransposed, S = Q K^T
// (lane = key, registers = 4 queries of each 16-query block), so P and dS
// are already the B operands of dV^T = dO^T P and dK^T = Q^T dS.
template <int HD>
__global__ __launch_bounds__(256, 2) void xattn_bwd_dkv_kernel(AttnArgs A) {
  constexpr int NQC = HD / 32, NOT = HD / 16, CPR = HD / 8;
  __shared__ __attribute__((aligned(1024))) uint16_t qt[64 * HD];
  __shared__ __attribute__((aligned(1024))) uint16_t dt[64 * HD];
  __shared__ float lse_s[64], d_s[64];
  const int k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  const int32_t j0 = blockIdx.z * 64;
  if (j0 >= Lk) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j16 = lane & 15, quad = lane >> 4;
  const float sl2 = A.scale * 1.4426950408889634f;
  // stage Q and bf16(dO): 64 rows x CPR chunks of 8 elements
  for (int e = tid; e < 64 * CPR; e += 256) {
    const int r = e / CPR, c = e % CPR;
    const int pos = r * HD + ((c ^ xa_swz<HD>(r)) * 8);
    uint4 qv = make_uint4(0, 0, 0, 0), dv = make_uint4(0, 0, 0, 0);
    if (r < Lq) {
      const int64_t row = q0 + r;
      qv = *reinterpret_cast<const uint4*>(A.Q + row * A.ldq + h * HD + c * 8);
      const float4 a = *reinterpret_cast<const float4*>(A.dO + row * A.ldo + h * HD + c * 8);
      const float4 b = *reinterpret_cast<const float4*>(A.dO + row * A.ldo + h * HD + c * 8 + 4);
      dv = make_uint4(pack_bf2(a.x, a.y), pack_bf2(a.z, a.w), pack_bf2(b.x, b.y), pack_bf2(b.z, b.w));
    }
    *reinterpret_cast<uint4*>(qt + pos) = qv;
    *reinterpret_cast<uint4*>(dt + pos) = dv;
  }
  if (tid < 64) {
    const bool live = tid < Lq;
    lse_s[tid] = live ? A.lse[(q0 + tid) * A.nheads + h] : INFINITY;  // P = 0 past Lq
    d_s[tid] = live ? A.dsum[(q0 + tid) * A.nheads + h] : 0.f;
  }
  __syncthreads();

  const int32_t key = j0 + wave * 16 + j16;  // this lane's key
  const int64_t krow = kv0 + min(key, Lk - 1);
  xbf16x8 kf[NQC], vf[NQC];
#pragma unroll
  for (int c = 0; c < NQC; ++c) {
    kf[c] = *reinterpret_cast<const xbf16x8*>(A.K + krow * A.ldkv + A.kcol + h * HD + c * 32 + quad * 8);
    vf[c] = *reinterpret_cast<const xbf16x8*>(A.V + krow * A.ldkv + A.vcol + h * HD + c * 32 + quad * 8);
  }
  // S[q][key] and dP[q][key] for the four 16-query blocks
  xf32x4 s[4], dp[4];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) s[qb] = dp[qb] = xf32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NQC; ++c)
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      s[qb] = xa_mfma(xa_frag<HD>(qt, qb * 16 + j16, 4 * c + quad), kf[c], s[qb]);
      dp[qb] = xa_mfma(xa_frag<HD>(dt, qb * 16 + j16, 4 * c + quad), vf[c], dp[qb]);
    }
  // P and dS as B operands: k-slot s of chunk c is query 32 c + 4 quad + (s & 3) + 16 (s >> 2)
  xbf16x8 pb[2], db[2];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int q = qb * 16 + quad * 4 + e;
      const float pv = exp2f(fmaf(s[qb][e], sl2, -lse_s[q]));
      pb[qb >> 1][(qb & 1) * 4 + e] = (__bf16)pv;
      db[qb >> 1][(qb & 1) * 4 + e] = (__bf16)(pv * (dp[qb][e] - d_s[q]));
    }
  const int tswz = xa_swz<HD>(4 * quad + (j16 >> 2));
  xf32x4 dv[NOT], dk[NOT];
#pragma unroll
  for (int t = 0; t < NOT; ++t) {
    dv[t] = dk[t] = xf32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      dv[t] = xa_mfma(xa_tr<HD>(dt, c, t, quad, j16, tswz), pb[c], dv[t]);
      dk[t] = xa_mfma(xa_tr<HD>(qt, c, t, quad, j16, tswz), db[c], dk[t]);
    }
  }
  if (key >= Lk) return;
  // lane holds dV^T / dK^T rows (head dims) 16 t + 4 quad .. +3 of its key
  uint16_t* vrow = A.dV + (kv0 + key) * A.lddkv + A.dvcol + h * HD + quad * 4;
  uint16_t* krw = A.dK + (kv0 + key) * A.lddkv + A.dkcol + h * HD + quad * 4;
#pragma unroll
  for (int t = 0; t < NOT; ++t) {
    *reinterpret_cast<uint2*>(vrow + t * 16) = make_uint2(pack_bf2(dv[t][0], dv[t][1]), pack_bf2(dv[t][2], dv[t][3]));
    *reinterpret_cast<uint2*>(krw + t * 16) =
        make_uint2(pack_bf2(dk[t][0] * A.scale, dk[t][1] * A.scale), pack_bf2(dk[t][2] * A.scale, dk[t][3] * A.scale));
  }
}

hipError_t launch_xattn(hipStream_t s, const AttnArgs& A, int32_t nsamples, bool backward) {
  if (A.Lq > 64 || A.Lq < 1 || A.max_lk < 1) return hipErrorInvalidValue;
  const dim3 grid(nsamples, A.nheads), gk(nsamples, A.nheads, (A.max_lk + 63) / 64);
  switch (A.hd) {
    case 64:
      if (backward) {
        xattn_bwd_dq_kernel<64><<<grid, 256, 0, s>>>(A);
        xattn_bwd_dkv_kernel<64><<<gk, 256, 0, s>>>(A);
      } else {
        xattn_fwd_kernel<64><<<grid, 256, 0, s>>>(A);
      }
      break;
    case 128:
      if (backward) {
        xattn_bwd_dq_kernel<128><<<grid, 256, 0, s>>>(A);
        xattn_bwd_dkv_kernel<128><<<gk, 256, 0, s>>>(A);
      } else {
        xattn_fwd_kernel<128><<<grid, 256, 0, s>>>(A);
      }
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------- loss ---
// Tenant t: rows [roff[t], roff[t+1]) of pred_pad [rows][ldp]; first `a`
// columns valid.  pred / target: the caller's [rows_t][a] buffers.

__global__ __launch_bounds__(256) void xloss_kernel(const XLossDesc* __restrict__ descs, const int32_t* __restrict__ roff,
                                                   const float* __restrict__ pred_pad, int32_t ldp,
                                                   float* __restrict__ dpred_pad) {
  __shared__ float red[256];
  const int32_t t = blockIdx.x;
  const XLossDesc D = descs[t];
  const int32_t r0 = roff[t], rows = roff[t + 1] - r0;
  const int64_t cnt = (int64_t)rows * D.a;
  const float scale = 2.0f / (float)cnt;
  float ss = 0.f;
  for (int64_t e = threadIdx.x; e < (int64_t)rows * ldp; e += 256) {
    const int64_t rr = e / ldp, c = e % ldp;
    const int64_t gi = (int64_t)(r0 + rr) * ldp + c;
    float g = 0.f;
    if (c < D.a) {
      const float y = pred_pad[gi];
      const float diff = y - D.target[rr * D.a + c];
      D.pred[rr * D.a + c] = y;
      g = scale * diff;
      ss += diff * diff;
    }
    dpred_pad[gi] = g;
  }
  red[threadIdx.x] = ss;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) D.loss[0] = red[0] / (float)cnt;
}

hipError_t launch_xloss(hipStream_t s, const XLossDesc* d, const int32_t* roff, int32_t G, const float* pred_pad,
                        int32_t ldp, float* dpred_pad) {
  xloss_kernel<<<G, 256, 0, s>>>(d, roff, pred_pad, ldp, dpred_pad);
  return hipGetLastError();
}


// ------------------------------------------------------------- flow prep ---
// One block per expert row: the tenant is found from the descriptors' row
// ranges, the sample from row / chunk.  Columns [0, a): bf16(t e + (1-t) A)
// and vel = e - A; [a, kap): 0; [kap, kap + d_time): bf16 of sin / cos of
// 1000 t w_j with w_j = 10000^(-j / (d_time/2)) (fp32 math).
__global__ __launch_bounds__(256) void flow_prep_kernel(const FlowDesc* __restrict__ d, int32_t G, int32_t chunk,
                                                        int32_t kap, int32_t d_time, uint16_t* __restrict__ in_rows,
                                                        int32_t ld) {
  const int64_t row = blockIdx.x;
  int32_t g = 0;
  while (g + 1 < G && row >= d[g + 1].roff) ++g;
  const FlowDesc D = d[g];
  const int64_t r = row - D.roff;
  if (r < 0 || r >= D.rows) return;
  const float tau = D.t[r / chunk];
  uint16_t* out = in_rows + row * ld;
  const int32_t half = d_time >> 1;
  const float l2 = 13.287712379549449f;  // log2(10000)
  for (int32_t c = threadIdx.x; c < kap + d_time; c += 256) {
    float v = 0.f;
    if (c < D.a) {
      const float e = D.noise[r * D.a + c], A = D.act[r * D.a + c];
      v = tau * e + (1.0f - tau) * A;
      D.vel[r * D.a + c] = e - A;
    } else if (c >= kap) {
      const int32_t j = c - kap;
      const int32_t jj = j < half ? j : j - half;
      const float ang = 1000.0f * tau * exp2f(-(float)jj / (float)half * l2);
      v = j < half ? sinf(ang) : cosf(ang);
    }
    out[c] = f2bf(v);
  }
}

hipError_t launch_flow_prep(hipStream_t s, const FlowDesc* d, int32_t G, int64_t total_rows, int32_t chunk,
                            int32_t kap, int32_t d_time, uint16_t* in_rows, int32_t ld) {
  if (G < 1 || total_rows < 1 || total_rows > 0x7fffffff || chunk < 1 || ld < kap + d_time) return hipErrorInvalidValue;
  flow_prep_kernel<<<(unsigned)total_rows, 256, 0, s>>>(d, G, chunk, kap, d_time, in_rows, ld);
  return hipGetLastError();
}

}  // namespace jnx

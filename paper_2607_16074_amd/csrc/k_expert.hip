// Kernels of the tenant-private action expert (forward, loss, weight
// gradients).  GEMMs go through the grouped bf16 GEMM (k_gemm.hip); this file
// holds the rest:
//   copy2d       grouped strided 2-D copy with zero padding and fp32 <-> bf16
//                conversion (operand padding, bf16 rounding points, saves)
//   transpose    grouped bf16 transpose with zero-padded columns (operands of
//                the data- and weight-gradient GEMMs)
//   prefix       tenant-ordered copy of every sample's valid backbone rows
//   rmsnorm      per-tenant-gain RMSNorm forward (fp32 -> bf16) and backward
//                (fp32), gain gradients by fixed-order column sums
//   attention    fp32 self- / cross-attention forward and backward on the
//                fp32 matrix cores, per (sample, head); a sample's queries
//                never see another sample's keys
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
// fp32 attention on the fp32 matrix cores (v_mfma_f32_32x32x2_f32).  Queries:
// rows q_row0 + 0..Lq-1 of Q (Lq <= 64, two groups of 32); keys / values: rows
// kv_row0 .. + Lk - 1 of K / V.  Self attention: the sample's own action rows;
// cross attention: the sample's rows of the tenant-ordered prefix (zoff), so a
// query never sees another sample's keys.
//
// MFMA lane layout (32x32x2): lane l supplies A[l & 31][l >> 5] and
// B[l >> 5][l & 31]; accumulator r of lane l is C[mrow(r, l)][l & 31].  Scores
// are computed transposed, S^T = K Q^T, so each lane owns one query column and
// softmax statistics need one exchange with lane l ^ 32.  In P V the k index of
// step t pairs key kfor(t, half) with the half's lane, which is exactly the key
// whose score that lane holds in register t: P never leaves registers.

typedef float f32x16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int mrow(int r, int half) { return 8 * (r >> 2) + 4 * half + (r & 3); }

__device__ __forceinline__ f32x16v mfma32(float a, float b, f32x16v c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
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

// Stage rows j0 .. j0+63 of K and V (head h, zero past Lk) into LDS with row
// stride SKV floats.  ds_read_b32 serves each half-wave from 32 banks, so an
// odd stride makes "one row per lane" reads conflict-free; "one column per
// lane" reads are conflict-free for any stride.
template <int HD, int SKV>
__device__ __forceinline__ void attn_stage_kv(const AttnArgs& A, int64_t kv0, int32_t Lk, int32_t j0, int h,
                                              float* sk, float* sv) {
  for (int e = threadIdx.x; e < 64 * HD / 4; e += 256) {
    const int rr = e / (HD / 4), c = 4 * (e % (HD / 4));
    float4 kq = make_float4(0.f, 0.f, 0.f, 0.f), vq = kq;
    if (j0 + rr < Lk) {
      const int64_t row = kv0 + j0 + rr;
      kq = *reinterpret_cast<const float4*>(A.K + row * A.ldkv + A.kcol + h * HD + c);
      vq = *reinterpret_cast<const float4*>(A.V + row * A.ldkv + A.vcol + h * HD + c);
    }
    float* kd = sk + rr * SKV + c;
    float* vd = sv + rr * SKV + c;
    kd[0] = kq.x; kd[1] = kq.y; kd[2] = kq.z; kd[3] = kq.w;
    vd[0] = vq.x; vd[1] = vq.y; vd[2] = vq.z; vd[3] = vq.w;
  }
}

// reg[i] = row[2i + half], i < HD/2, through 16-byte loads
template <int HD>
__device__ __forceinline__ void attn_row_regs(const float* row, int half, float (&reg)[HD / 2]) {
#pragma unroll
  for (int j = 0; j < HD / 4; ++j) {
    const float4 f = *reinterpret_cast<const float4*>(row + 4 * j);
    reg[2 * j] = half ? f.y : f.x;
    reg[2 * j + 1] = half ? f.w : f.z;
  }
}

// Forward: one workgroup per (sample, head); wave w takes query group w & 1
// and the 32-key blocks of parity w >> 1 of every 64-key tile; the two key
// halves merge their (max, sum, output) at the end.
template <int HD>
__global__ __launch_bounds__(256) void xattn_fwd_kernel(AttnArgs A) {
  constexpr int SKV = HD + 1;
  constexpr int NT = HD / 2, NCB = HD / 32;
  __shared__ float smem[2 * 64 * SKV];
  float* sk = smem;
  float* sv = smem + 64 * SKV;
  const int k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = wave & 1, par = wave >> 1, half = lane >> 5, col = lane & 31;
  const int q = 32 * g + col;
  const bool qlive = q < Lq, glive = 32 * g < Lq;
  float qreg[NT];
  attn_row_regs<HD>(A.Q + (int64_t)(q0 + min(q, Lq - 1)) * A.ldq + h * HD, half, qreg);
  if (!qlive) {
#pragma unroll
    for (int i = 0; i < NT; ++i) qreg[i] = 0.f;
  }
  f32x16v o[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[cb][r] = 0.f;
  float m = -INFINITY, l = 0.f;
  for (int32_t j0 = 0; j0 < Lk; j0 += 64) {
    __syncthreads();
    attn_stage_kv<HD, SKV>(A, kv0, Lk, j0, h, sk, sv);
    __syncthreads();
    const int32_t kb = j0 + 32 * par;
    if (kb >= Lk || !glive) continue;
    f32x16v sc;
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[r] = 0.f;
    const float* kr = sk + (32 * par + col) * SKV + half;
#pragma unroll 16
    for (int i = 0; i < NT; ++i) sc = mfma32(kr[2 * i], qreg[i], sc);
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      sc[r] = (kb + mrow(r, half) < Lk) ? sc[r] * A.scale : -INFINITY;
      mx = fmaxf(mx, sc[r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mn = fmaxf(m, mx);
    const float alpha = __expf(m - mn);
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      sc[r] = __expf(sc[r] - mn);
      ps += sc[r];
    }
    ps += __shfl_xor(ps, 32, 64);
    l = l * alpha + ps;
    m = mn;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) o[cb][r] *= alpha;
      const float* vr = sv + (32 * par) * SKV + 32 * cb + col;
#pragma unroll
      for (int t = 0; t < 16; ++t) o[cb] = mfma32(vr[mrow(t, half) * SKV], sc[t], o[cb]);
    }
  }
  // merge the two key halves of each query group
  constexpr int MS = NCB * 16 + 2;
  __syncthreads();
  float* mb = smem + (g * 64 + lane) * MS;
  if (par == 1) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mb[cb * 16 + r] = o[cb][r];
    mb[NCB * 16] = m;
    mb[NCB * 16 + 1] = l;
  }
  __syncthreads();
  if (par == 1 || !qlive) return;
  {
    const float m1 = mb[NCB * 16], l1 = mb[NCB * 16 + 1];
    const float mn = fmaxf(m, m1);
    const float a0 = m == -INFINITY ? 0.f : __expf(m - mn), a1 = m1 == -INFINITY ? 0.f : __expf(m1 - mn);
    l = l * a0 + l1 * a1;
    m = mn;
    const float inv = 1.f / l;
    float* orow = A.O + (int64_t)(q0 + q) * A.ldo + h * HD;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (o[cb][4 * a4 + e] * a0 + mb[cb * 16 + 4 * a4 + e] * a1) * inv;
        *reinterpret_cast<float4*>(orow + 32 * cb + 8 * a4 + 4 * half) = make_float4(v[0], v[1], v[2], v[3]);
      }
    if (half == 0) A.lse[(int64_t)(q0 + q) * A.nheads + h] = m + __logf(l);
  }
}

// Backward, query side: dQ = scale * dS K with dS = P * (dP - D), P recomputed
// from the saved log-sum-exp, dP^T = V dO^T, D = rowsum(dO * O).  Same wave
// roles as the forward; the key halves' partial dQ are summed at the end.
template <int HD>
__global__ __launch_bounds__(256) void xattn_bwd_dq_kernel(AttnArgs A) {
  constexpr int SKV = HD + 1;
  constexpr int NT = HD / 2, NCB = HD / 32;
  __shared__ float smem[2 * 64 * SKV];
  float* sk = smem;
  float* sv = smem + 64 * SKV;
  const int k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = wave & 1, par = wave >> 1, half = lane >> 5, col = lane & 31;
  const int q = 32 * g + col;
  const bool qlive = q < Lq, glive = 32 * g < Lq;
  float qreg[NT], dreg[NT];
  float Dq = 0.f, lse = 0.f;
  {
    const int64_t row = q0 + min(q, Lq - 1);
    attn_row_regs<HD>(A.Q + row * A.ldq + h * HD, half, qreg);
    attn_row_regs<HD>(A.dO + row * A.ldo + h * HD, half, dreg);
    const float* orr = A.O + row * A.ldo + h * HD;
#pragma unroll
    for (int j = 0; j < HD / 4; ++j) {
      const float4 f = *reinterpret_cast<const float4*>(orr + 4 * j);
      Dq = fmaf(dreg[2 * j], half ? f.y : f.x, Dq);
      Dq = fmaf(dreg[2 * j + 1], half ? f.w : f.z, Dq);
    }
    Dq += __shfl_xor(Dq, 32, 64);
    if (!qlive) {
      Dq = 0.f;
#pragma unroll
      for (int i = 0; i < NT; ++i) qreg[i] = dreg[i] = 0.f;
    }
    lse = qlive ? A.lse[row * A.nheads + h] : 0.f;
  }
  f32x16v dq[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[cb][r] = 0.f;
  for (int32_t j0 = 0; j0 < Lk; j0 += 64) {
    __syncthreads();
    attn_stage_kv<HD, SKV>(A, kv0, Lk, j0, h, sk, sv);
    __syncthreads();
    const int32_t kb = j0 + 32 * par;
    if (kb >= Lk || !glive) continue;
    f32x16v sc, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[r] = dp[r] = 0.f;
    const float* kr = sk + (32 * par + col) * SKV + half;
    const float* vr = sv + (32 * par + col) * SKV + half;
#pragma unroll 16
    for (int i = 0; i < NT; ++i) {
      sc = mfma32(kr[2 * i], qreg[i], sc);
      dp = mfma32(vr[2 * i], dreg[i], dp);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const bool ok = qlive && kb + mrow(r, half) < Lk;
      const float p = ok ? __expf(sc[r] * A.scale - lse) : 0.f;
      sc[r] = p * (dp[r] - Dq);  // dS
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const float* kc = sk + (32 * par) * SKV + 32 * cb + col;
#pragma unroll
      for (int t = 0; t < 16; ++t) dq[cb] = mfma32(kc[mrow(t, half) * SKV], sc[t], dq[cb]);
    }
  }
  constexpr int MS = NCB * 16;
  __syncthreads();
  float* mb = smem + (g * 64 + lane) * MS;
  if (par == 1) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mb[cb * 16 + r] = dq[cb][r];
  }
  __syncthreads();
  if (par == 1 || !qlive) return;
  float* qrow = A.dQ + (int64_t)(q0 + q) * A.lddq + h * HD;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (dq[cb][4 * a4 + e] + mb[cb * 16 + 4 * a4 + e]) * A.scale;
      *reinterpret_cast<float4*>(qrow + 32 * cb + 8 * a4 + 4 * half) = make_float4(v[0], v[1], v[2], v[3]);
    }
}

// Backward, key side: one wave per 32-key block (grid z covers the longest
// sample).  Scores are computed untransposed here, S = Q K^T (lane = key,
// registers = queries), so P and dS are already the B operands of
// dV^T = dO^T P and dK^T = Q^T dS with the query index permuted as in the
// forward: nothing is transposed through memory.
template <int HD>
__global__ __launch_bounds__(256, 1) void xattn_bwd_dkv_kernel(AttnArgs A) {
  constexpr int SQ = HD + 1;
  constexpr int NT = HD / 2, NCB = HD / 32;
  __shared__ float sq[64 * SQ], sdo[64 * SQ];
  __shared__ float sD[64], sL[64];
  const int k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  if ((int32_t)blockIdx.z * 128 >= Lk) return;  // uniform over the workgroup
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  for (int e = threadIdx.x; e < 64 * HD / 4; e += 256) {
    const int rr = e / (HD / 4), c = 4 * (e % (HD / 4));
    float4 qq = make_float4(0.f, 0.f, 0.f, 0.f), dd = qq;
    if (rr < Lq) {
      qq = *reinterpret_cast<const float4*>(A.Q + (int64_t)(q0 + rr) * A.ldq + h * HD + c);
      dd = *reinterpret_cast<const float4*>(A.dO + (int64_t)(q0 + rr) * A.ldo + h * HD + c);
    }
    float* qd = sq + rr * SQ + c;
    float* dd2 = sdo + rr * SQ + c;
    qd[0] = qq.x; qd[1] = qq.y; qd[2] = qq.z; qd[3] = qq.w;
    dd2[0] = dd.x; dd2[1] = dd.y; dd2[2] = dd.z; dd2[3] = dd.w;
  }
  {
    // D[q] = sum_c dO[q][c] O[q][c]: 4 threads per query, 16-byte loads
    const int qq = threadIdx.x >> 2, part = threadIdx.x & 3;
    float acc = 0.f;
    if (qq < Lq) {
      const float* orow = A.O + (int64_t)(q0 + qq) * A.ldo + h * HD;
      const float* drow = A.dO + (int64_t)(q0 + qq) * A.ldo + h * HD;
      for (int c = 4 * part; c < HD; c += 16) {
        const float4 o4 = *reinterpret_cast<const float4*>(orow + c);
        const float4 d4 = *reinterpret_cast<const float4*>(drow + c);
        acc = fmaf(o4.x, d4.x, fmaf(o4.y, d4.y, fmaf(o4.z, d4.z, fmaf(o4.w, d4.w, acc))));
      }
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    if (part == 0) {
      sD[qq] = acc;
      sL[qq] = qq < Lq ? A.lse[(int64_t)(q0 + qq) * A.nheads + h] : 0.f;
    }
  }
  __syncthreads();
  const int32_t kb = (int32_t)blockIdx.z * 128 + 32 * wave;
  if (kb >= Lk) return;  // no barrier follows
  const bool kvalid = kb + col < Lk;  // this lane's key
  float kreg[NT], vreg[NT];
  {
    const int64_t row = kv0 + min(kb + col, Lk - 1);
    attn_row_regs<HD>(A.K + row * A.ldkv + A.kcol + h * HD, half, kreg);
    attn_row_regs<HD>(A.V + row * A.ldkv + A.vcol + h * HD, half, vreg);
  }
  f32x16v dk[NCB], dv[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[cb][r] = dv[cb][r] = 0.f;
  for (int g = 0; 32 * g < Lq; ++g) {
    f32x16v sc, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[r] = dp[r] = 0.f;
    const float* qa = sq + (32 * g + col) * SQ + half;
    const float* da = sdo + (32 * g + col) * SQ + half;
#pragma unroll 16
    for (int i = 0; i < NT; ++i) {
      sc = mfma32(qa[2 * i], kreg[i], sc);  // S[query 32g + mrow(r)][key kb + col]
      dp = mfma32(da[2 * i], vreg[i], dp);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int qq = 32 * g + mrow(r, half);
      const bool ok = kvalid && qq < Lq;
      const float p = ok ? __expf(sc[r] * A.scale - sL[qq]) : 0.f;
      dp[r] = p * (dp[r] - sD[qq]);  // dS
      sc[r] = p;
    }
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int qr = 32 * g + mrow(t, half);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        dv[cb] = mfma32(sdo[qr * SQ + 32 * cb + col], sc[t], dv[cb]);
        dk[cb] = mfma32(sq[qr * SQ + 32 * cb + col], dp[t], dk[cb]);
      }
    }
  }
  // dV^T / dK^T accumulators: lane = key kb + col, register r = column 32cb + mrow(r, half)
  if (!kvalid) return;
  const int64_t row = kv0 + kb + col;
  float* dvr = A.dV + row * A.lddkv + A.dvcol + h * HD;
  float* dkr = A.dK + row * A.lddkv + A.dkcol + h * HD;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      const int c = 32 * cb + 8 * a4 + 4 * half;
      *reinterpret_cast<float4*>(dvr + c) =
          make_float4(dv[cb][4 * a4], dv[cb][4 * a4 + 1], dv[cb][4 * a4 + 2], dv[cb][4 * a4 + 3]);
      *reinterpret_cast<float4*>(dkr + c) =
          make_float4(dk[cb][4 * a4] * A.scale, dk[cb][4 * a4 + 1] * A.scale, dk[cb][4 * a4 + 2] * A.scale,
                      dk[cb][4 * a4 + 3] * A.scale);
    }
}

hipError_t launch_xattn(hipStream_t s, const AttnArgs& A, int32_t nsamples, bool backward) {
  if (A.Lq > 64 || A.Lq < 1 || A.max_lk < 1) return hipErrorInvalidValue;
  const dim3 grid(nsamples, A.nheads), gk(nsamples, A.nheads, (A.max_lk + 127) / 128);
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

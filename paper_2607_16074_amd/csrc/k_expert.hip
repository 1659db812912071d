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
//   attention    fp32 self- / cross-attention forward and backward, one
//                workgroup per (sample, head); a sample's queries never see
//                another sample's keys
//   loss         per-tenant mean squared error and its gradient
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

// ---------------------------------------------------------------- copy2d ---

__global__ __launch_bounds__(256) void copy2d_kernel(const CopyDesc* __restrict__ descs, int32_t ndesc) {
  int32_t p = 0;
  const int32_t b = blockIdx.x;
  while (p + 1 < ndesc && descs[p + 1].block_start <= b) ++p;
  const CopyDesc D = descs[p];
  const int64_t total = (int64_t)D.rows * D.cols;
  const int64_t base = (int64_t)(b - D.block_start) * 256 * 8;
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
    d[i].block_start = total;
    total += (int32_t)(((int64_t)d[i].rows * d[i].cols + 2047) / 2048);
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

__global__ __launch_bounds__(256) void transpose_kernel(const TransDesc* __restrict__ descs, int32_t ndesc) {
  __shared__ uint16_t tile[64][66];
  int32_t p = 0;
  const int32_t b = blockIdx.x;
  while (p + 1 < ndesc && descs[p + 1].block_start <= b) ++p;
  const TransDesc D = descs[p];
  const int32_t tcols = (D.cols + 63) / 64;
  const int32_t local = b - D.block_start;
  const int32_t r0 = (local / tcols) * 64, c0 = (local % tcols) * 64;
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

// dg_t[j] = sum over tenant t's rows of gx[row][j]  (grid: tenant x column block)
__global__ __launch_bounds__(256) void colsum_kernel(const float* __restrict__ gx, const int32_t* __restrict__ roff,
                                                    float* const* __restrict__ out, int32_t d) {
  const int32_t t = blockIdx.x;
  const int32_t j = blockIdx.y * 256 + threadIdx.x;
  if (j >= d) return;
  float s = 0.f;
  for (int32_t r = roff[t]; r < roff[t + 1]; ++r) s += gx[(int64_t)r * d + j];
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
                           int32_t rows, int32_t d, float eps, const float* dh, float* dx, float* gx,
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
  dim3 g2(G, (d + 255) / 256);
  colsum_kernel<<<g2, 256, 0, s>>>(gx, roff, dg, d);
  return hipGetLastError();
}

// -------------------------------------------------------------- attention ---
// One workgroup per (sample k, head h); queries: rows q_row0 + 0..Lq-1 of Q
// (Lq <= 64); keys / values: rows kv_row0 .. kv_row0 + Lk - 1 of K / V.  Self
// attention: kv rows = the sample's own action rows; cross attention: the
// sample's rows of the tenant-ordered prefix (zoff).  Thread t owns query row
// t >> 2 and a quarter of the head dims; keys are processed 32 at a time.

constexpr int kAQ = 64;   // max queries per sample
constexpr int kAK = 32;   // keys per step

template <int HD>
struct AttnSmem {
  float q[kAQ][HD + 1];
  float dO[kAQ][HD + 1];
  float k[kAK][HD + 1];
  float v[kAK][HD + 1];
  float p[kAQ][kAK + 1];
  float ds[kAQ][kAK + 1];
};

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

template <int HD>
__global__ __launch_bounds__(256) void xattn_fwd_kernel(AttnArgs A) {
  constexpr int QD = HD / 4;  // dims per thread
  __shared__ AttnSmem<HD> sm;
  const int32_t k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  const int t = threadIdx.x, r = t >> 2, qd = t & 3;
  const bool live = r < Lq;
  for (int e = t; e < kAQ * HD; e += 256) {
    const int rr = e / HD, c = e % HD;
    sm.q[rr][c] = rr < Lq ? A.Q[(int64_t)(q0 + rr) * A.ldq + h * HD + c] : 0.f;
  }
  float o[QD];
#pragma unroll
  for (int i = 0; i < QD; ++i) o[i] = 0.f;
  float m = -INFINITY, l = 0.f;
  for (int32_t j0 = 0; j0 < Lk; j0 += kAK) {
    __syncthreads();
    for (int e = t; e < kAK * HD; e += 256) {
      const int jj = e / HD, c = e % HD;
      const bool ok = j0 + jj < Lk;
      const int64_t row = kv0 + j0 + jj;
      sm.k[jj][c] = ok ? A.K[row * A.ldkv + A.kcol + h * HD + c] : 0.f;
      sm.v[jj][c] = ok ? A.V[row * A.ldkv + A.vcol + h * HD + c] : 0.f;
    }
    __syncthreads();
    float s[kAK / 4];
    float bm = -INFINITY;
#pragma unroll
    for (int u = 0; u < kAK / 4; ++u) {
      const int jj = qd + 4 * u;
      float acc = 0.f;
#pragma unroll 8
      for (int c = 0; c < HD; ++c) acc = fmaf(sm.q[r][c], sm.k[jj][c], acc);
      s[u] = (j0 + jj < Lk) ? acc * A.scale : -INFINITY;
      bm = fmaxf(bm, s[u]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 1, 64));
    bm = fmaxf(bm, __shfl_xor(bm, 2, 64));
    const float mn = fmaxf(m, bm);
    const float alpha = __expf(m - mn);
    float ls = 0.f;
#pragma unroll
    for (int u = 0; u < kAK / 4; ++u) {
      const float pv = __expf(s[u] - mn);
      sm.p[r][qd + 4 * u] = pv;
      ls += pv;
    }
    ls += __shfl_xor(ls, 1, 64);
    ls += __shfl_xor(ls, 2, 64);
    l = l * alpha + ls;
    m = mn;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < QD; ++i) o[i] *= alpha;
    for (int jj = 0; jj < kAK; ++jj) {
      const float pv = sm.p[r][jj];
#pragma unroll
      for (int i = 0; i < QD; ++i) o[i] = fmaf(pv, sm.v[jj][qd * QD + i], o[i]);
    }
  }
  if (!live) return;
  const float inv = 1.f / l;
  float* orow = A.O + (int64_t)(q0 + r) * A.ldo + h * HD + qd * QD;
#pragma unroll
  for (int i = 0; i < QD; i += 4)
    *reinterpret_cast<float4*>(orow + i) = make_float4(o[i] * inv, o[i + 1] * inv, o[i + 2] * inv, o[i + 3] * inv);
  if (qd == 0) A.lse[(int64_t)(q0 + r) * A.nheads + h] = m + __logf(l);
}

template <int HD>
__global__ __launch_bounds__(256) void xattn_bwd_kernel(AttnArgs A) {
  constexpr int QD = HD / 4;
  __shared__ AttnSmem<HD> sm;
  const int32_t k = blockIdx.x, h = blockIdx.y;
  int32_t q0, Lq, Lk;
  int64_t kv0;
  attn_rows(A, k, q0, Lq, kv0, Lk);
  const int t = threadIdx.x, r = t >> 2, qd = t & 3;
  const bool live = r < Lq;
  for (int e = t; e < kAQ * HD; e += 256) {
    const int rr = e / HD, c = e % HD;
    const bool ok = rr < Lq;
    sm.q[rr][c] = ok ? A.Q[(int64_t)(q0 + rr) * A.ldq + h * HD + c] : 0.f;
    sm.dO[rr][c] = ok ? A.dO[(int64_t)(q0 + rr) * A.ldo + h * HD + c] : 0.f;
  }
  // D_r = sum_c dO[r][c] O[r][c]
  float Dr = 0.f;
  if (live) {
    const float* orow = A.O + (int64_t)(q0 + r) * A.ldo + h * HD + qd * QD;
    const float* drow = A.dO + (int64_t)(q0 + r) * A.ldo + h * HD + qd * QD;
#pragma unroll 8
    for (int i = 0; i < QD; ++i) Dr = fmaf(orow[i], drow[i], Dr);
  }
  Dr += __shfl_xor(Dr, 1, 64);
  Dr += __shfl_xor(Dr, 2, 64);
  const float lse = live ? A.lse[(int64_t)(q0 + r) * A.nheads + h] : 0.f;
  float dq[QD];
#pragma unroll
  for (int i = 0; i < QD; ++i) dq[i] = 0.f;
  for (int32_t j0 = 0; j0 < Lk; j0 += kAK) {
    __syncthreads();
    for (int e = t; e < kAK * HD; e += 256) {
      const int jj = e / HD, c = e % HD;
      const bool ok = j0 + jj < Lk;
      const int64_t row = kv0 + j0 + jj;
      sm.k[jj][c] = ok ? A.K[row * A.ldkv + A.kcol + h * HD + c] : 0.f;
      sm.v[jj][c] = ok ? A.V[row * A.ldkv + A.vcol + h * HD + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kAK / 4; ++u) {
      const int jj = qd + 4 * u;
      float sacc = 0.f, pacc = 0.f;
#pragma unroll 8
      for (int c = 0; c < HD; ++c) {
        sacc = fmaf(sm.q[r][c], sm.k[jj][c], sacc);
        pacc = fmaf(sm.dO[r][c], sm.v[jj][c], pacc);
      }
      const bool ok = live && (j0 + jj < Lk);
      const float pv = ok ? __expf(sacc * A.scale - lse) : 0.f;
      sm.p[r][jj] = pv;
      sm.ds[r][jj] = pv * (pacc - Dr);
    }
    __syncthreads();
    // dQ[r] += scale * sum_j dS[r][j] K[j]
    for (int jj = 0; jj < kAK; ++jj) {
      const float w = sm.ds[r][jj] * A.scale;
#pragma unroll
      for (int i = 0; i < QD; ++i) dq[i] = fmaf(w, sm.k[jj][qd * QD + i], dq[i]);
    }
    // dV[j] = sum_r P[r][j] dO[r];  dK[j] = scale * sum_r dS[r][j] Q[r]
    {
      const int jj = t >> 3, c0 = (t & 7) * (HD / 8);
      float dv[HD / 8], dk[HD / 8];
#pragma unroll
      for (int i = 0; i < HD / 8; ++i) dv[i] = dk[i] = 0.f;
      for (int rr = 0; rr < Lq; ++rr) {
        const float pv = sm.p[rr][jj], dsv = sm.ds[rr][jj];
#pragma unroll
        for (int i = 0; i < HD / 8; ++i) {
          dv[i] = fmaf(pv, sm.dO[rr][c0 + i], dv[i]);
          dk[i] = fmaf(dsv, sm.q[rr][c0 + i], dk[i]);
        }
      }
      if (j0 + jj < Lk) {
        const int64_t row = kv0 + j0 + jj;
        float* dvp = A.dV + row * A.lddkv + A.dvcol + h * HD + c0;
        float* dkp = A.dK + row * A.lddkv + A.dkcol + h * HD + c0;
#pragma unroll
        for (int i = 0; i < HD / 8; i += 4) {
          *reinterpret_cast<float4*>(dvp + i) = make_float4(dv[i], dv[i + 1], dv[i + 2], dv[i + 3]);
          *reinterpret_cast<float4*>(dkp + i) =
              make_float4(dk[i] * A.scale, dk[i + 1] * A.scale, dk[i + 2] * A.scale, dk[i + 3] * A.scale);
        }
      }
    }
  }
  if (!live) return;
  float* qrow = A.dQ + (int64_t)(q0 + r) * A.lddq + h * HD + qd * QD;
#pragma unroll
  for (int i = 0; i < QD; i += 4) *reinterpret_cast<float4*>(qrow + i) = make_float4(dq[i], dq[i + 1], dq[i + 2], dq[i + 3]);
}

hipError_t launch_xattn(hipStream_t s, const AttnArgs& A, int32_t nsamples, bool backward) {
  if (A.Lq > kAQ || A.Lq < 1) return hipErrorInvalidValue;
  dim3 grid(nsamples, A.nheads);
  switch (A.hd) {
    case 64:
      if (backward) xattn_bwd_kernel<64><<<grid, 256, 0, s>>>(A); else xattn_fwd_kernel<64><<<grid, 256, 0, s>>>(A);
      break;
    case 128:
      if (backward) xattn_bwd_kernel<128><<<grid, 256, 0, s>>>(A); else xattn_fwd_kernel<128><<<grid, 256, 0, s>>>(A);
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

}  // namespace jnx

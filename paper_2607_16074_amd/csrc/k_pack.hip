// Pack (canonicalize + pad into one physical batch) and unpack (split back by
// the recorded slices).  Both are plain HBM copies: 16-byte lanes, one block
// per (sample, 16-row slab), coalesced along the row.
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

constexpr int kRowsPerBlock = 16;

__global__ __launch_bounds__(256) void pack_kernel(const ReqEntry* __restrict__ req_table,
                                                   const int32_t* __restrict__ sample_request,
                                                   const int32_t* __restrict__ sample_local,
                                                   const int32_t* __restrict__ seqlens,
                                                   const int32_t* __restrict__ cu_seqlens, int32_t d,
                                                   uint4* __restrict__ tokens, int32_t* __restrict__ token_sample,
                                                   int32_t* __restrict__ token_pos) {
  const int32_t i = blockIdx.x;
  const int32_t base = cu_seqlens[i];
  const int32_t rows = cu_seqlens[i + 1] - base;  // aligned rows of this sample
  const int32_t j0 = blockIdx.y * kRowsPerBlock;
  if (j0 >= rows) return;
  const int32_t nr = min(kRowsPerBlock, rows - j0);
  const int32_t L = seqlens[i];
  const ReqEntry e = req_table[sample_request[i]];
  const int32_t s = sample_local[i];
  const int32_t chunks = d / 8;  // 16-byte chunks per row
  const uint4* src = reinterpret_cast<const uint4*>(e.in) + ((int64_t)s * e.max_len + j0) * chunks;
  uint4* dst = tokens + (int64_t)(base + j0) * chunks;
  for (int32_t idx = threadIdx.x; idx < nr * chunks; idx += blockDim.x) {
    const int32_t r = idx / chunks;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (j0 + r < L) v = src[idx];
    dst[idx] = v;
  }
  if (threadIdx.x < nr) {
    const int32_t j = j0 + threadIdx.x;
    token_sample[base + j] = j < L ? i : -1;
    token_pos[base + j] = j < L ? j : -1;
  }
}

template <typename V>
__global__ __launch_bounds__(256) void unpack_kernel(const ReqEntry* __restrict__ req_table,
                                                     const int32_t* __restrict__ sample_request,
                                                     const int32_t* __restrict__ sample_local,
                                                     const int32_t* __restrict__ seqlens,
                                                     const int32_t* __restrict__ cu_seqlens, const V* __restrict__ rows,
                                                     int64_t row_vecs) {
  const int32_t i = blockIdx.x;
  const ReqEntry e = req_table[sample_request[i]];
  const int32_t j0 = blockIdx.y * kRowsPerBlock;
  const int32_t s = sample_local[i];
  // the host checks that the requests match the packed batch; a sample
  // beyond its request's buffer is still never written
  if (j0 >= e.max_len || s >= e.n) return;
  const int32_t nr = min(kRowsPerBlock, e.max_len - j0);
  const int32_t L = seqlens[i];
  V* dst = reinterpret_cast<V*>(e.out) + ((int64_t)s * e.max_len + j0) * row_vecs;
  const V* src = rows + (int64_t)(cu_seqlens[i] + j0) * row_vecs;
  for (int64_t idx = threadIdx.x; idx < nr * row_vecs; idx += blockDim.x) {
    const int32_t r = (int32_t)(idx / row_vecs);
    V v{};
    if (j0 + r < L) v = src[idx];
    dst[idx] = v;
  }
}

hipError_t launch_pack(hipStream_t s, const ReqEntry* req_table, const int32_t* sample_request,
                       const int32_t* sample_local, const int32_t* seqlens, const int32_t* cu_seqlens, int32_t N,
                       int32_t d, int32_t align, int32_t max_rows, void* tokens, int32_t* token_sample,
                       int32_t* token_pos) {
  (void)align;
  dim3 grid(N, (max_rows + kRowsPerBlock - 1) / kRowsPerBlock);
  pack_kernel<<<grid, 256, 0, s>>>(req_table, sample_request, sample_local, seqlens, cu_seqlens, d,
                                   reinterpret_cast<uint4*>(tokens), token_sample, token_pos);
  return hipGetLastError();
}

hipError_t launch_unpack(hipStream_t s, const ReqEntry* req_table, const int32_t* sample_request,
                         const int32_t* sample_local, const int32_t* seqlens, const int32_t* cu_seqlens, int32_t N,
                         int32_t max_req_len, const void* rows, int64_t row_bytes, bool vec16) {
  dim3 grid(N, (max_req_len + kRowsPerBlock - 1) / kRowsPerBlock);
  // vec16: the caller checked that the source, every destination and the row
  // pitch are 16-byte aligned
  if (vec16)
    unpack_kernel<uint4><<<grid, 256, 0, s>>>(req_table, sample_request, sample_local, seqlens, cu_seqlens,
                                              reinterpret_cast<const uint4*>(rows), row_bytes / 16);
  else
    unpack_kernel<uint32_t><<<grid, 256, 0, s>>>(req_table, sample_request, sample_local, seqlens, cu_seqlens,
                                                 reinterpret_cast<const uint32_t*>(rows), row_bytes / 4);
  return hipGetLastError();
}

}  // namespace jnx

// Internal declarations shared by the host library and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "joynexus.h"

namespace jnx {

// Device request table entry (one per request), written by jn_pack_group and
// patched by jn_unpack with the output pointer.
struct ReqEntry {
  const void* in;      // bf16 [n][max_len][d]
  void* out;           // unpack destination [n][max_len][row_bytes]
  int32_t max_len;
  int32_t n;
  int32_t first;       // packed index of the request's first sample
  int32_t reserved;
};
static_assert(sizeof(ReqEntry) == 32, "ReqEntry layout");

// ------------------------------------------------------------ launchers ---
// All launchers enqueue on `s`; shapes were validated by the caller.

hipError_t launch_pack(hipStream_t s, const ReqEntry* req_table, const int32_t* sample_request,
                       const int32_t* sample_local, const int32_t* seqlens, const int32_t* cu_seqlens,
                       int32_t N, int32_t d, int32_t align, int32_t max_rows, void* tokens,
                       int32_t* token_sample, int32_t* token_pos);

hipError_t launch_unpack(hipStream_t s, const ReqEntry* req_table, const int32_t* sample_request,
                         const int32_t* sample_local, const int32_t* seqlens, const int32_t* cu_seqlens,
                         int32_t N, int32_t max_req_len, const void* rows, int64_t row_bytes, bool vec16);

// x_out (fp32, optional) = widened x_bf16; h = RMS(x) * g  (bf16)
hipError_t launch_rmsnorm_bf16in(hipStream_t s, const void* x_bf16, float* x_out, const void* g,
                                 void* h, int32_t rows, int32_t d, float eps);
// h = RMS(x) * g (bf16) from the fp32 residual stream
hipError_t launch_rmsnorm_f32in(hipStream_t s, const float* x, const void* g, void* h, int32_t rows,
                                int32_t d, float eps);

enum GemmEpi : int32_t {
  EPI_BF16 = 0,          // C bf16 = acc
  EPI_GELU_BF16 = 1,     // C bf16 = gelu(acc)
  EPI_RESID_F32 = 2,     // C fp32 += acc
  EPI_GEGLU_BF16 = 3,    // weights gate|up interleaved at load; C bf16 = gelu(gate) * up
  EPI_F32 = 4,           // C fp32 = acc
  EPI_GELU_SAVE = 5,     // aux fp32 = acc; C bf16 = gelu(acc)
  EPI_GELUGRAD_BF16 = 6  // C bf16 = acc * gelu'(aux fp32)
};

// Operand layouts of a grouped problem (GemmArgs::trans): X stored [K][M]
// (element (m, k) at X[k * ldx + m]), W stored [K][N].
constexpr int GEMM_TRANS_X = 1, GEMM_TRANS_W = 2;

// One GEMM problem: C[M][N] (+)= epi(X[M][K] W[N][K]^T); bf16 X, W row-major
// unless `trans` says otherwise.
struct GemmArgs {
  const uint16_t* X;
  const uint16_t* W;
  const uint16_t* W2;   // GeGLU up weights
  void* C;
  float* aux;           // GELU pre-activation (saved or read)
  int64_t ldx, ldw, ldc, ldaux;
  int32_t M, N, K;
  int32_t tiles_m, tiles_n, tile_start;  // filled by the launchers
  int32_t trans;        // GEMM_TRANS_* bits (grouped launches on 256x256 tiles only)
  int64_t split_c;      // split-K: elements between the fp32 partial outputs of
                        // consecutive K ranges (blockIdx.y); 0 when unsplit
  int32_t xcd_ranges;   // split-K ring launches: K ranges dealt to XCD groups (set by the launcher)
};

// Grouped launch over nprob problems sharing one epilogue: the host fills
// the problems, calls gemm_grouped_prepare (tile ranges, returns the tile
// total, or -1 if a problem is not M, N, K > 0 with K % 64 == 0 and
// N % 32 == 0), uploads them and launches.  shape from gemm_grouped_tile_shape.
// Problems with transposed operands (all of one launch alike) run on the
// 256x256 tiles (shape 0, which gemm_grouped_tile_shape returns for them, or
// -1 where their offsets do not fit the loop's 32-bit ones); with both
// operands transposed K need not be a multiple of 64.  Combinations launched:
// EPI_F32 with GEMM_TRANS_W or both, EPI_GELUGRAD_BF16 with GEMM_TRANS_W.
int gemm_grouped_tile_shape(const GemmArgs* probs, int32_t nprob);
int32_t gemm_grouped_prepare(GemmArgs* probs, int32_t nprob, int shape);
hipError_t launch_gemm_grouped(hipStream_t s, int epi, const GemmArgs* dprobs, int32_t nprob, int32_t total_tiles,
                               int shape, int trans = 0);

// C[M][N] (+)= epi(A[M][K] * B[N][K]^T); A, B bf16 row-major with leading
// dims lda, ldb (elements); for EPI_GEGLU_BF16, B is w_gate and B2 is w_up,
// each [N][K], and C has N columns.
//
// Launches with few tiles for the GPU and a long K (epilogues EPI_BF16,
// EPI_RESID_F32, EPI_GELU_BF16) split K into gemm_split() ranges when
// `split_ws` holds gemm_split_bytes(): each range writes fp32 partials and a
// reduction adds them in range order, then applies the epilogue.  The split
// depends only on (epi, M, N, K).
hipError_t launch_gemm(hipStream_t s, int epi, const void* A, int64_t lda, const void* B,
                       const void* B2, int64_t ldb, void* C, int64_t ldc, int32_t M, int32_t N,
                       int32_t K, int tile_hint, void* split_ws = nullptr, size_t split_bytes = 0);
int gemm_split(int epi, int32_t M, int32_t N, int32_t K);
size_t gemm_split_bytes(int epi, int32_t M, int32_t N, int32_t K);

// Varlen attention over the packed batch (bidirectional or causal inside each
// sample).  qkv: bf16 [T][(H + 2 Hkv) hd] (q | k | v); out: bf16 [T][d],
// d = H hd.  Query head h reads key/value head h / (H / Hkv).  Alignment rows
// of `out` are zeroed.
hipError_t launch_attention(hipStream_t s, const void* qkv, void* out, const int32_t* seqlens,
                            const int32_t* cu_seqlens, int32_t N, int32_t d, int32_t n_heads, int32_t n_kv_heads,
                            bool causal, int32_t max_seqlen, int32_t align);
// In-place rotary embedding of the first `heads` head slices (hd wide) of
// every row of qkv [T][ld] whose token_pos >= 0: pair (i, i + hd/2) rotated
// by token_pos * theta^(-2i/hd).
hipError_t launch_rope(hipStream_t s, void* qkv, int32_t ld, const int32_t* token_pos, int32_t T, int32_t heads,
                       int32_t hd, float theta);

// ---- heads ----
// pooled[sample_tenant_rank[i]][:] = mean over valid rows of hidden for sample i
hipError_t launch_pool(hipStream_t s, const void* hidden, const int32_t* seqlens,
                       const int32_t* cu_seqlens, const int32_t* rank, int32_t N, int32_t d,
                       float* pooled);

// Grouped fp32 GEMM descriptor for the tenant heads:
//   C(m,n) = sum_k A(m,k) B(k,n),  A(m,k) = A[m*sam + k*sak],  B(k,n) = B[k*sbk + n*sbn].
// Tenant-ordered operands are addressed from the tenant's first row: the
// kernel adds off_g * bump{A,B,C} to the base pointers, with
// off_g = tenant_sample_off[tenant] read on the device.  The one dimension
// equal to the tenant's row count n_g (M for forward / data-gradient, K for
// weight-gradient) is given as -1 and read on the device as well.
struct HeadGemm {
  const float* A;
  const float* B;
  float* C;
  const float* bias;  // forward: C(m,n) += bias[n]          (may be null)
  float* Cact;        // forward: also store gelu(C) (same ldc / bump as C)
  const float* Zg;    // data-gradient: C *= gelu'(Zg)  (same ldc / bump as C)
  float* db;          // weight-gradient: db[m] = sum_k A(m,k), by tn == 0 tiles
  float* part;        // ksplit > 1: K range t of tile (m, n) writes its raw sum to
                      // part[t * part_plane + off * bumpC + m * ldc + n]; the
                      // reduce launch adds the ranges in order and applies the epilogue
  int64_t part_plane;
  int64_t sam, sak, sbk, sbn, ldc;
  int64_t bumpA, bumpB, bumpC;
  int32_t M, N, K;
  int32_t tenant;
  int32_t tiles_n;
  int32_t ksplit;     // K ranges (1: the tile writes C with its epilogue)
};
struct HeadTile {
  int32_t desc;
  int32_t tm;
  int32_t tn;
  int32_t tk;  // K range (ksplit > 1)
};
hipError_t launch_head_gemm(hipStream_t s, const HeadGemm* descs, const HeadTile* tiles, int32_t n_tiles,
                            const int32_t* tenant_sample_off);
// Sum of the K ranges of split descriptors, then bias / GELU' / GELU as in
// the unsplit epilogue; tiles (desc, tm, tn, 0) of the split descriptors.
hipError_t launch_head_reduce(hipStream_t s, const HeadGemm* descs, const HeadTile* tiles, int32_t n_tiles,
                              const int32_t* tenant_sample_off);
// K ranges of a head GEMM of contraction length K (a function of K only, so
// a tenant's result does not depend on the rest of the batch).
inline int32_t head_ksplit(int64_t K) {
  const int64_t s = K / 256;
  return K < 512 ? 1 : (int32_t)(s > 8 ? 8 : s);
}

// Per-tenant mean squared error over n_g * out elements:
//   loss = mean((y - t)^2), dy = 2 (y - t) / (n_g * out), actions = y.
// y and dy are tenant-ordered ([N][ld], rows from off_g); target and actions
// are the tenant's own [n_g][out] buffers.
struct LossDesc {
  const float* y;
  const float* target;
  float* dy;
  float* loss;
  float* actions;
  int32_t out;
  int64_t ld;
  int32_t tenant;
  int32_t reserved;
};
// part: 16 G floats of scratch (per-tenant partial sums, two launches).
hipError_t launch_mse(hipStream_t s, const LossDesc* descs, int32_t G, const int32_t* tenant_sample_off, float* part);

// ---- action expert (k_expert.hip) ----
// dst[r][c] = cvt(src[r][c]) for r < src_rows, c < src_cols, else 0; r < rows, c < cols.
struct CopyDesc {
  const void* src;
  void* dst;
  int64_t src_ld, dst_ld;
  int32_t rows, cols, src_rows, src_cols;
  int32_t src_bf16, dst_bf16;
  int32_t block_start, vec;  // filled by copy2d_prepare
};
int32_t copy2d_prepare(CopyDesc* d, int32_t n);

// dst[i] = ((src[0][i] + src[1][i]) + ...) + src[S-1][i], i < n (parts
// n elements apart, fp32; n % 4 == 0, 16-byte aligned): the K ranges of a
// split weight gradient added in range order.
struct KSumDesc {
  const float* src;
  float* dst;
  int64_t n;
  int32_t S;
  int32_t block_start;  // filled by ksum_prepare
};
int32_t ksum_prepare(KSumDesc* d, int32_t n);
hipError_t launch_ksum(hipStream_t s, const KSumDesc* d, int32_t n, int32_t blocks);
hipError_t launch_copy2d(hipStream_t s, const CopyDesc* d, int32_t n, int32_t blocks);

// bf16 dst[c][r] = src[r][c] (r < rows), 0 for rows <= r < rows_pad; c < cols.
struct TransDesc {
  const uint16_t* src;
  uint16_t* dst;
  int64_t src_ld, dst_ld;
  int32_t rows, cols, rows_pad, block_start;
};
int32_t transpose_prepare(TransDesc* d, int32_t n);
hipError_t launch_transpose(hipStream_t s, const TransDesc* d, int32_t n, int32_t blocks);

// zoff[k] for tenant-order samples k (prefix sums of their valid lengths) and
// the tenant-ordered copy z of their backbone rows (rows >= cap dropped).
hipError_t launch_prefix(hipStream_t s, const void* hidden, const int32_t* tenant_perm, const int32_t* seqlens,
                         const int32_t* cu_seqlens, int32_t N, int32_t max_seqlen, int32_t d, int64_t cap,
                         int32_t* zoff, void* z);

// RMSNorm with per-tenant gains (rows tenant-contiguous, roff [G+1] device).
hipError_t launch_xrms_fwd(hipStream_t s, const float* x, const void* const* gains, const int32_t* roff, int32_t G,
                           int32_t rows, int32_t d, float eps, void* h);
// dx += dRMS(x, g) . dh ; dg[t] = column sums over tenant t's rows (gx scratch
// [rows][d], part scratch [G][16][d]).
hipError_t launch_xrms_bwd(hipStream_t s, const float* x, const void* const* gains, const int32_t* roff, int32_t G,
                           int32_t rows, int32_t d, float eps, const float* dh, float* dx, float* gx, float* part,
                           float* const* dg);

// fp32 attention of each tenant-order sample k over its own keys: queries
// rows [k*Lq, (k+1)*Lq) of Q; keys / values rows [kv0, kv0 + Lk) with
// kv0 = zoff[k], Lk = zoff[k+1] - zoff[k] (cross, clamped to kv_cap) or the
// sample's own query rows (self, zoff null).
struct AttnArgs {
  const uint16_t* Q;  // bf16
  const uint16_t* K;
  const uint16_t* V;
  float* O;        // forward output / backward input (fp32)
  uint16_t* Ob;    // forward output, bf16 copy of O (leading dimension ldo)
  float* lse;      // forward output / backward input, [rows][nheads], log2 domain
  float* dsum;     // backward scratch, [rows][nheads]: sum(dO * O) per query
  const float* dO;
  uint16_t* dQ;    // bf16 gradients
  uint16_t* dK;
  uint16_t* dV;
  const int32_t* zoff;
  int64_t ldq, ldkv, ldo, lddq, lddkv, kv_cap;
  int32_t kcol, vcol, dkcol, dvcol;
  int32_t Lq, hd, nheads, max_lk;    // max_lk: largest key count of any sample
  float scale;
};
hipError_t launch_xattn(hipStream_t s, const AttnArgs& A, int32_t nsamples, bool backward);

// Flow-matching inputs of one tenant's expert rows (rows = n * chunk, tenant
// arrival order): input row [x | 0 | phi(t)] (bf16, ld columns: x = t*noise +
// (1-t)*act in the first a, zeros up to kap, the d_time flow-time features
// after) and vel = noise - act (fp32 [rows][a]).
struct FlowDesc {
  const float* t;       // [n]
  const float* noise;   // [rows][a]
  const float* act;     // [rows][a]
  float* vel;           // [rows][a]
  int64_t roff;         // first row of the tenant in the expert's row space
  int32_t rows, a;
};
hipError_t launch_flow_prep(hipStream_t s, const FlowDesc* d, int32_t G, int64_t total_rows, int32_t chunk,
                            int32_t kap, int32_t d_time, uint16_t* in_rows, int32_t ld);

struct XLossDesc {
  const float* target;  // [rows_t][a]
  float* pred;          // [rows_t][a]
  float* loss;          // [1]
  int32_t a, reserved;
};
hipError_t launch_xloss(hipStream_t s, const XLossDesc* d, const int32_t* roff, int32_t G, const float* pred_pad,
                        int32_t ldp, float* dpred_pad);

// ------------------------------------------------------------ optimizer ---

struct AdamwTensor {
  float* p;
  const float* g;
  float* m;
  float* v;
  uint16_t* b16;        // optional bf16 copy of the new parameters
  int64_t numel;
  int32_t tenant, block_start;
};
// per tenant: p = p * decay - step_size * m / (sqrt(v) * inv_sqrt_bc2 + eps)
struct AdamwTenant {
  float decay, step_size, inv_sqrt_bc2, eps, b1, b2, reserved0, reserved1;
};
constexpr int64_t kAdamwBlockElems = 4096;
int32_t adamw_prepare(AdamwTensor* t, int32_t n);  // fills block_start, returns the block count
hipError_t launch_adamw(hipStream_t s, const AdamwTensor* t, int32_t n, const AdamwTenant* ten, int32_t blocks);

}  // namespace jnx

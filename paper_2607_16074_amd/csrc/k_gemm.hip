// bf16 GEMM for the backbone projections on gfx950 matrix cores.
//
//   C[M][N] (+)= epi( X[M][K] * W[N][K]^T )     X = activations, W = weights
//
// Tiling: a workgroup of 4 wavefronts (2 x 2) owns a BN x BM tile (weight rows
// x tokens); each wavefront accumulates (BN/2) x (BM/2) with
// v_mfma_f32_32x32x16_bf16.  The weight tile is the MFMA "A" operand, the
// token tile the "B" operand, so each lane ends with 4 consecutive output
// columns of one token row -- the epilogue writes 8-byte (bf16) / 16-byte
// (fp32) vectors along the row-major output.  K advances 64 at a time through
// double-buffered LDS (rows padded to 144 B: conflict-free 16-byte reads);
// the next K slab is fetched from global memory into registers while the
// current one feeds the MFMAs.  One barrier per K slab.
//
// Launch order: workgroups are dealt round-robin to the 8 XCDs; the tile id
// is remapped so that each XCD owns one contiguous range of tiles, walked in
// groups of 8 token-tiles, so concurrently resident tiles share weight and
// activation panels in that XCD's L2.
//
// Epilogues: bf16 store, GELU -> bf16, fp32 residual add (in place), and
// GeGLU, whose gate and up weights are interleaved in 32-row blocks while the
// weight tile is loaded, so the gate and up accumulators of an output column
// land in the same lane.
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;         // K slab
constexpr int kLDK = kBK + 8;   // LDS row pitch (elements): 144 B
constexpr int kGroupM = 8;      // token tiles per L2 group

template <int BN, int BM, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                      const uint16_t* __restrict__ W,
                                                      const uint16_t* __restrict__ W2, int64_t ldw,
                                                      void* __restrict__ C, int64_t ldc, int32_t M, int32_t N,
                                                      int32_t K, int32_t tiles_m, int32_t tiles_n) {
  constexpr bool GLU = EPI == EPI_GEGLU_BF16;
  constexpr int WN = BN / 2, WM = BM / 2;  // per-wave tile
  constexpr int TN = WN / 32, TM = WM / 32;
  constexpr int RW = BN / 32, RX = BM / 32;  // 16-byte chunks per thread per slab
  __shared__ __attribute__((aligned(16))) uint16_t Ws[2][BN][kLDK];
  __shared__ __attribute__((aligned(16))) uint16_t Xs[2][BM][kLDK];

  // ---- XCD-aware tile order
  const int32_t ntiles = tiles_m * tiles_n;
  const int32_t b = blockIdx.x;
  const int32_t xcd = b & 7, local = b >> 3;
  const int32_t q = ntiles >> 3, r = ntiles & 7;
  const int32_t pid = xcd * q + min(xcd, r) + local;
  const int32_t per_group = kGroupM * tiles_n;
  const int32_t group = pid / per_group;
  const int32_t first_m = group * kGroupM;
  const int32_t gsize = min(tiles_m - first_m, kGroupM);
  const int32_t tm = first_m + (pid % per_group) % gsize;
  const int32_t tn = (pid % per_group) / gsize;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wn = wave >> 1, wm = wave & 1;
  const int lrow = tid >> 3;        // 0..31: row within a 32-row band for loads
  const int lchunk = (tid & 7) * 8; // element offset of this thread's 16-byte chunk

  // ---- global row sources (clamped into range: ragged tiles load valid rows)
  const int32_t NL = GLU ? 2 * N : N;  // rows of the (interleaved) weight operand
  const uint16_t* wsrc[RW];
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    if constexpr (GLU) {
      int32_t col = tn * (BN / 2) + (i >> 1) * 32 + lrow;
      col = min(col, N - 1);
      wsrc[i] = ((i & 1) ? W2 : W) + (int64_t)col * ldw + lchunk;
    } else {
      int32_t row = min(tn * BN + i * 32 + lrow, NL - 1);
      wsrc[i] = W + (int64_t)row * ldw + lchunk;
    }
  }
  const int32_t xrow0 = tm * BM + lrow;

  uint4 rw[RW], rx[RX];
  auto load_slab = [&](int32_t k0) {
#pragma unroll
    for (int i = 0; i < RW; ++i) rw[i] = *reinterpret_cast<const uint4*>(wsrc[i] + k0);
#pragma unroll
    for (int i = 0; i < RX; ++i) {
      const int32_t row = min(xrow0 + i * 32, M - 1);
      rx[i] = *reinterpret_cast<const uint4*>(X + (int64_t)row * ldx + k0 + lchunk);
    }
  };
  auto store_slab = [&](int buf) {
#pragma unroll
    for (int i = 0; i < RW; ++i) *reinterpret_cast<uint4*>(&Ws[buf][i * 32 + lrow][lchunk]) = rw[i];
#pragma unroll
    for (int i = 0; i < RX; ++i) *reinterpret_cast<uint4*>(&Xs[buf][i * 32 + lrow][lchunk]) = rx[i];
  };

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int KT = K / kBK;
  load_slab(0);
  store_slab(0);
  __syncthreads();
  const int frow = lane & 31;
  const int fk = (lane >> 5) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) load_slab((kt + 1) * kBK);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8 fw[TN], fx[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i)
        fw[i] = *reinterpret_cast<const bf16x8*>(&Ws[cur][wn * WN + i * 32 + frow][kk * 16 + fk]);
#pragma unroll
      for (int j = 0; j < TM; ++j)
        fx[j] = *reinterpret_cast<const bf16x8*>(&Xs[cur][wm * WM + j * 32 + frow][kk * 16 + fk]);
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[i], fx[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) store_slab(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane owns output columns n..n+3 of token row m
  const int hi4 = (lane >> 5) * 4;
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int32_t m = tm * BM + wm * WM + j * 32 + (lane & 31);
    if (m >= M) continue;
    if constexpr (GLU) {
#pragma unroll
      for (int i = 0; i < TN; i += 2) {
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int32_t n = tn * (BN / 2) + wn * (WN / 2) + (i >> 1) * 32 + rr * 8 + hi4;
          if (n >= N) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = gelu_f(acc[i][j][rr * 4 + e]) * acc[i + 1][j][rr * 4 + e];
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
              make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < TN; ++i) {
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int32_t n = tn * BN + wn * WN + i * 32 + rr * 8 + hi4;
          if (n >= N) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][rr * 4 + e];
          if constexpr (EPI == EPI_RESID_F32) {
            float4* p = reinterpret_cast<float4*>(reinterpret_cast<float*>(C) + (int64_t)m * ldc + n);
            float4 o = *p;
            o.x += v[0];
            o.y += v[1];
            o.z += v[2];
            o.w += v[3];
            *p = o;
          } else {
            if constexpr (EPI == EPI_GELU_BF16) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = gelu_f(v[e]);
            }
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
          }
        }
      }
    }
  }
}

template <int BN, int BM>
static hipError_t launch_tile(hipStream_t s, int epi, const void* A, int64_t lda, const void* B, const void* B2,
                              int64_t ldb, void* C, int64_t ldc, int32_t M, int32_t N, int32_t K) {
  const int32_t NL = epi == EPI_GEGLU_BF16 ? 2 * N : N;
  const int32_t tiles_m = (M + BM - 1) / BM, tiles_n = (NL + BN - 1) / BN;
  dim3 grid(tiles_m * tiles_n);
  auto X = reinterpret_cast<const uint16_t*>(A);
  auto Wp = reinterpret_cast<const uint16_t*>(B);
  auto W2 = reinterpret_cast<const uint16_t*>(B2);
  switch (epi) {
    case EPI_BF16:
      gemm_kernel<BN, BM, EPI_BF16><<<grid, 256, 0, s>>>(X, lda, Wp, W2, ldb, C, ldc, M, N, K, tiles_m, tiles_n);
      break;
    case EPI_GELU_BF16:
      gemm_kernel<BN, BM, EPI_GELU_BF16><<<grid, 256, 0, s>>>(X, lda, Wp, W2, ldb, C, ldc, M, N, K, tiles_m, tiles_n);
      break;
    case EPI_RESID_F32:
      gemm_kernel<BN, BM, EPI_RESID_F32><<<grid, 256, 0, s>>>(X, lda, Wp, W2, ldb, C, ldc, M, N, K, tiles_m, tiles_n);
      break;
    case EPI_GEGLU_BF16:
      gemm_kernel<BN, BM, EPI_GEGLU_BF16><<<grid, 256, 0, s>>>(X, lda, Wp, W2, ldb, C, ldc, M, N, K, tiles_m, tiles_n);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Tile choice: fewest "tile-waves" over the 256 CUs, weighted by a per-shape
// efficiency factor (smaller tiles re-read more operand bytes per flop).
// The same rule serves grouped and per-tenant launches.
int gemm_pick_tile(int epi, int32_t M, int32_t N) {
  const int32_t NL = epi == EPI_GEGLU_BF16 ? 2 * N : N;
  struct Cand { int bn, bm; double eff; } cands[] = {{256, 256, 1.0}, {256, 128, 1.12}, {128, 128, 1.35}};
  int best = 0;
  double best_cost = 1e300;
  for (int c = 0; c < 3; ++c) {
    const int64_t tiles = (int64_t)((M + cands[c].bm - 1) / cands[c].bm) * ((NL + cands[c].bn - 1) / cands[c].bn);
    const double waves = (double)((tiles + 255) / 256);
    const double cost = waves * cands[c].bn * cands[c].bm * cands[c].eff;
    if (cost < best_cost * 0.999) {
      best_cost = cost;
      best = c;
    }
  }
  return best;
}

hipError_t launch_gemm(hipStream_t s, int epi, const void* A, int64_t lda, const void* B, const void* B2, int64_t ldb,
                       void* C, int64_t ldc, int32_t M, int32_t N, int32_t K, int tile_hint) {
  if (M <= 0 || N <= 0 || K <= 0 || K % kBK != 0 || N % 32 != 0) return hipErrorInvalidValue;
  const int t = tile_hint > 0 ? tile_hint - 1 : gemm_pick_tile(epi, M, N);
  switch (t) {
    case 0: return launch_tile<256, 256>(s, epi, A, lda, B, B2, ldb, C, ldc, M, N, K);
    case 1: return launch_tile<256, 128>(s, epi, A, lda, B, B2, ldb, C, ldc, M, N, K);
    default: return launch_tile<128, 128>(s, epi, A, lda, B, B2, ldb, C, ldc, M, N, K);
  }
}

}  // namespace jnx

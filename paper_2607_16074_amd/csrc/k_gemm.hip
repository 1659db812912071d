// bf16 GEMM for the backbone projections on gfx950 matrix cores.
//
//   C[M][N] (+)= epi( X[M][K] * W[N][K]^T )     X = activations, W = weights
//
// Tiling: a workgroup of WGN x WGM wavefronts owns a BN x BM tile (weight rows
// x tokens; 256x256 with 8 wavefronts for large launches); each wavefront
// accumulates (BN/WGN) x (BM/WGM) with v_mfma_f32_32x32x16_bf16.  The weight tile is the MFMA "A" operand, the
// token tile the "B" operand, so each lane ends with 4 consecutive output
// columns of one token row and the epilogue writes 8-byte (bf16) / 16-byte
// (fp32) vectors along the row-major output.
//
// Operand staging: global_load_lds_dwordx4 moves 16-byte chunks straight from
// global memory into LDS (no register staging).  K advances 64 per stage
// (one 128-byte segment of every operand row) through two stages, so one slab
// is in flight while the other is consumed.  Chunk c of LDS row r sits at
// position c ^ swz(r), swz(r) = (r >> 1) & 7: two 128-byte rows share a 256-byte
// bank row, and with this swizzle every 16-lane phase of a fragment read
// (rows lane & 31, chunk 2*step + (lane >> 5)) covers all 64 banks (derived
// from the bank-conflict counter's response to probe patterns; the GEMM runs
// conflict-free).  Each DMA instruction fills 1 KB = 8 rows; the lane ->
// source-chunk assignment applies the swizzle.  Per slab, four K=16 steps:
// the fragments of step s+1 are read under the MFMAs of step s; the next
// slab's DMA is interleaved with the first MFMAs; the one barrier per slab
// sits before the last step's MFMAs, which then cover the read of the next
// slab's first fragments.
//
// Launch order: tiles are walked in groups of 16 token-tiles (token tile
// fastest).  Workgroups are dealt round-robin to the 8 XCDs, so each XCD's
// resident tiles share a token tile and walk the weight tiles, and every
// weight slab is requested by all XCDs at about the same time.  Measured on
// the 2048-wide workloads, giving each XCD a contiguous block of tiles (an
// explicit XCD remap) is no faster with 4x8 blocks and 13% slower with 16x2.
//
// Epilogues: bf16 store, GELU -> bf16, fp32 residual add (in place), and
// GeGLU, whose gate and up weight rows are interleaved in 32-row blocks as
// they are loaded, so the gate and up accumulators of an output column land
// in the same lane.
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define JN_GPTR(p) ((__attribute__((address_space(1))) void*)(p))
#define JN_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int kBK = 64;       // K per stage (128-byte rows)
constexpr int kStages = 2;    // double buffer
constexpr int kGroupM = 16;   // token tiles per L2 group

__device__ __forceinline__ int lds_swz(int r) { return (r >> 1) & 7; }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// s_waitcnt with only the LDS / scalar-memory counter constrained.
template <int N>
__device__ __forceinline__ void wait_lgkmcnt() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (N << 8));
}

template <int T>
__device__ __forceinline__ void gemm_frags(bf16x8 (&f)[T], const uint16_t* stage, int row0, int pos) {
#pragma unroll
  for (int i = 0; i < T; ++i) f[i] = *reinterpret_cast<const bf16x8*>(stage + (row0 + i * 32) * kBK + pos * 8);
}

template <int TN, int TM>
__device__ __forceinline__ void gemm_mfma(f32x16 (&acc)[TN][TM], const bf16x8 (&fw)[TN], const bf16x8 (&fx)[TM]) {
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[i], fx[j], acc[i][j], 0, 0, 0);
}

template <int BN, int BM, int WGN, int WGM, int EPI>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int32_t pid, uint16_t* __restrict__ lds) {
  const uint16_t* __restrict__ X = g.X;
  const uint16_t* __restrict__ W = g.W;
  const uint16_t* __restrict__ W2 = g.W2;
  void* __restrict__ C = g.C;
  const int64_t ldx = g.ldx, ldw = g.ldw, ldc = g.ldc;
  const int32_t M = g.M, N = g.N, K = g.K, tiles_n = g.tiles_n, tiles_m = g.tiles_m;
  constexpr bool GLU = EPI == EPI_GEGLU_BF16;
  constexpr int NW = WGN * WGM;              // wavefronts
  constexpr int WN = BN / WGN, WM = BM / WGM;  // per-wave tile
  constexpr int TN = WN / 32, TM = WM / 32;
  constexpr int ROWS = BN + BM;              // weight rows then token rows in a stage
  constexpr int NI = ROWS / (8 * NW);        // 1 KB DMA instructions per wave per stage
  constexpr int STAGE = ROWS * kBK;          // elements per stage
  static_assert(ROWS % (8 * NW) == 0 && TN >= 1 && TM >= 1, "tile shape");
  static_assert(!GLU || TN % 2 == 0, "GeGLU pairs gate/up tiles inside a wave");

  // ---- grouped tile order
  const int32_t per_group = kGroupM * tiles_n;
  const int32_t group = pid / per_group;
  const int32_t first_m = group * kGroupM;
  const int32_t gsize = min(tiles_m - first_m, kGroupM);
  const int32_t tm = first_m + (pid % per_group) % gsize;
  const int32_t tn = (pid % per_group) / gsize;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wn = wave / WGM, wm = wave % WGM;

  // ---- DMA sources: this wave's instruction i fills stage rows 8*(wave*NI+i) ..
  // +7 (1 KB); lane -> (row lane>>3, position lane&7), and the position holds
  // logical chunk position ^ swz(row) of that row's 128-byte K segment.
  const int32_t NL = GLU ? 2 * N : N;
  const uint16_t* src[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int row = 8 * (wave * NI + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ lds_swz(row);
    if (row < BN) {
      if constexpr (GLU) {
        const int32_t col = min(tn * (BN / 2) + (row >> 6) * 32 + (row & 31), N - 1);
        src[i] = (((row >> 5) & 1) ? W2 : W) + (int64_t)col * ldw + chunk * 8;
      } else {
        src[i] = W + (int64_t)min(tn * BN + row, NL - 1) * ldw + chunk * 8;
      }
    } else {
      src[i] = X + (int64_t)min(tm * BM + row - BN, M - 1) * ldx + chunk * 8;
    }
  }
  uint16_t* const dst0 = lds + wave * NI * 512;  // 512 elements = 1 KB per instruction

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int KT = K / kBK;
  // fragment rows and their swizzle (row0 of every fragment is a multiple of 32)
  const int sw = lds_swz(lane & 31), half = lane >> 5;
  const int wrow = wn * WN + (lane & 31), xrow = BN + wm * WM + (lane & 31);

  // prologue: slabs 0 and 1 in flight
#pragma unroll
  for (int i = 0; i < NI; ++i)
    __builtin_amdgcn_global_load_lds(JN_GPTR(src[i]), JN_LPTR(dst0 + i * 512), 16, 0, 0);
  if (KT > 1) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
      __builtin_amdgcn_global_load_lds(JN_GPTR(src[i] + kBK), JN_LPTR(dst0 + STAGE + i * 512), 16, 0, 0);
    wait_vmcnt<NI>();
  } else {
    wait_vmcnt<0>();
  }
  __builtin_amdgcn_s_barrier();

  // Per slab: four K=16 steps; the fragments of step s+1 are read while the
  // MFMAs of step s run.  The DMA of slab kt+1 (into the buffer slab kt-1
  // used) is interleaved with the first MFMAs of slab kt.  The stage barrier
  // sits before the last step's MFMAs: each wave has waited for its slab kt+1
  // DMA and for its last reads of slab kt, meets the others, reads step 0 of
  // slab kt+1 and only then issues the last eight MFMAs of slab kt, which
  // cover that read.
  bf16x8 fw[2][TN], fx[2][TM];
  gemm_frags<TN>(fw[0], lds, wrow, half ^ sw);
  gemm_frags<TM>(fx[0], lds, xrow, half ^ sw);
  for (int kt = 0; kt < KT; ++kt) {
    const uint16_t* cur = lds + (kt & 1) * STAGE;
    const bool fill = kt >= 1 && kt + 1 < KT;  // slab kt+1 goes into the buffer slab kt-1 used
    uint16_t* const fdst = dst0 + ((kt + 1) & 1) * STAGE;
#pragma unroll
    for (int step = 0; step < 4; ++step) {
      const int b = step & 1;
      if (step < 3) {
        const int pos = (2 * (step + 1) + half) ^ sw;
        gemm_frags<TN>(fw[b ^ 1], cur, wrow, pos);
        gemm_frags<TM>(fx[b ^ 1], cur, xrow, pos);
      } else if (kt + 1 < KT) {
        wait_vmcnt<0>();
        wait_lgkmcnt<0>();
        __builtin_amdgcn_s_barrier();
        const uint16_t* nxt = lds + ((kt + 1) & 1) * STAGE;
        gemm_frags<TN>(fw[0], nxt, wrow, half ^ sw);
        gemm_frags<TM>(fx[0], nxt, xrow, half ^ sw);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < TN * TM; ++q) {
        const int i = q / TM, j = q % TM;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[b][i], fx[b][j], acc[i][j], 0, 0, 0);
        // DMA d of slab kt+1 after MFMA d of the slab (as early as possible)
        constexpr int PER = (NI + TN * TM - 1) / (TN * TM);  // DMAs per MFMA
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const int d = (step * TN * TM + q) * PER + e;
          if (d < NI && fill)
            __builtin_amdgcn_global_load_lds(JN_GPTR(src[d] + (kt + 1) * kBK), JN_LPTR(fdst + d * 512), 16, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
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
          for (int e = 0; e < 4; ++e) v[e] = gelu_fast_f(acc[i][j][rr * 4 + e]) * acc[i + 1][j][rr * 4 + e];
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
          } else if constexpr (EPI == EPI_F32) {
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(C) + (int64_t)m * ldc + n) =
                make_float4(v[0], v[1], v[2], v[3]);
          } else if constexpr (EPI == EPI_GELU_SAVE) {
            *reinterpret_cast<float4*>(g.aux + (int64_t)m * g.ldaux + n) = make_float4(v[0], v[1], v[2], v[3]);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = gelu_f(v[e]);
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
          } else if constexpr (EPI == EPI_GELUGRAD_BF16) {
            const float4 z = *reinterpret_cast<const float4*>(g.aux + (int64_t)m * g.ldaux + n);
            v[0] *= gelu_grad_f(z.x);
            v[1] *= gelu_grad_f(z.y);
            v[2] *= gelu_grad_f(z.z);
            v[3] *= gelu_grad_f(z.w);
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
          } else {
            if constexpr (EPI == EPI_GELU_BF16) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = gelu_fast_f(v[e]);
            }
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
          }
        }
      }
    }
  }
}

// Split-K: K range blockIdx.y of a launch whose g.K is the per-range length.
__device__ __forceinline__ GemmArgs split_range(const GemmArgs& g) {
  GemmArgs r = g;
  const int32_t s = blockIdx.y;
  if (s) {
    r.X += (int64_t)s * g.K;
    r.W += (int64_t)s * g.K;
    r.C = reinterpret_cast<float*>(g.C) + (int64_t)s * g.split_c;
  }
  return r;
}

template <int BN, int BM, int WGN, int WGM, int EPI>
__global__ __launch_bounds__(64 * WGN * WGM, 1) void gemm_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(1024))) uint16_t lds[kStages * (BN + BM) * kBK];
  gemm_tile<BN, BM, WGN, WGM, EPI>(split_range(g), blockIdx.x, lds);
}

// Sum of the split-K partials in range order, then the epilogue.  Thread =
// 4 consecutive output columns of one row.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int32_t S,
                                                            int64_t stride, int32_t M, int32_t N,
                                                            void* __restrict__ C, int64_t ldc) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int32_t q = N / 4;
  if (e >= (int64_t)M * q) return;
  const int32_t m = (int32_t)(e / q), n = (int32_t)(e % q) * 4;
  float4 acc = *reinterpret_cast<const float4*>(part + (int64_t)m * N + n);
  for (int32_t s = 1; s < S; ++s) {
    const float4 v = *reinterpret_cast<const float4*>(part + s * stride + (int64_t)m * N + n);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  if constexpr (EPI == EPI_RESID_F32) {
    float4* p = reinterpret_cast<float4*>(reinterpret_cast<float*>(C) + (int64_t)m * ldc + n);
    float4 o = *p;
    o.x += acc.x;
    o.y += acc.y;
    o.z += acc.z;
    o.w += acc.w;
    *p = o;
  } else {
    if constexpr (EPI == EPI_GELU_BF16) {
      acc.x = gelu_fast_f(acc.x);
      acc.y = gelu_fast_f(acc.y);
      acc.z = gelu_fast_f(acc.z);
      acc.w = gelu_fast_f(acc.w);
    }
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
        make_uint2(pack_bf2(acc.x, acc.y), pack_bf2(acc.z, acc.w));
  }
}

// One launch over several independent problems (one per tenant): block b
// runs tile b - tile_start[p] of the problem p whose tile range holds b.
template <int BN, int BM, int WGN, int WGM, int EPI>
__global__ __launch_bounds__(64 * WGN * WGM, 1) void gemm_grouped_kernel(const GemmArgs* __restrict__ probs,
                                                                         int32_t nprob) {
  __shared__ __attribute__((aligned(1024))) uint16_t lds[kStages * (BN + BM) * kBK];
  const int32_t b = blockIdx.x;
  int32_t p = 0;
  while (p + 1 < nprob && probs[p + 1].tile_start <= b) ++p;
  const GemmArgs g = probs[p];
  gemm_tile<BN, BM, WGN, WGM, EPI>(g, b - g.tile_start, lds);
}


// Ping-pong variant of the 256x256 tile (8 wavefronts), used for the plain
// bf16 and fp32-residual epilogues.  Waves w and w+4 share a SIMD; group 0
// (waves 0-3) and group 1 (waves 4-7) alternate between a memory phase (all
// 24 fragments of one K=64 slab from LDS, plus their share of a later slab's
// DMA) and a compute phase (the slab's 32 MFMAs, which only read registers),
// one workgroup barrier per phase, group 1 one phase behind group 0.  Slab
// kt+1 is fetched by group 0 during its memory phase of slab kt and by group
// 1 during its compute phase of slab kt-1; every wave waits for its own DMA
// before the barrier that precedes the first read of that slab.  Per output
// element the MFMA sequence (K order, operand lane layout) equals the
// non-ping-pong kernel's, so both produce identical bits.  Measured against
// the interleaved loop: +9.5% on the K=16384 residual projection, +4% on the
// K=2048 one, equal or slightly better elsewhere; the GeGLU projection is 4%
// slower with it and keeps the interleaved loop.
template <int EPI>
__global__ __launch_bounds__(512, 1) void gemm_pp_kernel(GemmArgs g) {
  constexpr int BN = 256, BM = 256, WGN = 2, WGM = 4;
  constexpr int NW = WGN * WGM;
  constexpr int WN = BN / WGN, WM = BM / WGM;
  constexpr int TN = WN / 32, TM = WM / 32;
  constexpr int ROWS = BN + BM;
  constexpr int NI = ROWS / (8 * NW);
  constexpr int STAGE = ROWS * kBK;
  static_assert(EPI == EPI_BF16 || EPI == EPI_RESID_F32, "ping-pong epilogues");
  __shared__ __attribute__((aligned(1024))) uint16_t lds[kStages * ROWS * kBK];
  const uint16_t* __restrict__ X = g.X;
  const uint16_t* __restrict__ W = g.W;
  void* __restrict__ C = g.C;
  const int64_t ldx = g.ldx, ldw = g.ldw, ldc = g.ldc;
  const int32_t M = g.M, N = g.N, K = g.K, tiles_n = g.tiles_n, tiles_m = g.tiles_m;
  const int32_t pid = blockIdx.x;

  const int32_t per_group = kGroupM * tiles_n;
  const int32_t group = pid / per_group;
  const int32_t first_m = group * kGroupM;
  const int32_t gsize = min(tiles_m - first_m, kGroupM);
  const int32_t tm = first_m + (pid % per_group) % gsize;
  const int32_t tn = (pid % per_group) / gsize;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wn = wave / WGM, wm = wave % WGM;
  const int grp = wave >> 2;

  const uint16_t* src[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int row = 8 * (wave * NI + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ lds_swz(row);
    if (row < BN)
      src[i] = W + (int64_t)min(tn * BN + row, N - 1) * ldw + chunk * 8;
    else
      src[i] = X + (int64_t)min(tm * BM + row - BN, M - 1) * ldx + chunk * 8;
  }
  uint16_t* const dst0 = lds + wave * NI * 512;

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int KT = K / kBK;
  const int sw = lds_swz(lane & 31), half = lane >> 5;
  const int wrow = wn * WN + (lane & 31), xrow = BN + wm * WM + (lane & 31);

  // slab 0 from every wave; group 1 also issues its share of slab 1 and then
  // waits one extra barrier, which puts it one phase behind group 0
#pragma unroll
  for (int i = 0; i < NI; ++i)
    __builtin_amdgcn_global_load_lds(JN_GPTR(src[i]), JN_LPTR(dst0 + i * 512), 16, 0, 0);
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  if (grp == 1) {
    if (KT > 1) {
#pragma unroll
      for (int i = 0; i < NI; ++i)
        __builtin_amdgcn_global_load_lds(JN_GPTR(src[i] + kBK), JN_LPTR(dst0 + STAGE + i * 512), 16, 0, 0);
    }
    __builtin_amdgcn_s_barrier();
  }

  bf16x8 fw[4][TN], fx[4][TM];
  for (int kt = 0; kt < KT; ++kt) {
    const uint16_t* cur = lds + (kt & 1) * STAGE;
    // ---- memory phase: slab kt's fragments (+ group 0's share of slab kt+1)
    __builtin_amdgcn_sched_barrier(0);
    if (grp == 0 && kt + 1 < KT) {
      uint16_t* const fdst = dst0 + ((kt + 1) & 1) * STAGE;
#pragma unroll
      for (int i = 0; i < NI; ++i)
        __builtin_amdgcn_global_load_lds(JN_GPTR(src[i] + (kt + 1) * kBK), JN_LPTR(fdst + i * 512), 16, 0, 0);
    }
#pragma unroll
    for (int step = 0; step < 4; ++step) {
      const int pos = (2 * step + half) ^ sw;
      gemm_frags<TN>(fw[step], cur, wrow, pos);
      gemm_frags<TM>(fx[step], cur, xrow, pos);
    }
    wait_lgkmcnt<0>();
    if (grp == 1) wait_vmcnt<0>();  // group 1's share of slab kt+1 (issued a phase earlier)
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // ---- compute phase: 32 MFMAs from registers (+ group 1's share of slab kt+2)
    const bool fill = grp == 1 && kt + 2 < KT;
    uint16_t* const gdst = dst0 + (kt & 1) * STAGE;
#pragma unroll
    for (int step = 0; step < 4; ++step) {
#pragma unroll
      for (int q = 0; q < TN * TM; ++q) {
        const int i = q / TM, j = q % TM;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[step][i], fx[step][j], acc[i][j], 0, 0, 0);
        const int d = step * TN * TM + q;
        if ((d & 3) == 3 && fill)
          __builtin_amdgcn_global_load_lds(JN_GPTR(src[d >> 2] + (kt + 2) * kBK), JN_LPTR(gdst + (d >> 2) * 512),
                                           16, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (grp == 0) wait_vmcnt<0>();  // group 0's share of slab kt+1
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  }
  if (grp == 0) __builtin_amdgcn_s_barrier();  // equal barrier counts in both groups

  const int hi4 = (lane >> 5) * 4;
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int32_t m = tm * BM + wm * WM + j * 32 + (lane & 31);
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int32_t n = tn * BN + wn * WN + i * 32 + rr * 8 + hi4;
        if (n >= N) continue;
        float a[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) a[e] = acc[i][j][rr * 4 + e];
        if constexpr (EPI == EPI_RESID_F32) {
          float4* p = reinterpret_cast<float4*>(reinterpret_cast<float*>(C) + (int64_t)m * ldc + n);
          float4 o = *p;
          o.x += a[0];
          o.y += a[1];
          o.z += a[2];
          o.w += a[3];
          *p = o;
        } else {
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
              make_uint2(pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]));
        }
      }
    }
  }
}

template <int BN, int BM, int WGN, int WGM>
static hipError_t launch_tile(hipStream_t s, int epi, GemmArgs g, int32_t splits = 1) {
  const int32_t NL = epi == EPI_GEGLU_BF16 ? 2 * g.N : g.N;
  g.tiles_m = (g.M + BM - 1) / BM;
  g.tiles_n = (NL + BN - 1) / BN;
  g.tile_start = 0;
  dim3 grid(g.tiles_m * g.tiles_n, splits), block(64 * WGN * WGM);
#define JN_GEMM_CASE(E) \
  case E: gemm_kernel<BN, BM, WGN, WGM, E><<<grid, block, 0, s>>>(g); break;
  switch (epi) {
    JN_GEMM_CASE(EPI_BF16)
    JN_GEMM_CASE(EPI_GELU_BF16)
    JN_GEMM_CASE(EPI_RESID_F32)
    JN_GEMM_CASE(EPI_GEGLU_BF16)
    JN_GEMM_CASE(EPI_F32)
    JN_GEMM_CASE(EPI_GELU_SAVE)
    JN_GEMM_CASE(EPI_GELUGRAD_BF16)
    default:
      return hipErrorInvalidValue;
  }
#undef JN_GEMM_CASE
  return hipGetLastError();
}

template <int BN, int BM, int WGN, int WGM>
static hipError_t launch_grouped_tile(hipStream_t s, int epi, const GemmArgs* dprobs, int32_t nprob,
                                      int32_t total_tiles) {
  dim3 grid(total_tiles), block(64 * WGN * WGM);
#define JN_GEMM_CASE(E) \
  case E: gemm_grouped_kernel<BN, BM, WGN, WGM, E><<<grid, block, 0, s>>>(dprobs, nprob); break;
  switch (epi) {
    JN_GEMM_CASE(EPI_BF16)
    JN_GEMM_CASE(EPI_RESID_F32)
    JN_GEMM_CASE(EPI_F32)
    JN_GEMM_CASE(EPI_GELU_SAVE)
    JN_GEMM_CASE(EPI_GELUGRAD_BF16)
    default:
      return hipErrorInvalidValue;
  }
#undef JN_GEMM_CASE
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

// Split-K: tile shape and K split S chosen together by an estimated time:
// waves of tiles * S over kSplitCUs, each a tile of 2 * BN * BM * K / S flops
// (times the shape factor) at the per-CU rate measured for this GEMM, plus
// the fp32 partials written and read back (2 * 4 * S * M * N bytes) at a
// sustained HBM rate.  Splits are considered only for launches of at most
// kSplitCUs / 2 tiles, with ranges of K / S >= 1024 (16 slabs) and S a power
// of two; S = 1 reproduces gemm_pick_tile's choice.  Fixed constants keep the
// size query and the launch in agreement on any device.
constexpr int32_t kSplitCUs = 256;
constexpr double kCuFlops = 4.3e12;    // ~1.1 PFLOP/s over 256 CUs
constexpr double kPartialBw = 5.0e12;  // bytes/s for the partial round trip

static void gemm_plan(int epi, int32_t M, int32_t N, int32_t K, int* tile, int* splits) {
  *tile = gemm_pick_tile(epi, M, N);
  *splits = 1;
  if (epi != EPI_BF16 && epi != EPI_RESID_F32 && epi != EPI_GELU_BF16) return;
  if (M <= 0 || N <= 0 || K <= 0 || N % 4 != 0) return;
  static const int bn[3] = {256, 256, 128}, bm[3] = {256, 128, 128};
  static const double eff[3] = {1.0, 1.12, 1.35};
  double best = 1e300;
  for (int t = 0; t < 3; ++t) {
    const int64_t tiles = (int64_t)((M + bm[t] - 1) / bm[t]) * ((N + bn[t] - 1) / bn[t]);
    for (int S = 1; S <= 64; S *= 2) {
      if (S > 1 && (tiles * 2 > kSplitCUs || K % (kBK * S) != 0 || K / S < 1024)) break;
      const double waves = (double)((tiles * S + kSplitCUs - 1) / kSplitCUs);
      double cost = waves * 2.0 * bn[t] * bm[t] * eff[t] * ((double)K / S) / kCuFlops;
      if (S > 1) cost += 8.0 * S * (double)M * N / kPartialBw;
      if (cost < best * 0.999) {
        best = cost;
        *tile = t;
        *splits = S;
      }
    }
  }
}

int gemm_split(int epi, int32_t M, int32_t N, int32_t K) {
  int t, S;
  gemm_plan(epi, M, N, K, &t, &S);
  return S;
}

size_t gemm_split_bytes(int epi, int32_t M, int32_t N, int32_t K) {
  const int S = gemm_split(epi, M, N, K);
  return S > 1 ? (size_t)S * M * N * sizeof(float) : 0;
}

hipError_t launch_gemm(hipStream_t s, int epi, const void* A, int64_t lda, const void* B, const void* B2, int64_t ldb,
                       void* C, int64_t ldc, int32_t M, int32_t N, int32_t K, int tile_hint, void* split_ws,
                       size_t split_bytes) {
  if (M <= 0 || N <= 0 || K <= 0 || K % kBK != 0 || N % 32 != 0) return hipErrorInvalidValue;
  int t_split = 0, S = 1;
  if (tile_hint <= 0) gemm_plan(epi, M, N, K, &t_split, &S);
  if (S > 1 && split_ws && split_bytes >= (size_t)S * M * N * sizeof(float)) {
    GemmArgs g{};
    g.X = reinterpret_cast<const uint16_t*>(A);
    g.W = reinterpret_cast<const uint16_t*>(B);
    g.C = split_ws;
    g.ldx = lda;
    g.ldw = ldb;
    g.ldc = N;
    g.M = M;
    g.N = N;
    g.K = K / S;
    g.split_c = (int64_t)M * N;
    hipError_t e;
    switch (t_split) {
      case 0: e = launch_tile<256, 256, 2, 4>(s, EPI_F32, g, S); break;
      case 1: e = launch_tile<256, 128, 4, 2>(s, EPI_F32, g, S); break;
      default: e = launch_tile<128, 128, 2, 2>(s, EPI_F32, g, S); break;
    }
    if (e != hipSuccess) return e;
    const int64_t work = (int64_t)M * (N / 4);
    const dim3 grid((unsigned)((work + 255) / 256));
    const float* part = reinterpret_cast<const float*>(split_ws);
    switch (epi) {
      case EPI_BF16: splitk_reduce_kernel<EPI_BF16><<<grid, 256, 0, s>>>(part, S, g.split_c, M, N, C, ldc); break;
      case EPI_RESID_F32:
        splitk_reduce_kernel<EPI_RESID_F32><<<grid, 256, 0, s>>>(part, S, g.split_c, M, N, C, ldc);
        break;
      default: splitk_reduce_kernel<EPI_GELU_BF16><<<grid, 256, 0, s>>>(part, S, g.split_c, M, N, C, ldc); break;
    }
    return hipGetLastError();
  }
  GemmArgs g{};
  g.X = reinterpret_cast<const uint16_t*>(A);
  g.W = reinterpret_cast<const uint16_t*>(B);
  g.W2 = reinterpret_cast<const uint16_t*>(B2);
  g.C = C;
  g.ldx = lda;
  g.ldw = ldb;
  g.ldc = ldc;
  g.M = M;
  g.N = N;
  g.K = K;
  const int t = tile_hint > 0 ? tile_hint - 1 : gemm_pick_tile(epi, M, N);
  switch (t) {
    case 0:
      if (epi == EPI_BF16 || epi == EPI_RESID_F32) {
        g.tiles_m = (g.M + 255) / 256;
        g.tiles_n = (g.N + 255) / 256;
        g.tile_start = 0;
        if (epi == EPI_BF16)
          gemm_pp_kernel<EPI_BF16><<<dim3(g.tiles_m * g.tiles_n), dim3(512), 0, s>>>(g);
        else
          gemm_pp_kernel<EPI_RESID_F32><<<dim3(g.tiles_m * g.tiles_n), dim3(512), 0, s>>>(g);
        return hipGetLastError();
      }
      return launch_tile<256, 256, 2, 4>(s, epi, g);
    case 1: return launch_tile<256, 128, 4, 2>(s, epi, g);
    default: return launch_tile<128, 128, 2, 2>(s, epi, g);
  }
}

int gemm_grouped_tile_shape(int32_t max_m) { return max_m >= 1024 ? 1 : 2; }

int32_t gemm_grouped_prepare(GemmArgs* probs, int32_t nprob, int shape) {
  const int BN = shape == 1 ? 256 : 128, BM = 128;
  int32_t total = 0;
  for (int32_t p = 0; p < nprob; ++p) {
    const GemmArgs& g = probs[p];
    if (g.M <= 0 || g.N <= 0 || g.K <= 0 || g.K % kBK != 0 || g.N % 32 != 0) return -1;
    probs[p].tiles_m = (probs[p].M + BM - 1) / BM;
    probs[p].tiles_n = (probs[p].N + BN - 1) / BN;
    probs[p].tile_start = total;
    total += probs[p].tiles_m * probs[p].tiles_n;
  }
  return total;
}

hipError_t launch_gemm_grouped(hipStream_t s, int epi, const GemmArgs* dprobs, int32_t nprob, int32_t total_tiles,
                               int shape) {
  if (nprob <= 0 || total_tiles <= 0) return hipErrorInvalidValue;
  if (shape == 1) return launch_grouped_tile<256, 128, 4, 2>(s, epi, dprobs, nprob, total_tiles);
  return launch_grouped_tile<128, 128, 2, 2>(s, epi, dprobs, nprob, total_tiles);
}

}  // namespace jnx

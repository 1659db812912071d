// bf16 GEMM for the backbone projections on gfx950 matrix cores.
//
//   C[M][N] (+)= epi( X[M][K] * W[N][K]^T )     X = activations, W = weights
//
// MFMA: v_mfma_f32_16x16x32_bf16.  The weight tile is the MFMA "A" operand
// and the token tile the "B" operand: lane l holds 8 consecutive K values of
// weight row l & 15 and of token row l & 15, K block 8 * (l >> 4), and ends
// with 4 consecutive output columns 4 * (l >> 4) .. +3 of token row l & 15,
// so the epilogue writes 8-byte (bf16) / 16-byte (fp32) vectors along the
// row-major output.  Measured on the 2048-wide shapes the 16x16x32 form runs
// 3-10% faster than 32x32x16 with the same operand traffic (the chip is
// power-limited and this form needs less energy per flop); a K=64 slab is two
// K=32 steps.  Every loop below issues, per output element, the same MFMA
// sequence (slab order, K=32 steps in order, the same lane layout), so all
// tile shapes and loops give identical bits.
//
// Operand staging: global_load_lds_dwordx4 moves 16-byte chunks straight from
// global memory into LDS (no register staging).  K advances 64 per slab (one
// 128-byte segment of every operand row).  Chunk c of LDS row r sits at
// position c ^ swz(r), swz(r) = (r >> 1) & 7: two 128-byte rows share a
// 256-byte bank row, and every 16-lane phase of a fragment read (16
// consecutive rows, one chunk) covers all 64 banks.  Each DMA instruction
// fills 1 KB = 8 rows; the lane -> source-chunk assignment applies the
// swizzle.
//
// Loops: the 256x256 tile (4 wavefronts, one per SIMD) runs a ring-buffered
// loop (gemm_ring_kernel, gemm_grouped_ring_kernel); the smaller tiles of
// short launches and of small grouped problems run an interleaved
// double-buffered loop (gemm_tile).
//
// Launch order: tiles are walked in groups of 32 token-tiles (token tile
// fastest).  Workgroups are dealt round-robin to the 8 XCDs, so the 32 tiles
// an XCD holds at a time form a block of 4 token tiles x 8 weight tiles, and
// every weight slab is requested by all XCDs at about the same time.
// Measured in the step on the 2048-wide workload: groups of 32 give 290.1 ms
// per step against 292.9 (16), 298.7 (8), 292.0 (64) and 300.6 (128); an
// explicit XCD remap giving each XCD a contiguous block of tiles was no
// faster with 4x8 blocks and 13% slower with 16x2 (32x32x16 loop).
//
// Epilogues: bf16 store, GELU -> bf16, fp32 residual add (in place), fp32
// store, GELU with fp32 pre-activation save, GELU' product, and GeGLU, whose
// gate and up weight rows are interleaved in 16-row blocks as they are
// loaded, so the gate and up accumulators of an output column land in the
// same lane.
#include <algorithm>

#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

#define JN_GPTR(p) ((__attribute__((address_space(1))) void*)(p))
#define JN_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int kBK = 64;       // K per slab (128-byte rows)
constexpr int kStages = 3;    // LDS stages of the interleaved loop (prefetch distance 2)
constexpr int kGroupM = 32;   // token tiles per L2 group

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

// T fragments of 16 rows each (rows row0, row0 + 16, ...), chunk position pos.
template <int T>
__device__ __forceinline__ void gemm_frags(bf16x8 (&f)[T], const uint16_t* stage, int row0, int pos) {
#pragma unroll
  for (int i = 0; i < T; ++i) f[i] = *reinterpret_cast<const bf16x8*>(stage + (row0 + i * 16) * kBK + pos * 8);
}

// Source row of weight-tile row r: plain, or for GeGLU the gate / up rows
// interleaved in 16-row blocks (block 2b = gate columns 16b.., 2b+1 = up).
template <bool GLU>
__device__ __forceinline__ const uint16_t* weight_row(const uint16_t* W, const uint16_t* W2, int64_t ldw, int32_t tn,
                                                      int BN, int r, int32_t N) {
  if constexpr (GLU) {
    const int32_t col = min(tn * (BN / 2) + (r >> 5) * 16 + (r & 15), N - 1);
    return (((r >> 4) & 1) ? W2 : W) + (int64_t)col * ldw;
  } else {
    return W + (int64_t)min(tn * BN + r, N - 1) * ldw;
  }
}

// Two floats -> two bf16 (round to nearest even) by one v_cvt_pk_bf16_f32;
// pack_bf2 converts each value alone and merges them with a shift and an
// OR.  Same bits.  Used in the GeGLU epilogue only: in the QKV kernel's staged
// epilogue the packed form changed the register allocation of the main loop
// (operand fragments moved through the accumulation registers, 16% slower).
typedef float gemm_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 gemm_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf2_cvt(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(gemm_f32x2{lo, hi}, gemm_bf16x2));
}

// Epilogue shared by the loops: accumulator block (i, j) covers weight rows
// 16 i .. of the wave's part and tokens 16 j ..; lane l owns output columns
// n .. n+3, n = 16 i + 4 (l >> 4), of token row 16 j + (l & 15).
template <int BN, int BM, int WGN, int WGM, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, const f32x4 (&acc)[BN / WGN / 16][BM / WGM / 16],
                                              int32_t tm, int32_t tn, int wn, int wm, int lane) {
  constexpr bool GLU = EPI == EPI_GEGLU_BF16;
  constexpr int WN = BN / WGN, WM = BM / WGM;
  constexpr int TN = WN / 16, TM = WM / 16;
  void* __restrict__ C = g.C;
  const int64_t ldc = g.ldc;
  const int32_t M = g.M, N = g.N;
  const int q4 = (lane >> 4) * 4;
  if constexpr (EPI == EPI_RESID_F32 || EPI == EPI_GELUGRAD_BF16) {
    // Read-modify epilogues: the fp32 operands (residual rows, or saved
    // pre-activations) of JB token-row blocks are all requested before the
    // first store of the batch, so a batch costs one memory round trip
    // instead of one per block.  Lanes outside the output read element (0, 0)
    // of the operand and store nothing.
    constexpr int JB = TM < 32 / TN ? TM : 32 / TN;
    static_assert(TM % JB == 0, "batch of token-row blocks");
    const float* src = EPI == EPI_RESID_F32 ? reinterpret_cast<const float*>(C) : g.aux;
    const int64_t ldr = EPI == EPI_RESID_F32 ? ldc : g.ldaux;
#pragma unroll
    for (int j0 = 0; j0 < TM; j0 += JB) {
      float4 r[JB][TN];
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const int32_t m = tm * BM + wm * WM + (j0 + jj) * 16 + (lane & 15);
        const int32_t mr = m < M ? m : 0;
#pragma unroll
        for (int i = 0; i < TN; ++i) {
          const int32_t n = tn * BN + wn * WN + i * 16 + q4;
          const int32_t nr = n < N ? n : 0;
          r[jj][i] = *reinterpret_cast<const float4*>(src + (int64_t)mr * ldr + nr);
        }
      }
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        const int32_t m = tm * BM + wm * WM + (j0 + jj) * 16 + (lane & 15);
        if (m >= M) continue;
#pragma unroll
        for (int i = 0; i < TN; ++i) {
          const int32_t n = tn * BN + wn * WN + i * 16 + q4;
          if (n >= N) continue;
          const f32x4 a = acc[i][j0 + jj];
          const float4 z = r[jj][i];
          if constexpr (EPI == EPI_RESID_F32) {
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(C) + (int64_t)m * ldc + n) =
                make_float4(z.x + a[0], z.y + a[1], z.z + a[2], z.w + a[3]);
          } else {
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
                make_uint2(pack_bf2(a[0] * gelu_grad_f(z.x), a[1] * gelu_grad_f(z.y)),
                           pack_bf2(a[2] * gelu_grad_f(z.z), a[3] * gelu_grad_f(z.w)));
          }
        }
      }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int32_t m = tm * BM + wm * WM + j * 16 + (lane & 15);
    if (m >= M) continue;
    if constexpr (GLU) {
#pragma unroll
      for (int i = 0; i < TN; i += 2) {
        const int32_t n = tn * (BN / 2) + wn * (WN / 2) + (i >> 1) * 16 + q4;
        if (n >= N) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = gelu_fast_f(acc[i][j][e]) * acc[i + 1][j][e];
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(C) + (int64_t)m * ldc + n) =
            make_uint2(pack_bf2_cvt(v[0], v[1]), pack_bf2_cvt(v[2], v[3]));
      }
    } else {
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int32_t n = tn * BN + wn * WN + i * 16 + q4;
        if (n >= N) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][e];
        if constexpr (EPI == EPI_F32) {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(C) + (int64_t)m * ldc + n) =
              make_float4(v[0], v[1], v[2], v[3]);
        } else if constexpr (EPI == EPI_GELU_SAVE) {
          *reinterpret_cast<float4*>(g.aux + (int64_t)m * g.ldaux + n) = make_float4(v[0], v[1], v[2], v[3]);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = gelu_f(v[e]);
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

// Position of tile pid in the grouped walk (kGroupM token tiles per group).
__device__ __forceinline__ void tile_of(int32_t pid, int32_t tiles_m, int32_t tiles_n, int32_t& tm, int32_t& tn) {
  const int32_t per_group = kGroupM * tiles_n;
  const int32_t first_m = (pid / per_group) * kGroupM;
  const int32_t gsize = min(tiles_m - first_m, kGroupM);
  tm = first_m + (pid % per_group) % gsize;
  tn = (pid % per_group) / gsize;
}

// Interleaved double-buffered loop (tiles of short and grouped launches).
// Per slab, two K=32 steps: the fragments of step 1 are read under the MFMAs
// of step 0; the next slab's DMA (into the buffer the previous slab used) is
// interleaved with the first MFMAs; the one barrier per slab sits before the
// second step's MFMAs, which then cover the read of the next slab's first
// fragments.
template <int BN, int BM, int WGN, int WGM, int EPI>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int32_t pid, uint16_t* __restrict__ lds) {
  const uint16_t* __restrict__ X = g.X;
  const int64_t ldx = g.ldx;
  const int32_t M = g.M, K = g.K;
  constexpr bool GLU = EPI == EPI_GEGLU_BF16;
  constexpr int NW = WGN * WGM;                // wavefronts
  constexpr int WN = BN / WGN, WM = BM / WGM;  // per-wave tile
  constexpr int TN = WN / 16, TM = WM / 16;
  constexpr int ROWS = BN + BM;                // weight rows then token rows in a stage
  constexpr int NI = ROWS / (8 * NW);          // 1 KB DMA instructions per wave per stage
  constexpr int STAGE = ROWS * kBK;            // elements per stage
  static_assert(ROWS % (8 * NW) == 0 && TN >= 1 && TM >= 1, "tile shape");
  static_assert(!GLU || TN % 2 == 0, "GeGLU pairs gate/up blocks inside a wave");

  int32_t tm, tn;
  tile_of(pid, g.tiles_m, g.tiles_n, tm, tn);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wn = wave / WGM, wm = wave % WGM;

  // ---- DMA sources: this wave's instruction i fills stage rows 8*(wave*NI+i)
  // .. +7 (1 KB); lane -> (row lane>>3, position lane&7), and the position
  // holds logical chunk position ^ swz(row) of that row's 128-byte K segment.
  const uint16_t* src[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int row = 8 * (wave * NI + i) + (lane >> 3);
    const int chunk = (lane & 7) ^ lds_swz(row);
    if (row < BN)
      src[i] = weight_row<GLU>(g.W, g.W2, g.ldw, tn, BN, row, g.N) + chunk * 8;
    else
      src[i] = X + (int64_t)min(tm * BM + row - BN, M - 1) * ldx + chunk * 8;
  }
  uint16_t* const dst0 = lds + wave * NI * 512;  // 512 elements = 1 KB per instruction

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = K / kBK;
  const int sw = lds_swz(lane & 15), quad = lane >> 4;
  const int wrow = wn * WN + (lane & 15), xrow = BN + wm * WM + (lane & 15);

  // prologue: slabs 0 .. kStages-2; slab kt+kStages-1 is fetched during slab
  // kt's first half into the stage slab kt-1 used
  static_assert(kStages == 3, "prefetch distance 2");
#pragma unroll
  for (int i = 0; i < NI; ++i)
    __builtin_amdgcn_global_load_lds(JN_GPTR(src[i]), JN_LPTR(dst0 + i * 512), 16, 0, 0);
  {
    const int s1 = min(1, KT - 1);
#pragma unroll
    for (int i = 0; i < NI; ++i)
      __builtin_amdgcn_global_load_lds(JN_GPTR(src[i] + s1 * kBK), JN_LPTR(dst0 + STAGE + i * 512), 16, 0, 0);
  }
  wait_vmcnt<NI>();  // slab 0 landed
  __builtin_amdgcn_s_barrier();

  // The loop body has no branches (each one in the MFMA stream costs tens of
  // cycles of issue): past the last slab the fetches repeat slab KT-1 into a
  // free stage, and the last next-slab fragment reads read a free stage.
  bf16x8 fw[2][TN], fx[2][TM];
  gemm_frags<TN>(fw[0], lds, wrow, quad ^ sw);
  gemm_frags<TM>(fx[0], lds, xrow, quad ^ sw);
  int st = 0;  // kt % 3
  for (int kt = 0; kt < KT; ++kt) {
    const int st1 = st == 2 ? 0 : st + 1, st2 = st == 0 ? 2 : st - 1;  // (kt + 1) % 3, (kt + 2) % 3
    const uint16_t* cur = lds + st * STAGE;
    const int sf = min(kt + 2, KT - 1);  // slab fetched into the stage slab kt-1 used
    uint16_t* const fdst = dst0 + st2 * STAGE;
#pragma unroll
    for (int step = 0; step < 2; ++step) {
      if (step == 0) {
        const int pos = (4 + quad) ^ sw;
        gemm_frags<TN>(fw[1], cur, wrow, pos);
        gemm_frags<TM>(fx[1], cur, xrow, pos);
      } else {
        wait_vmcnt<NI>();  // slab kt+1 landed; slab kt+2's fetch may stay in flight
        wait_lgkmcnt<0>();
        __builtin_amdgcn_s_barrier();
        const uint16_t* nxt = lds + st1 * STAGE;
        gemm_frags<TN>(fw[0], nxt, wrow, quad ^ sw);
        gemm_frags<TM>(fx[0], nxt, xrow, quad ^ sw);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < TN * TM; ++q) {
        const int i = q / TM, j = q % TM;
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[step][i], fx[step][j], acc[i][j], 0, 0, 0);
        // DMA d of slab kt+1 after MFMA d of the slab (as early as possible)
        constexpr int PER = (NI + TN * TM - 1) / (TN * TM);  // DMAs per MFMA
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const int d = (step * TN * TM + q) * PER + e;
          if (d < NI)
            __builtin_amdgcn_global_load_lds(JN_GPTR(src[d] + sf * kBK), JN_LPTR(fdst + d * 512), 16, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    st = st1;
  }
  wait_lgkmcnt<0>();
  wait_vmcnt<0>();  // the repeated slabs' DMAs land before the LDS is released
  // accumulators pinned to the accumulation registers (as in ring_tile)
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) asm volatile("" : "+a"(acc[i][j]));

  gemm_epilogue<BN, BM, WGN, WGM, EPI>(g, acc, tm, tn, wn, wm, lane);
}

// Split-K: K range s of a launch whose g.K is the per-range length.
__device__ __forceinline__ GemmArgs split_range(const GemmArgs& g, int32_t s) {
  GemmArgs r = g;
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
  gemm_tile<BN, BM, WGN, WGM, EPI>(split_range(g, blockIdx.y), blockIdx.x, lds);
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

// bf16 / GELU-bf16 epilogue of the 256x256 ring loop: the tile is staged
// through the (then free) LDS, row stride padded by 16 bytes (132 KB), so that
// global memory sees whole rows (16-byte lanes, 256 / NW rows per wave, 2 rows
// per instruction); written directly from the MFMA layout, each lane would
// touch 8 bytes of 16 different rows per instruction.  The caller has passed a
// barrier after the loop's last LDS access.  Wave w holds accumulator rows
// wm * 16 TM ...  The GeGLU tile (GELU-bound) and the fp32 residual add keep
// the direct path: with four waves the staged residual add (two 128-row halves,
// each read-add-write of C behind a barrier) measured 0.83 ms on the 2048x2048
// O projection against 0.75 direct, and 4.21 against 3.78 ms on the down
// projection.
template <int EPI, int TM, int NW>
__device__ __forceinline__ void ring_epilogue_bf16(const GemmArgs& g, const f32x4 (&acc)[8][TM], uint16_t* lds,
                                                   int32_t tm, int32_t tn, int wn, int wm, int wave, int lane) {
  constexpr int OS = 256 + 8;  // LDS row stride (elements)
  const int q4 = (lane >> 4) * 4;
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int row = wm * 16 * TM + j * 16 + (lane & 15);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = EPI == EPI_GELU_BF16 ? gelu_fast_f(acc[i][j][e]) : acc[i][j][e];
      *reinterpret_cast<uint2*>(lds + row * OS + wn * 128 + i * 16 + q4) =
          make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
    }
  }
  wait_lgkmcnt<0>();
  __builtin_amdgcn_s_barrier();
  const int c = lane & 31, rr = lane >> 5;  // 32 chunks of 16 bytes per row
  const int32_t n = tn * 256 + c * 8;
  constexpr int RW = 256 / NW;  // rows per wave
#pragma unroll
  for (int it = 0; it < RW / 2; ++it) {
    const int row = wave * RW + it * 2 + rr;
    const int32_t m = tm * 256 + row;
    const uint4 v = *reinterpret_cast<const uint4*>(lds + row * OS + c * 8);
    if (m < g.M && n < g.N) *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(g.C) + (int64_t)m * g.ldc + n) = v;
  }
}

// Buffer resource of a row-major bf16 panel starting at `base`, `bytes` long
// (loads past the end return zero).  Word 3 is the CDNA raw-buffer format.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t panel_rsrc(const uint16_t* base, int64_t bytes) {
  const int32_t n = (int32_t)min(bytes, (int64_t)0x7fffffff);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), (short)0, n, 0x00020000);
}

// Chunk position swizzle of k-line k of a transposed operand's half-slab
// (32 chunks of 16 bytes per line): the 16 k-lines one ds_read_b64_tr_b16
// touches (8 per half-wave, 2 chunks each) cover every LDS bank once per
// half-wave (checked with a bank model on the CPU).
__device__ __forceinline__ int tswz(int k) { return 2 * ((k & 3) | ((k & 8) >> 1)); }

// Ring-buffered loop of the 256x256 tile on 4 wavefronts, one per SIMD, each
// 128 weight rows x 128 tokens (64 accumulator blocks, kept in the
// accumulation registers).  Per K=64 slab kt, phase 0 runs the first k-half's
// 64 MFMAs while reading the second half's fragments and fetching the token
// half of slab kt+2; every wave then waits for its own DMA of slab kt+1 and a
// workgroup barrier; phase 1 runs the second half's MFMAs while reading slab
// kt+1's first-half fragments and fetching the weight half of slab kt+2.  The
// LDS holds two weight slots and three token slots (5 x 32 KB = 160 KB): a
// slot is refilled only after the barrier that follows its last fragment
// read.  The stream has no branches: past the last slab the DMAs repeat slab
// KT-1 into free slots and the fragment reads read a free slot, so every
// phase issues the same instructions; each DMA is one buffer load to LDS with
// a per-lane 32-bit offset and the slab offset in a scalar register.
// Measured on the 2048-wide shapes against the 8-wave ping-pong loop it
// replaces (two waves per SIMD alternating memory and compute phases): GeGLU
// 8.27 -> 7.36 ms, QKV 1.63 -> 1.50 ms.  Per-phase cycle stamps showed what
// the 8-wave loop and the first 4-wave versions lost: each conditional branch
// in the MFMA stream cost 30-50 cycles of issue, and global_load_lds with a
// 64-bit address computed per instruction cost more than the buffer form.
// Tile pid of problem g; lds holds 5 x 32 KB.
//
// TR: operands stored transposed (GEMM_TRANS_X: X is [K][M], element (m, k)
// at X[k * ldx + m]; GEMM_TRANS_W: W is [K][N]).  A transposed operand's
// half-slab is 64 k-lines of 256 rows (512 B per line, 2 lines per DMA
// instruction), its 16-byte chunks at position chunk ^ tswz(k); a fragment
// is two ds_read_b64_tr_b16 (k-slots 0..3 and 4..7 of the lane's k block), so
// the MFMA sequence per output element is the one of the row-major layout.
// Loads past line K of a transposed operand return zero (buffer range), so
// with both operands transposed K need not be a multiple of 64.
template <int EPI, int TR>
__device__ __forceinline__ void ring_tile(const GemmArgs& g, int32_t pid, uint16_t* __restrict__ lds) {
  constexpr bool TX = (TR & GEMM_TRANS_X) != 0, TW = (TR & GEMM_TRANS_W) != 0;
  constexpr int BN = 256, BM = 256, WGN = 2, WGM = 2;
  constexpr int WN = BN / WGN, WM = BM / WGM;
  constexpr int TN = WN / 16, TM = WM / 16;
  constexpr int NI = 8;            // 1 KB DMA instructions per wave per half-slab
  constexpr int SLOT = 256 * kBK;  // elements per half-slab slot
  constexpr bool GLU = EPI == EPI_GEGLU_BF16;
  const int32_t M = g.M, K = g.K;

  int32_t tm, tn;
  tile_of(pid, g.tiles_m, g.tiles_n, tm, tn);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wn = wave / WGM, wm = wave % WGM;

  // panels of this tile: token rows tm*256.., weight rows (GeGLU: gate and up
  // columns tn*128..) -- rows past the end are clamped to the last one
  const int32_t m0 = tm * BM;
  const int32_t c0 = GLU ? tn * (BN / 2) : tn * BN;
  static_assert(!(GLU && TW), "GeGLU weights are row-major");
  const uint16_t* const xb = TX ? g.X + m0 : g.X + (int64_t)m0 * g.ldx;
  const uint16_t* const wb = TW ? g.W + c0 : g.W + (int64_t)c0 * g.ldw;
  const uint16_t* const wb2 = GLU ? g.W2 + (int64_t)c0 * g.ldw : wb;
  const __amdgpu_buffer_rsrc_t xr =
      panel_rsrc(xb, TX ? ((int64_t)K * g.ldx - m0) * 2 : (int64_t)(M - m0) * g.ldx * 2);
  const __amdgpu_buffer_rsrc_t wr =
      panel_rsrc(wb, TW ? ((int64_t)K * g.ldw - c0) * 2 : (int64_t)(g.N - c0) * g.ldw * 2);
  const __amdgpu_buffer_rsrc_t wr2 = panel_rsrc(wb2, (int64_t)(g.N - c0) * g.ldw * 2);
  // row-major operand: wave w fetches rows 64w .. 64w+63 of the half-slab, 8
  // rows per instruction; transposed: k-lines 16w .. 16w+15, 2 per instruction
  uint32_t xo[NI], wo[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int r = 64 * wave + 8 * i + (lane >> 3);
    const int chunk = (lane & 7) ^ lds_swz(r);
    const int kl = 16 * wave + 2 * i + (lane >> 5);
    const int tchunk = (lane & 31) ^ tswz(kl);
    if constexpr (TX)
      xo[i] = (uint32_t)(((int64_t)kl * g.ldx + tchunk * 8) * 2);
    else
      xo[i] = (uint32_t)(((int64_t)(min(m0 + r, M - 1) - m0) * g.ldx + chunk * 8) * 2);
    if constexpr (TW) {
      wo[i] = (uint32_t)(((int64_t)kl * g.ldw + tchunk * 8) * 2);
    } else {
      const int32_t col = GLU ? min(c0 + (r >> 5) * 16 + (r & 15), g.N - 1) : min(c0 + r, g.N - 1);
      wo[i] = (uint32_t)(((int64_t)(col - c0) * g.ldw + chunk * 8) * 2);
    }
  }
  // byte step between slabs: one 128-byte row segment (in the scalar offset),
  // or 64 k-lines of a transposed operand (in the lane offset, which the
  // buffer range check covers, so lines past K read zero)
  const int32_t xso = TX ? (int32_t)(kBK * 2 * g.ldx) : kBK * 2;
  const int32_t wso = TW ? (int32_t)(kBK * 2 * g.ldw) : kBK * 2;
  const int dro = wave * NI * 512;         // this wave's 1 KB blocks inside a slot
  uint16_t* const ring2 = lds;             // weight slabs, slot kt % 2
  uint16_t* const ring3 = lds + 2 * SLOT;  // token slabs, slot kt % 3
  // DMA i of slab `slab` into a slot; in GeGLU tiles, instruction i covers
  // weight rows of one 16-row block, all gate (W) or all up (W2)
#define JN_DMA_W(i, slab, slot)                                                                                  \
  __builtin_amdgcn_raw_ptr_buffer_load_lds((GLU && (((i) >> 1) & 1)) ? wr2 : wr,                                \
                                           JN_LPTR(ring2 + (slot) * SLOT + dro + (i) * 512), 16,                \
                                           TW ? wo[i] + (uint32_t)((slab) * wso) : wo[i], TW ? 0 : (slab) * wso, 0, 0)
#define JN_DMA_X(i, slab, slot)                                                                                  \
  __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, JN_LPTR(ring3 + (slot) * SLOT + dro + (i) * 512), 16,            \
                                           TX ? xo[i] + (uint32_t)((slab) * xso) : xo[i], TX ? 0 : (slab) * xso, 0, \
                                           0)

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = (K + kBK - 1) / kBK;
  const int sw = lds_swz(lane & 15), quad = lane >> 4;
  const int wrow = wn * WN + (lane & 15), xrow = wm * WM + (lane & 15);
  // transposed reads (inline assembly, covered by the loop's LDS waits at
  // every phase boundary): lane (quad, e = (lane & 15) / 4, c = lane & 3) reads k-line
  // 8 quad + e (+4) at rows rbase + 4c; tr_base(part) | 16 ts, XORed with 16 f
  // per fragment f, addresses the swizzled chunk (bits 4-6 are free below)
  const int te = (lane & 15) >> 2, tc = lane & 3;
  const int tlane = (8 * quad + te) * 256 + 8 * (tc >> 1) + 4 * (tc & 1) + 16 * ((te & 3) | ((quad & 1) << 2));
  const int twl = tlane + 128 * wn, txl = tlane + 128 * wm;
  // fragment f (16 rows) of k-half h of a half-slab slot
  auto frag_w = [&](const uint16_t* slot, int f, int h) -> bf16x8 {
    if constexpr (TW) {
      const uint16_t* p = slot + 8192 * h + (twl ^ (16 * f));
      const bf16x4 lo = __builtin_bit_cast(bf16x4, lds_read_tr_b16<0>(p));
      const bf16x4 hi = __builtin_bit_cast(bf16x4, lds_read_tr_b16<2048>(p));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    } else {
      return *reinterpret_cast<const bf16x8*>(slot + (wrow + 16 * f) * kBK + ((4 * h + quad) ^ sw) * 8);
    }
  };
  auto frag_x = [&](const uint16_t* slot, int f, int h) -> bf16x8 {
    if constexpr (TX) {
      const uint16_t* p = slot + 8192 * h + (txl ^ (16 * f));
      const bf16x4 lo = __builtin_bit_cast(bf16x4, lds_read_tr_b16<0>(p));
      const bf16x4 hi = __builtin_bit_cast(bf16x4, lds_read_tr_b16<2048>(p));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    } else {
      return *reinterpret_cast<const bf16x8*>(slot + (xrow + 16 * f) * kBK + ((4 * h + quad) ^ sw) * 8);
    }
  };

  // prologue: slabs 0 and 1 (both halves), then slab 0's first-half fragments
  {
    const int s1 = min(1, KT - 1);
#pragma unroll
    for (int i = 0; i < NI; ++i) JN_DMA_W(i, 0, 0);
#pragma unroll
    for (int i = 0; i < NI; ++i) JN_DMA_X(i, 0, 0);
#pragma unroll
    for (int i = 0; i < NI; ++i) JN_DMA_X(i, s1, 1);
#pragma unroll
    for (int i = 0; i < NI; ++i) JN_DMA_W(i, s1, 1);
    wait_vmcnt<2 * NI>();
  }
  __builtin_amdgcn_s_barrier();
  bf16x8 fa[TN + TM], fb[TN + TM];  // first-half / second-half fragments: weights, then tokens
#pragma unroll
  for (int i = 0; i < TN; ++i) fa[i] = frag_w(ring2, i, 0);
#pragma unroll
  for (int j = 0; j < TM; ++j) fa[TN + j] = frag_x(ring3, j, 0);
  wait_lgkmcnt<0>();

  int slot3 = 0;  // kt % 3
  for (int kt = 0; kt < KT; ++kt) {
    const int slot2 = kt & 1;
    const int next3 = slot3 == 2 ? 0 : slot3 + 1;   // (kt + 1) % 3
    const int prev3 = slot3 == 0 ? 2 : slot3 - 1;   // (kt + 2) % 3
    const int sf = min(kt + 2, KT - 1);             // slab fetched this iteration
    // ---- phase 0: first k-half MFMAs; second-half fragments; token DMA of slab kt+2
    {
      const uint16_t* cw = ring2 + slot2 * SLOT;
      const uint16_t* cx = ring3 + slot3 * SLOT;
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < TN * TM; ++q) {
        const int i = q / TM, j = q % TM;
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fa[TN + j], acc[i][j], 0, 0, 0);
        if ((q & 3) == 0) {
          const int f = q >> 2;
          if (f < TN)
            fb[f] = frag_w(cw, f, 1);
          else
            fb[f] = frag_x(cx, f - TN, 1);
        }
        if ((q & 7) == 6) JN_DMA_X(q >> 3, sf, prev3);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // slab kt+1 landed (the token DMA of slab kt+2, issued last, may stay in flight)
    wait_lgkmcnt<0>();
    wait_vmcnt<NI>();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // ---- phase 1: second k-half MFMAs; slab kt+1's first-half fragments; weight DMA of slab kt+2
    {
      const uint16_t* nw = ring2 + (slot2 ^ 1) * SLOT;
      const uint16_t* nx = ring3 + next3 * SLOT;
#pragma unroll
      for (int q = 0; q < TN * TM; ++q) {
        const int i = q / TM, j = q % TM;
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[i], fb[TN + j], acc[i][j], 0, 0, 0);
        if ((q & 3) == 0) {
          const int f = q >> 2;
          if (f < TN)
            fa[f] = frag_w(nw, f, 0);
          else
            fa[f] = frag_x(nx, f - TN, 0);
        }
        if ((q & 7) == 6) JN_DMA_W(q >> 3, sf, slot2);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    wait_lgkmcnt<0>();
    slot3 = next3;
  }
#undef JN_DMA_W
#undef JN_DMA_X
  wait_vmcnt<0>();  // the repeated slabs' DMAs land before the LDS is reused or released
  // Pin the accumulators to the accumulation registers where the loop ends.
  // Left to itself, the register allocator placed some accumulators of the
  // epilogues that can store straight from either register file (fp32 store,
  // fp32 pre-activation save) in vector registers and copied them into
  // accumulation registers before every MFMA of the loop (with spills to
  // scratch in the grouped variants).
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) asm volatile("" : "+a"(acc[i][j]));

  if constexpr (EPI == EPI_BF16 || EPI == EPI_GELU_BF16) {
    __builtin_amdgcn_s_barrier();
    ring_epilogue_bf16<EPI, TM, 4>(g, acc, lds, tm, tn, wn, wm, wave, lane);
  } else {
    gemm_epilogue<BN, BM, WGN, WGM, EPI>(g, acc, tm, tn, wn, wm, lane);
  }
}

// One launch of ring tiles over g (split-K ranges from blockIdx.y as in
// gemm_kernel).  With g.xcd_ranges (S = gridDim.y ranges, S | 8, at most
// kGroupM token tiles, 8 / S | tiles_n) workgroup b + gridDim.x y, which the
// hardware places on XCD x = (b + gridDim.x y) % 8, takes K range
// x / (8 / S) and, of that range, the tiles of one block of tiles_n / (8 / S)
// weight tiles over all token tiles.  In the grouped walk every XCD held one
// token tile over all K ranges and all weight tiles, so each of the 8 L2s
// fetched the whole weight matrix; now an XCD fetches one range's token rows
// and a 1/(8/S) share of that range's weight columns.  Which workgroup
// computes a (range, tile) changes nothing else.
template <int EPI>
__global__ __launch_bounds__(256, 1) void gemm_ring_kernel(GemmArgs g0) {
  __shared__ __attribute__((aligned(1024))) uint16_t lds[5 * 256 * kBK];
  int32_t pid = blockIdx.x, s = blockIdx.y;
  if (g0.xcd_ranges) {
    const int32_t lin = blockIdx.x + blockIdx.y * gridDim.x;
    const int32_t x = lin & 7, slot = lin >> 3, nx = 8 / gridDim.y;
    s = x / nx;
    const int32_t tm = slot % g0.tiles_m;
    const int32_t tn = (x % nx) * (g0.tiles_n / nx) + slot / g0.tiles_m;
    pid = tn * g0.tiles_m + tm;  // tile_of's inverse for tiles_m <= kGroupM
  }
  ring_tile<EPI, 0>(split_range(g0, s), pid, lds);
}

// Grouped ring tiles: problem p owns tiles [tile_start, tile_start + tiles).
template <int EPI, int TR>
__global__ __launch_bounds__(256, 1) void gemm_grouped_ring_kernel(const GemmArgs* __restrict__ probs, int32_t nprob) {
  __shared__ __attribute__((aligned(1024))) uint16_t lds[5 * 256 * kBK];
  const int32_t b = blockIdx.x;
  int32_t p = 0;
  while (p + 1 < nprob && probs[p + 1].tile_start <= b) ++p;
  const GemmArgs g = probs[p];
  ring_tile<EPI, TR>(g, b - g.tile_start, lds);
}

template <int BN, int BM, int WGN, int WGM>
static hipError_t launch_tile(hipStream_t s, int epi, GemmArgs g, int32_t splits = 1);

// The 256x256 ring loop over all tiles of g (grid.y = split-K ranges).  Its
// per-lane panel offsets are 32-bit: leading dimensions beyond 4M elements
// take the 256x128 loop (same MFMA sequence per output element).
static hipError_t launch_ring(hipStream_t s, int epi, GemmArgs g, int32_t splits = 1) {
  if ((int64_t)256 * std::max(g.ldx, g.ldw) * 2 > (int64_t)0x7fffffff)
    return launch_tile<256, 128, 4, 2>(s, epi, g, splits);
  const int32_t NL = epi == EPI_GEGLU_BF16 ? 2 * g.N : g.N;
  g.tiles_m = (g.M + 255) / 256;
  g.tiles_n = (NL + 255) / 256;
  g.tile_start = 0;
  g.xcd_ranges = splits > 1 && 8 % splits == 0 && g.tiles_m <= kGroupM && g.tiles_n % (8 / splits) == 0;
  const dim3 grid(g.tiles_m * g.tiles_n, splits), block(256);
  switch (epi) {
    case EPI_BF16: gemm_ring_kernel<EPI_BF16><<<grid, block, 0, s>>>(g); break;
    case EPI_GELU_BF16: gemm_ring_kernel<EPI_GELU_BF16><<<grid, block, 0, s>>>(g); break;
    case EPI_RESID_F32: gemm_ring_kernel<EPI_RESID_F32><<<grid, block, 0, s>>>(g); break;
    case EPI_GEGLU_BF16: gemm_ring_kernel<EPI_GEGLU_BF16><<<grid, block, 0, s>>>(g); break;
    case EPI_F32: gemm_ring_kernel<EPI_F32><<<grid, block, 0, s>>>(g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int BN, int BM, int WGN, int WGM>
static hipError_t launch_tile(hipStream_t s, int epi, GemmArgs g, int32_t splits) {
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

static hipError_t launch_grouped_ring(hipStream_t s, int epi, const GemmArgs* dprobs, int32_t nprob,
                                      int32_t total_tiles, int trans) {
  dim3 grid(total_tiles), block(256);
#define JN_GEMM_CASE(E, T) \
  case E * 4 + T: gemm_grouped_ring_kernel<E, T><<<grid, block, 0, s>>>(dprobs, nprob); break;
  switch (epi * 4 + trans) {
    JN_GEMM_CASE(EPI_BF16, 0)
    JN_GEMM_CASE(EPI_RESID_F32, 0)
    JN_GEMM_CASE(EPI_F32, 0)
    JN_GEMM_CASE(EPI_GELU_SAVE, 0)
    JN_GEMM_CASE(EPI_GELUGRAD_BF16, 0)
    JN_GEMM_CASE(EPI_F32, GEMM_TRANS_W)
    JN_GEMM_CASE(EPI_GELUGRAD_BF16, GEMM_TRANS_W)
    JN_GEMM_CASE(EPI_F32, GEMM_TRANS_X | GEMM_TRANS_W)
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

static int32_t gemm_tail_split(int epi, int32_t M, int32_t N, int32_t K, int32_t* m1, int* t1, int* t2);

size_t gemm_split_bytes(int epi, int32_t M, int32_t N, int32_t K) {
  const int S = gemm_split(epi, M, N, K);
  size_t bytes = S > 1 ? (size_t)S * M * N * sizeof(float) : 0;
  int32_t m1;
  int t1, t2;
  const int32_t St = gemm_tail_split(epi, M, N, K, &m1, &t1, &t2);
  if (St > 1) bytes = std::max(bytes, (size_t)St * (M - m1) * N * sizeof(float));
  return bytes;
}

// One launch over all rows of g with tile shape t (0: 256x256 ring loop,
// 1: 256x128, 2: 128x128).
static hipError_t launch_rows(hipStream_t s, int epi, GemmArgs g, int t) {
  switch (t) {
    case 0: return launch_ring(s, epi, g);
    case 1: return launch_tile<256, 128, 4, 2>(s, epi, g);
    default: return launch_tile<128, 128, 2, 2>(s, epi, g);
  }
}

// Split-K: S launches' worth of K ranges as one grid (blockIdx.y = range),
// fp32 partials into split_ws, then their sum in range order with the
// epilogue (EPI_BF16, EPI_RESID_F32 or EPI_GELU_BF16).
static hipError_t launch_split(hipStream_t s, int epi, const void* A, int64_t lda, const void* B, int64_t ldb,
                               void* C, int64_t ldc, int32_t M, int32_t N, int32_t K, int t, int32_t S,
                               void* split_ws) {
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
  switch (t) {
    case 0: e = launch_ring(s, EPI_F32, g, S); break;
    case 1: e = launch_tile<256, 128, 4, 2>(s, EPI_F32, g, S); break;
    default: e = launch_tile<128, 128, 2, 2>(s, EPI_F32, g, S); break;
  }
  if (e != hipSuccess) return e;
  const int64_t work = (int64_t)M * (N / 4);
  const dim3 grid((unsigned)((work + 255) / 256));
  const float* part = reinterpret_cast<const float*>(split_ws);
  switch (epi) {
    case EPI_BF16: splitk_reduce_kernel<EPI_BF16><<<grid, 256, 0, s>>>(part, S, g.split_c, M, N, C, ldc); break;
    case EPI_RESID_F32: splitk_reduce_kernel<EPI_RESID_F32><<<grid, 256, 0, s>>>(part, S, g.split_c, M, N, C, ldc); break;
    case EPI_GELU_BF16: splitk_reduce_kernel<EPI_GELU_BF16><<<grid, 256, 0, s>>>(part, S, g.split_c, M, N, C, ldc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Row split against the last, partly filled wave of tiles: rows [0, m1) run
// as 256x256 ring tiles and rows [m1, M) as a second launch with a smaller
// shape t2, chosen by the same time estimate as gemm_plan (tile-waves over
// the 256 CUs, per-shape efficiency) plus the gap between two launches.  For
// example 2,368 tiles of 256x256 (9.25 waves) become 9 full waves plus one
// wave of 128x128 tiles.  Measured: the K=16384 down projection 2.3% faster
// at 75.5K tokens and 7.5% at 9.4K, the O projection 13% at 9.4K, GeGLU 3.6%
// at 4.7K; the leading part stays on the ring loop because the smaller tiles'
// loop is much slower per flop than the estimate assumes (a 256x128 +
// 128x128 plan of the down projection at 4.7K tokens took 0.56 ms against
// 0.39 ms for one partial wave of 256x256 tiles).  Every tile shape runs the
// same MFMA sequence per output element, so the split does not change any bit.
constexpr double kLaunchGap = 6e-6;  // seconds between two launches on one stream

static void gemm_plan_rows(int epi, int32_t M, int32_t N, int32_t K, int* t1, int32_t* m1, int* t2) {
  const int32_t NL = epi == EPI_GEGLU_BF16 ? 2 * N : N;
  static const int bn[3] = {256, 256, 128}, bm[3] = {256, 128, 128};
  static const double eff[3] = {1.0, 1.12, 1.35};
  auto cost_of = [&](int t, int32_t rows) {
    const int64_t tiles = (int64_t)((rows + bm[t] - 1) / bm[t]) * ((NL + bn[t] - 1) / bn[t]);
    const double waves = (double)((tiles + kSplitCUs - 1) / kSplitCUs);
    return waves * 2.0 * bn[t] * bm[t] * eff[t] * (double)K / kCuFlops;
  };
  *t1 = gemm_pick_tile(epi, M, N);
  *m1 = M;
  *t2 = *t1;
  double best = cost_of(*t1, M);
  const int32_t tma = (M + 255) / 256;
  for (int32_t r = tma - 1; r >= 1 && r >= tma - 64; --r) {
    const int32_t ma = r * 256;
    for (int b = 1; b < 3; ++b) {
      const double cost = cost_of(0, ma) + cost_of(b, M - ma) + kLaunchGap;
      if (cost < best * 0.98) {
        best = cost;
        *t1 = 0;
        *m1 = ma;
        *t2 = b;
      }
    }
  }
}

// The row-split tail of a long contraction runs split over K on 256x256 ring
// tiles.  A tail of at most 128 ring tiles on 128x128 tiles keeps the matrix
// cores ~18% busy (each such tile moves twice the operand bytes per flop of a
// ring tile; measured on the K=16384 down projection of the 2B-shaped
// backbone, 1,801 rows: ~0.3 ms per launch), against ~60% on ring tiles; split
// S ways (the largest power of two with tiles * S <= kSplitCUs, K/S >= 1024
// and K % (64 S) == 0) the tail fills one wave of ring tiles and a reduction
// adds the S fp32 partials in range order.  Only for K >= kTailSplitK: there
// the 128x128 tail costs more than a tenth of the launch.  A tail row summed
// in K ranges differs in the last bits from the same row computed in one
// pass (in another batch it may not lie in a tail), so for such launches
// grouped and isolated runs agree to rounding instead of bitwise.  Returns S
// (1: no split) with the row plan of gemm_plan_rows.
constexpr int32_t kTailSplitK = 8192;

static int32_t gemm_tail_split(int epi, int32_t M, int32_t N, int32_t K, int32_t* m1, int* t1, int* t2) {
  gemm_plan_rows(epi, M, N, K, t1, m1, t2);
  if (*m1 >= M || *m1 <= 0 || K < kTailSplitK) return 1;
  if (epi != EPI_BF16 && epi != EPI_RESID_F32 && epi != EPI_GELU_BF16) return 1;
  if (N % 4 != 0) return 1;
  const int64_t tiles = (int64_t)((M - *m1 + 255) / 256) * ((N + 255) / 256);
  int32_t S = 1;
  while (S < 16 && tiles * (2 * S) <= kSplitCUs && K % (kBK * 2 * S) == 0 && K / (2 * S) >= 1024) S *= 2;
  return S;
}

hipError_t launch_gemm(hipStream_t s, int epi, const void* A, int64_t lda, const void* B, const void* B2, int64_t ldb,
                       void* C, int64_t ldc, int32_t M, int32_t N, int32_t K, int tile_hint, void* split_ws,
                       size_t split_bytes) {
  if (M <= 0 || N <= 0 || K <= 0 || K % kBK != 0 || N % 32 != 0) return hipErrorInvalidValue;
  int t_split = 0, S = 1;
  if (tile_hint <= 0) gemm_plan(epi, M, N, K, &t_split, &S);
  if (S > 1 && split_ws && split_bytes >= (size_t)S * M * N * sizeof(float))
    return launch_split(s, epi, A, lda, B, ldb, C, ldc, M, N, K, t_split, S, split_ws);
  GemmArgs g{};
  g.X = reinterpret_cast<const uint16_t*>(A);
  g.W = reinterpret_cast<const uint16_t*>(B);
  g.W2 = reinterpret_cast<const uint16_t*>(B2);
  g.C = C;
  g.ldx = lda;
  g.ldw = ldb;
  g.ldc = ldc;
  g.N = N;
  g.K = K;
  if (tile_hint > 0) {
    g.M = M;
    return launch_rows(s, epi, g, tile_hint - 1);
  }
  int t1, t2;
  int32_t m1;
  const int32_t St = gemm_tail_split(epi, M, N, K, &m1, &t1, &t2);
  if (m1 > 0) {
    g.M = m1;
    const hipError_t e = launch_rows(s, epi, g, t1);
    if (e != hipSuccess || m1 == M) return e;
  }
  const size_t esize = (epi == EPI_RESID_F32 || epi == EPI_F32) ? 4 : 2;
  void* Ct = static_cast<char*>(C) + (size_t)m1 * ldc * esize;
  const void* At = reinterpret_cast<const uint16_t*>(A) + (int64_t)m1 * lda;
  if (St > 1 && split_ws && split_bytes >= (size_t)St * (M - m1) * N * sizeof(float))
    return launch_split(s, epi, At, lda, B, ldb, Ct, ldc, M - m1, N, K, 0, St, split_ws);
  g.X += (int64_t)m1 * lda;
  g.C = Ct;
  g.M = M - m1;
  return launch_rows(s, epi, g, t2);
}

// Ring tiles (shape 0) once the largest problem has kGroupedRingRows rows and
// every leading dimension fits their 32-bit panel offsets; then 256x128 and
// 128x128 interleaved tiles.
constexpr int32_t kGroupedRingRows = 512;

int gemm_grouped_tile_shape(const GemmArgs* probs, int32_t nprob) {
  int32_t max_m = 0;
  bool ring_ok = true, trans = false;
  constexpr int64_t kMax = 0x7fffffff;
  for (int32_t p = 0; p < nprob; ++p) {
    const GemmArgs& g = probs[p];
    max_m = std::max(max_m, g.M);
    // per-lane panel offsets: 256 rows of a row-major operand, or its whole
    // K lines (plus one slab) for a transposed one
    const int64_t kx = (int64_t)g.K + kBK, span_x = (g.trans & GEMM_TRANS_X) ? kx * g.ldx : 256 * g.ldx;
    const int64_t span_w = (g.trans & GEMM_TRANS_W) ? kx * g.ldw : 256 * g.ldw;
    if (2 * std::max(span_x, span_w) > kMax) ring_ok = false;
    trans = trans || g.trans != 0;
  }
  if (trans) return ring_ok ? 0 : -1;
  if (ring_ok && max_m >= kGroupedRingRows) return 0;
  return max_m >= 1024 ? 1 : 2;
}

int32_t gemm_grouped_prepare(GemmArgs* probs, int32_t nprob, int shape) {
  if (shape < 0 || shape > 2 || nprob <= 0) return -1;
  const int BN = shape == 2 ? 128 : 256, BM = shape == 0 ? 256 : 128;
  int32_t total = 0;
  for (int32_t p = 0; p < nprob; ++p) {
    const GemmArgs& g = probs[p];
    const bool ragged_ok = g.trans == (GEMM_TRANS_X | GEMM_TRANS_W);
    if (g.trans != probs[0].trans || g.trans < 0 || g.trans > 3 || (g.trans && shape != 0)) return -1;
    if (g.M <= 0 || g.N <= 0 || g.K <= 0 || (!ragged_ok && g.K % kBK != 0) || g.N % 32 != 0) return -1;
    probs[p].tiles_m = (probs[p].M + BM - 1) / BM;
    probs[p].tiles_n = (probs[p].N + BN - 1) / BN;
    probs[p].tile_start = total;
    total += probs[p].tiles_m * probs[p].tiles_n;
  }
  return total;
}

hipError_t launch_gemm_grouped(hipStream_t s, int epi, const GemmArgs* dprobs, int32_t nprob, int32_t total_tiles,
                               int shape, int trans) {
  if (nprob <= 0 || total_tiles <= 0 || (trans && shape != 0)) return hipErrorInvalidValue;
  if (shape == 0) return launch_grouped_ring(s, epi, dprobs, nprob, total_tiles, trans);
  if (shape == 1) return launch_grouped_tile<256, 128, 4, 2>(s, epi, dprobs, nprob, total_tiles);
  return launch_grouped_tile<128, 128, 2, 2>(s, epi, dprobs, nprob, total_tiles);
}

}  // namespace jnx

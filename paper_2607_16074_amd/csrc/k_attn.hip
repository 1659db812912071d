// Segment-masked varlen attention over the packed batch (forward), gfx950,
// and the rotary position embedding applied to q and k before it.
//
// Every sample attends over its own valid rows only -- bidirectionally, or
// causally (row j sees rows 0..j) -- nothing crosses a sample (hence a
// tenant) boundary and alignment rows are neither keys nor queries (their
// output rows are written as zero).  With fewer key/value heads than query
// heads, query head h reads key/value head h / (H / Hkv).
//
// Work item = (sample, head, 128-query tile); a workgroup = 4 wavefronts x 32
// query rows.  (sample, head) groups are dealt round-robin to the 8 XCDs
// (hardware places workgroup b on XCD b % 8) with all query tiles of a group
// on one XCD: they share its L2 for the group's keys and values, and a run of
// long samples (one tenant's) is spread over every XCD.
//
// Per step of KB keys, the K and V tiles ([KB][HD] bf16, row-major) are
// moved global -> LDS by direct DMA (global_load_lds_dwordx4), double
// buffered: the DMA of step j+1 runs under the compute of step j, one
// workgroup barrier per step.  Each LDS row is a permutation of its 16-byte
// chunks (chunk c stored at c ^ swz(row)), chosen per head width so that
// both reads below touch every LDS bank once per 256 bytes.
//
// Scores: S^T = K Q^T with v_mfma_f32_32x32x16_bf16, K the "A" operand
// (16-byte LDS reads), Q held in registers as "B", so each lane owns one
// query row's scores for 16 of every 32 keys and the online-softmax row
// max / sum need only its registers plus one exchange with lane ^ 32
// (v_permlane32_swap, no LDS round trip).  Both products run their
// contraction chunks outermost, so independent accumulators alternate, and
// read the next chunk's fragments before the current chunk's MFMAs.  The
// probabilities then sit in the operand layout of O^T += V^T P^T (keys
// contracted in the permuted order the score layout gives), so P stays in
// registers.  The V^T operand is read from the row-major V tile with
// ds_read_b64_tr_b16: in each 16-lane group, lane j addresses 4 elements of
// key row k0 + j/4 at column n0 + 4(j%4) and receives, transposed, the
// column n0 + (lane % 16) of rows k0..k0+3 -- 4 consecutive keys of one
// head-dim row, as the MFMA wants.  Statistics in fp32, P rounded to bf16.
// Head width 256 runs attn16_fwd_kernel: the same algorithm with 8 waves x 16
// query rows and v_mfma_f32_16x16x32_bf16 (two waves per SIMD).
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define JN_GPTR(p) ((__attribute__((address_space(1))) void*)(p))
#define JN_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int kQRows = 128;  // query rows per workgroup (4 waves x 32, or 8 x 16 at head width 256)
constexpr float kRescale = 8.0f;  // log2 headroom before the running max is moved
constexpr int kKeys = 64;    // keys per step (64 measured best for head widths 64 and 256)

// Chunk permutation of LDS row r (HD/8 chunks of 16 bytes per row).  K
// fragment reads touch 16 consecutive rows (one chunk each) per 16 lanes;
// transposed V reads touch rows k0..k0+3 (k0 % 4 == 0) x 4 adjacent chunks
// per 16 lanes.  Both cover 16 distinct 16-byte bank slots with:
//   HD 32  (4 rows per 256-byte bank row): (r >> 2) & 3
//   HD 64  (2 rows per bank row):          bit-reversed ((r >> 1) & 7)
//   HD 128:                                4 * (r & 3) + ((r >> 2) & 3)
//   HD 256 (r = 4 q + e):                  2 * (e + 4 * ((q ^ q / 2) & 1)) + q / 2
// At head width 256 a transposed read (16 lanes = 4 rows x 2 chunks) is
// served together with a second 16-lane group, and the bank-conflict
// counter located the pairs: groups q and q ^ 1 and groups q and q ^ 2.
// The HD 128 rule puts rows r and r ^ 4 on one bank slot pair (19% of the
// kernel's cycles in conflicts), 2 * (r & 7) + r / 8 rows r and r ^ 8 (9.5%);
// this rule pairs rows r and r ^ 12 only, which no served pair holds
// together (0 conflict cycles, and still 16 distinct slots for the 16 rows of
// a K fragment read).
template <int HD>
__device__ __forceinline__ int attn_swz(int r) {
  if constexpr (HD == 32) {
    return (r >> 2) & 3;
  } else if constexpr (HD == 64) {
    const int x = (r >> 1) & 7;
    return ((x & 1) << 2) | (x & 2) | (x >> 2);
  } else if constexpr (HD == 128) {
    return ((r & 3) << 2) | ((r >> 2) & 3);
  } else {
    const int q = (r >> 2) & 3, e = r & 3;
    return ((e | (((q ^ (q >> 1)) & 1) << 2)) << 1) | ((q >> 1) & 1);
  }
}

template <int N>
__device__ __forceinline__ void attn_wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(N | (7 << 4) | (15 << 8) | (0 << 14));
}

struct AttnShape {
  int32_t d;        // output row width = H * hd
  int32_t ld;       // qkv row width = (H + 2 Hkv) * hd
  int32_t kv_col;   // first key column (H * hd)
  int32_t v_col;    // first value column ((H + Hkv) * hd)
  int32_t n_kv;     // key/value heads
  int32_t group;    // query heads per key/value head
  int32_t qtiles;   // 128-query tiles per sample (of the longest sample)
  int32_t total;    // (sample, key/value head) groups
  int32_t nblocks;  // work-item slots (blocks of the one-item-per-workgroup mapping)
  float scale_log2;
};

template <int HD, int KB, bool CAUSAL>
__global__ __launch_bounds__(256, (HD >= 256 && KB >= 64) ? 1 : 2) void attn_fwd_kernel(
    const uint16_t* __restrict__ qkv, uint16_t* __restrict__ out, const int32_t* __restrict__ seqlens,
    const int32_t* __restrict__ cu_seqlens, AttnShape sh) {
  constexpr int CPR = HD / 8;            // 16-byte chunks per row
  constexpr int TILE = KB * HD;          // elements of one K (or V) tile
  constexpr int NDMA = 2 * TILE / 512;   // 1 KB DMA instructions per stage (K tile, then V tile)
  constexpr int DPW = NDMA / 4;          // per wavefront
  constexpr int RPI = 512 / HD;          // rows per DMA instruction
  constexpr int NQC = HD / 16;           // 16-wide head-dim chunks (score contraction)
  constexpr int NOT = HD / 32;           // 32-row tiles of O^T
  constexpr int NKT = KB / 32;           // 32-key score tiles per step
  constexpr int NKC = KB / 16;           // 16-key P^T operands per step
  static_assert(NDMA % 4 == 0 && KB % 32 == 0, "tile shape");
  __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2 * TILE];

  // XCD-aware work mapping: (sample, key/value head) group g goes to XCD
  // g % 8, and the query tiles of all its query heads to consecutive slots of
  // that XCD (block b runs on XCD b % 8, slot b / 8).  Groups interleave
  // across XCDs, so samples of very different lengths spread evenly, while
  // each group's keys and values are read by one XCD only.
  const int32_t b = blockIdx.x;
  const int32_t slot = b >> 3;
  const int32_t units = sh.group * sh.qtiles;
  const int32_t kg = (slot / units) * 8 + (b & 7);
  if (kg >= sh.total) return;
  const int32_t r_in = slot % units;
  const int32_t qt = r_in % sh.qtiles;
  const int32_t i = kg / sh.n_kv, kvh = kg % sh.n_kv;
  const int32_t h = kvh * sh.group + r_in / sh.qtiles;
  const int32_t d = sh.d;
  const int32_t L = seqlens[i];
  const int32_t base = cu_seqlens[i];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  if (qt == 0) {  // alignment rows of this sample: zero output
    const int32_t pad = cu_seqlens[i + 1] - base - L;
    for (int32_t e = tid; e < pad * (HD / 8); e += 256) {
      const int32_t row = base + L + e / (HD / 8);
      *reinterpret_cast<uint4*>(out + (int64_t)row * d + h * HD + (e % (HD / 8)) * 8) = make_uint4(0, 0, 0, 0);
    }
  }
  const int32_t q0 = qt * kQRows;
  if (q0 >= L) return;

  const int64_t ld = sh.ld;
  const float scale_log2 = sh.scale_log2;
  const uint16_t* Qg = qkv + h * HD;
  const uint16_t* Kg = qkv + sh.kv_col + kvh * HD;
  const uint16_t* Vg = qkv + sh.v_col + kvh * HD;

  // this wave's DMA instructions u = wave*DPW + k fill 1 KB each; lane ->
  // row (v*RPI + lane / CPR) of the K or V tile, physical chunk lane % CPR,
  // which holds logical chunk (lane % CPR) ^ swz(row)
  auto issue_stage = [&](int32_t kb, int stage) {
#pragma unroll
    for (int k = 0; k < DPW; ++k) {
      const int u = wave * DPW + k;
      const bool isv = u >= NDMA / 2;
      const int v = isv ? u - NDMA / 2 : u;
      const int r = v * RPI + lane / CPR;
      const int c = (lane % CPR) ^ attn_swz<HD>(r);
      const int32_t key = min(kb + r, L - 1);
      const uint16_t* src = (isv ? Vg : Kg) + (int64_t)(base + key) * ld + c * 8;
      __builtin_amdgcn_global_load_lds(JN_GPTR(src), JN_LPTR(&lds[stage][u * 512]), 16, 0, 0);
    }
  };

  const int32_t qw = q0 + wave * 32;  // this wave's first query row
  const bool active = qw < L;
  const int32_t qrow = min(qw + (lane & 31), L - 1);
  const int half = lane >> 5;
  bf16x8 qf[NQC];
#pragma unroll
  for (int c = 0; c < NQC; ++c)
    qf[c] = *reinterpret_cast<const bf16x8*>(Qg + (int64_t)(base + qrow) * ld + c * 16 + half * 8);

  // per-lane LDS offsets: K fragment rows kt*32 + lane%32 (swizzle period 16)
  const int krow = lane & 31;
  const int kswz = attn_swz<HD>(krow);
  // transposed V reads: 16-lane group gq = lane / 16, j = lane % 16
  const int j16 = lane & 15;
  const int vrow0 = 4 * half + (j16 >> 2);                           // + kc*16 (+8)
  const int vcol = ((lane >> 4) & 1) * 16 + 4 * (j16 & 3);           // + t*32
  const int vswz0 = attn_swz<HD>(vrow0), vswz1 = attn_swz<HD>(vrow0 + 8);

  f32x16 o[NOT];
#pragma unroll
  for (int t = 0; t < NOT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const int hi4 = half * 4;

  issue_stage(0, 0);
  // causal: keys past the tile's last query are never needed
  const int32_t kend = CAUSAL ? min(L, q0 + kQRows) : L;
  const int32_t nsteps = (kend + KB - 1) / KB;
  for (int32_t jstep = 0; jstep < nsteps; ++jstep) {
    const int32_t kb = jstep * KB;
    attn_wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();  // step j's tiles landed; step j-1's buffer is free
    if (jstep + 1 < nsteps) issue_stage(kb + KB, (jstep + 1) & 1);
    if (!active) continue;
    if (CAUSAL && kb > qw + 31) continue;  // every key of the step is later than the wave's queries
    const uint16_t* Ks = &lds[jstep & 1][0];
    const uint16_t* Vs = &lds[jstep & 1][TILE];

    // S^T for NKT 32-key tiles: dim chunk c outer, so the tiles' accumulators
    // alternate, with the K fragments of chunk c+1 read before the MFMAs of
    // chunk c (each accumulator still sums c = 0..NQC-1 in order)
    f32x16 s[NKT];
    bf16x8 kf[2][NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
      kf[0][kt] = *reinterpret_cast<const bf16x8*>(Ks + (kt * 32 + krow) * HD + ((half ^ kswz) * 8));
    }
#pragma unroll
    for (int c = 0; c < NQC; ++c) {
      if (c + 1 < NQC) {
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
          kf[(c + 1) & 1][kt] =
              *reinterpret_cast<const bf16x8*>(Ks + (kt * 32 + krow) * HD + (((2 * (c + 1) + half) ^ kswz) * 8));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[c & 1][kt], qf[c], s[kt], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // Online softmax in the log2 domain (scores scaled by log2(e)/sqrt(hd)).
    // The running max m only moves when some query of the wave gains more
    // than kRescale (2^8 headroom for p = 2^(s - m) in fp32 and bf16); O and
    // the running sum l always share the same m, so the final O / l is exact
    // whichever m was used.  Keys past the sample are masked in the last step
    // only (wave-uniform branch).  The probabilities use the hardware exp2
    // (v_exp_f32; results below 2^-126 flush to zero, far below P's bf16
    // rounding): the library exp2f adds a denormal-range fix-up of about four
    // instructions per score, which measured 7-21% of this kernel's time.
    float mloc = -INFINITY;
    if (kb + KB > L || (CAUSAL && kb + KB - 1 > qw)) {
      const int32_t qlane = qw + (lane & 31);
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int32_t key = kb + kt * 32 + (r >> 2) * 8 + hi4 + (r & 3);
          if (key >= L || (CAUSAL && key > qlane)) s[kt][r] = -INFINITY;
        }
    }
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[kt][r]);
    mloc = max_xor32(mloc) * scale_log2;
    if (__any(mloc > m_run + kRescale)) {
      const float m_new = fmaxf(m_run, mloc);
      if (__all(m_run == -INFINITY)) {
        m_run = m_new;  // first update: O and l are still zero
      } else {
        const float alpha = exp2f(m_run - m_new);
        l_run *= alpha;
        m_run = m_new;
#pragma unroll
        for (int t = 0; t < NOT; ++t)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[t][e] *= alpha;
      }
    }
    float lsum = 0.f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[kt][r], scale_log2, -m_run));
        s[kt][r] = p;
        lsum += p;
      }
    lsum = sum_xor32(lsum);
    l_run += lsum;

    // P^T operands: 16-key chunk kc holds registers 8*(kc&1) .. +7 of tile kc>>1,
    // i.e. keys kc*16 + 4*half + 0..3 and kc*16 + 8 + 4*half + 0..3
    bf16x8 pf[NKC];
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kc][e] = (__bf16)s[kc >> 1][(kc & 1) * 8 + e];
    // O^T += V^T P^T: key chunk kc outer, so the head-dim blocks'
    // accumulators alternate, with the V^T fragments of chunk kc+1 read
    // before the MFMAs of chunk kc (each o[t] still sums kc = 0..NKC-1 in order)
    auto read_v = [&](int kc, bf16x8 (&vf)[NOT]) {
      const int r0 = kc * 16 + vrow0;
#pragma unroll
      for (int t = 0; t < NOT; ++t) {
        const int col = t * 32 + vcol;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (__attribute__((address_space(3))) bf16x4*)(Vs + r0 * HD + (((col >> 3) ^ vswz0) * 8) + (col & 7)));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (__attribute__((address_space(3))) bf16x4*)(Vs + (r0 + 8) * HD + (((col >> 3) ^ vswz1) * 8) + (col & 7)));
        vf[t] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    };
    bf16x8 vb[2][NOT];
    read_v(0, vb[0]);
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      if (kc + 1 < NKC) read_v(kc + 1, vb[(kc + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < NOT; ++t) o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vb[kc & 1][t], pf[kc], o[t], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if (!active) return;
  const int32_t q = qw + (lane & 31);
  if constexpr (HD <= 64) {
    const float inv = 1.0f / l_run;
    // lane (query l % 32, half l / 32) holds head-dim columns 32 t + 8 rr +
    // 4 (l / 32) .. +3; swapping the packed blocks rr+1 of the low half with
    // the blocks rr of the high half (rr even) leaves each lane 8 consecutive
    // columns, 32 t + 8 rr + 8 (l / 32), for one 16-byte store (at head width
    // 128 the causal kernel then spilled registers, so it keeps 8-byte stores)
    uint16_t* orow = out + (int64_t)(base + q) * d + h * HD + 2 * hi4;
#pragma unroll
    for (int t = 0; t < NOT; ++t)
#pragma unroll
      for (int rr = 0; rr < 4; rr += 2) {
        const auto a = __builtin_amdgcn_permlane32_swap(pack_bf2(o[t][rr * 4] * inv, o[t][rr * 4 + 1] * inv),
                                                        pack_bf2(o[t][rr * 4 + 4] * inv, o[t][rr * 4 + 5] * inv),
                                                        false, false);
        const auto c = __builtin_amdgcn_permlane32_swap(pack_bf2(o[t][rr * 4 + 2] * inv, o[t][rr * 4 + 3] * inv),
                                                        pack_bf2(o[t][rr * 4 + 6] * inv, o[t][rr * 4 + 7] * inv),
                                                        false, false);
        if (q < L) *reinterpret_cast<uint4*>(orow + t * 32 + rr * 8) = make_uint4(a[0], c[0], a[1], c[1]);
      }
  } else {
    if (q >= L) return;
    const float inv = 1.0f / l_run;
    uint16_t* orow = out + (int64_t)(base + q) * d + h * HD;
#pragma unroll
    for (int t = 0; t < NOT; ++t)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
        *reinterpret_cast<uint2*>(orow + t * 32 + rr * 8 + hi4) =
            make_uint2(pack_bf2(o[t][rr * 4] * inv, o[t][rr * 4 + 1] * inv),
                       pack_bf2(o[t][rr * 4 + 2] * inv, o[t][rr * 4 + 3] * inv));
  }
}


// Head width 256: 8 wavefronts x 16 query rows with v_mfma_f32_16x16x32_bf16,
// so that two waves share each SIMD and one wave's softmax and LDS reads run
// under the other's matrix products (4 waves x 32 rows need ~480 registers
// per lane: one wave per SIMD, whose MFMA, VALU and LDS work then run one
// after another).  Per wave: O^T 16 x 256 in 64 registers, Q in 32, scores of
// a 64-key step in 16.  Measured: 0.56 -> 0.45 ms on the 2B-shaped batch,
// 15-23% faster on 300-3000-token samples; at head width 128 the same layout
// was no faster on 300-token samples and 9% slower on 1000-token ones, so
// that width keeps attn_fwd_kernel.
// Its 128 KB of K/V stages leave room for one workgroup per compute unit, so
// a workgroup that fetched its Q rows and first stage only after starting
// left the compute unit idle for that fetch, and between workgroups: timer
// stamps on the 2B-shaped batch put ~13K of a work item's ~38K cycles
// outside the key loop.  The grid is therefore one workgroup per compute
// unit, each running a fixed list of work items, with the next item's first
// K/V stage and Q rows fetched under the current item's last key step
// (8.1 -> 7.1 ms per 18-layer step).  The output is written 16 bytes per
// lane after a lane swap (8.1 -> 6.5 ms with both).  The work of an item,
// hence every output bit, is unchanged.
//   S^T = K Q^T: A = K (16 keys x 32 dims), B = Q (32 dims x 16 queries);
//     lane l holds query l % 16 and keys 4 (l / 16) .. +3 of each 16-key block.
//   O^T += V^T P^T over a 32-key chunk (blocks 2c, 2c+1): B slot 8 q + e of
//     lane l (q = l / 16) is key 4 q + e of block 2c for e < 4 and key
//     4 q + e - 4 of block 2c+1 otherwise -- the scores' own layout -- and the
//     A operand (16 head-dim rows) takes the same key order from two
//     transposed reads of 4 keys each.
template <int HD, bool CAUSAL>
__global__ __launch_bounds__(512, 1) void attn16_fwd_kernel(const uint16_t* __restrict__ qkv, uint16_t* __restrict__ out,
                                                          const int32_t* __restrict__ seqlens,
                                                          const int32_t* __restrict__ cu_seqlens, AttnShape sh) {
  constexpr int KB = 64;                 // keys per step
  constexpr int NW = 8;                  // wavefronts
  constexpr int CPR = HD / 8;            // 16-byte chunks per row
  constexpr int TILE = KB * HD;          // elements of one K (or V) tile
  constexpr int NDMA = 2 * TILE / 512;   // 1 KB DMA instructions per stage (K tile, then V tile)
  constexpr int DPW = NDMA / NW;         // per wavefront
  constexpr int RPI = 512 / HD;          // rows per DMA instruction
  constexpr int NQC = HD / 32;           // 32-wide head-dim chunks (score contraction)
  constexpr int NOT = HD / 16;           // 16-row blocks of O^T
  static_assert(HD == 256, "head width");
  static_assert(NDMA % NW == 0, "tile shape");
  __shared__ __attribute__((aligned(1024))) uint16_t lds[2][2 * TILE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j16 = lane & 15, quad = lane >> 4;
  const int32_t d = sh.d;
  const int64_t ld = sh.ld;
  const float scale_log2 = sh.scale_log2;
  const int32_t units = sh.group * sh.qtiles;

  // A workgroup runs the work items of blocks blockIdx.x, + gridDim.x, ...
  // (block b: the mapping of attn_fwd_kernel, so b % 8 still names the XCD
  // when gridDim.x % 8 == 0).  The first K/V stage and the Q rows of the
  // next item are fetched under the last key step of the current one.
  struct Item {
    int32_t h, kvh, L, base, q0, nsteps;
  };
  auto decode = [&](int32_t b, Item& it) -> bool {  // false: the block has no work
    const int32_t slot = b >> 3;
    const int32_t kg = (slot / units) * 8 + (b & 7);
    if (kg >= sh.total) return false;
    const int32_t r_in = slot % units;
    const int32_t qt = r_in % sh.qtiles;
    const int32_t i = kg / sh.n_kv;
    it.kvh = kg % sh.n_kv;
    it.h = it.kvh * sh.group + r_in / sh.qtiles;
    it.L = seqlens[i];
    it.base = cu_seqlens[i];
    if (qt == 0) {  // alignment rows of this sample: zero output
      const int32_t pad = cu_seqlens[i + 1] - it.base - it.L;
      for (int32_t e = tid; e < pad * (HD / 8); e += 512) {
        const int32_t row = it.base + it.L + e / (HD / 8);
        *reinterpret_cast<uint4*>(out + (int64_t)row * d + it.h * HD + (e % (HD / 8)) * 8) = make_uint4(0, 0, 0, 0);
      }
    }
    it.q0 = qt * kQRows;
    if (it.q0 >= it.L) return false;
    const int32_t kend = CAUSAL ? min(it.L, it.q0 + kQRows) : it.L;
    it.nsteps = (kend + KB - 1) / KB;
    return true;
  };
  auto next_item = [&](int32_t b, Item& it) -> int32_t {  // first block >= b (same residue) with work
    for (; b < sh.nblocks; b += gridDim.x)
      if (decode(b, it)) return b;
    return sh.nblocks;
  };
  auto issue_stage = [&](const Item& it, int32_t kb, int stage) {
    const uint16_t* Kg = qkv + sh.kv_col + it.kvh * HD;
    const uint16_t* Vg = qkv + sh.v_col + it.kvh * HD;
#pragma unroll
    for (int k = 0; k < DPW; ++k) {
      const int u = wave * DPW + k;
      const bool isv = u >= NDMA / 2;
      const int v = isv ? u - NDMA / 2 : u;
      const int r = v * RPI + lane / CPR;
      const int c = (lane % CPR) ^ attn_swz<HD>(r);
      const int32_t key = min(kb + r, it.L - 1);
      const uint16_t* src = (isv ? Vg : Kg) + (int64_t)(it.base + key) * ld + c * 8;
      __builtin_amdgcn_global_load_lds(JN_GPTR(src), JN_LPTR(&lds[stage][u * 512]), 16, 0, 0);
    }
  };
  bf16x8 qf[NQC];
  auto load_q = [&](const Item& it) {
    const int32_t qrow = min(it.q0 + wave * 16 + j16, it.L - 1);
    const uint16_t* Qg = qkv + it.h * HD + (int64_t)(it.base + qrow) * ld + quad * 8;
#pragma unroll
    for (int c = 0; c < NQC; ++c) qf[c] = *reinterpret_cast<const bf16x8*>(Qg + c * 32);
  };

  Item cur, nxt;
  int32_t b = next_item(blockIdx.x, cur);
  if (b >= sh.nblocks) return;
  load_q(cur);
  issue_stage(cur, 0, 0);

  // K fragment of 16-key block kb16, dim chunk c: row 16 kb16 + j16, logical
  // 16-byte chunk 4 c + quad; rows 16 kb16 + j share the swizzle of row j
  const int kswz = attn_swz<HD>(j16);
  // V^T reads: group quad, lane j16 addresses key row 4 quad + j16 / 4 (+ 32 c,
  // + 16 for the second half) at head-dim column 16 t + 4 (j16 % 4); those rows
  // share one swizzle
  const int vrow = 4 * quad + (j16 >> 2);
  const int vswz = attn_swz<HD>(vrow);

  int par = 0;  // buffer of the current item's first step
  while (true) {
    const int32_t qw = cur.q0 + wave * 16;  // this wave's first query row
    const bool active = qw < cur.L;
    f32x4 o[NOT];
#pragma unroll
    for (int t = 0; t < NOT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;
    int32_t bn = sh.nblocks;  // next block with work, found in the last step
    for (int32_t jstep = 0; jstep < cur.nsteps; ++jstep) {
      const int32_t kb = jstep * KB;
      const int stage = (par + jstep) & 1;
      attn_wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();  // step j's tiles landed; step j-1's buffer is free
      const bool last = jstep + 1 == cur.nsteps;
      if (!last) {
        issue_stage(cur, kb + KB, stage ^ 1);
      } else {
        bn = next_item(b + gridDim.x, nxt);
        if (bn < sh.nblocks) issue_stage(nxt, 0, stage ^ 1);
      }
      // every key of the step later than the wave's queries: nothing to do
      const bool work = active && !(CAUSAL && kb > qw + 15);
      const uint16_t* Ks = &lds[stage][0];
      const uint16_t* Vs = &lds[stage][TILE];

      // scores: dim chunk c outer, so the four 16-key blocks' accumulators
      // alternate; the K fragments of chunk c+1 are read before the MFMAs of
      // chunk c (each accumulator still sums c = 0..NQC-1 in order)
      f32x4 s[4];
      if (work) {
        bf16x8 kf[2][4];
#pragma unroll
        for (int kb16 = 0; kb16 < 4; ++kb16) {
          s[kb16] = f32x4{0.f, 0.f, 0.f, 0.f};
          kf[0][kb16] = *reinterpret_cast<const bf16x8*>(Ks + (kb16 * 16 + j16) * HD + ((quad ^ kswz) * 8));
        }
#pragma unroll
        for (int c = 0; c < NQC; ++c) {
          if (c + 1 < NQC) {
#pragma unroll
            for (int kb16 = 0; kb16 < 4; ++kb16)
              kf[(c + 1) & 1][kb16] = *reinterpret_cast<const bf16x8*>(Ks + (kb16 * 16 + j16) * HD +
                                                                       (((4 * (c + 1) + quad) ^ kswz) * 8));
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int kb16 = 0; kb16 < 4; ++kb16)
            s[kb16] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[c & 1][kb16], qf[c], s[kb16], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if (last && bn < sh.nblocks) load_q(nxt);  // Q is not read again in this item
      if (!work) continue;
      // online softmax (see attn_fwd_kernel); the four lanes of a query are
      // lane ^ 16 and lane ^ 32 apart
      float mloc = -INFINITY;
      if (kb + KB > cur.L || (CAUSAL && kb + KB - 1 > qw)) {
        const int32_t qlane = qw + j16;
#pragma unroll
        for (int kb16 = 0; kb16 < 4; ++kb16)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int32_t key = kb + kb16 * 16 + quad * 4 + e;
            if (key >= cur.L || (CAUSAL && key > qlane)) s[kb16][e] = -INFINITY;
          }
      }
#pragma unroll
      for (int kb16 = 0; kb16 < 4; ++kb16)
#pragma unroll
        for (int e = 0; e < 4; ++e) mloc = fmaxf(mloc, s[kb16][e]);
      mloc = max_xor32(max_xor16(mloc)) * scale_log2;
      if (__any(mloc > m_run + kRescale)) {
        const float m_new = fmaxf(m_run, mloc);
        if (__all(m_run == -INFINITY)) {
          m_run = m_new;  // first update: O and l are still zero
        } else {
          const float alpha = exp2f(m_run - m_new);
          l_run *= alpha;
          m_run = m_new;
#pragma unroll
          for (int t = 0; t < NOT; ++t) o[t] *= alpha;
        }
      }
      float lsum = 0.f;
#pragma unroll
      for (int kb16 = 0; kb16 < 4; ++kb16)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[kb16][e], scale_log2, -m_run));
          s[kb16][e] = p;
          lsum += p;
        }
      lsum = sum_xor32(sum_xor16(lsum));
      l_run += lsum;

      bf16x8 pf[2];
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pf[c][e] = (__bf16)s[2 * c][e];
          pf[c][4 + e] = (__bf16)s[2 * c + 1][e];
        }
      // P.V: the V^T fragments of head-dim block t+2 are read before the
      // MFMAs of block t
      auto read_v = [&](int t, bf16x8 (&vf)[2]) {
        const int col = t * 16 + 4 * (j16 & 3);
        const int pos = (((col >> 3) ^ vswz) * 8) + (col & 7);
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int r0 = c * 32 + vrow;
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4*)(Vs + r0 * HD + pos));
          const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4*)(Vs + (r0 + 16) * HD + pos));
          vf[c] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
      };
      bf16x8 vb[2][2];
      read_v(0, vb[0]);
#pragma unroll
      for (int t = 0; t < NOT; ++t) {
        if (t + 1 < NOT) read_v(t + 1, vb[(t + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int c = 0; c < 2; ++c) o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb[t & 1][c], pf[c], o[t], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    if (active) {
      // lane (j16, quad) holds head-dim columns 16 t + 4 quad .. +3 of query
      // j16; swapping the packed blocks t+1 of quads 0, 2 with the blocks t
      // of quads 1, 3 leaves each lane 8 consecutive columns: 16 t (quad 0),
      // 16 t + 16 (1), 16 t + 8 (2), 16 t + 24 (3), one 16-byte store each
      const int32_t q = qw + j16;
      const float inv = 1.0f / l_run;
      uint16_t* orow = out + (int64_t)(cur.base + q) * d + cur.h * HD + 16 * (quad & 1) + 8 * (quad >> 1);
#pragma unroll
      for (int t = 0; t < NOT; t += 2) {
        const auto a = __builtin_amdgcn_permlane16_swap(pack_bf2(o[t][0] * inv, o[t][1] * inv),
                                                        pack_bf2(o[t + 1][0] * inv, o[t + 1][1] * inv), false, false);
        const auto c = __builtin_amdgcn_permlane16_swap(pack_bf2(o[t][2] * inv, o[t][3] * inv),
                                                        pack_bf2(o[t + 1][2] * inv, o[t + 1][3] * inv), false, false);
        if (q < cur.L) *reinterpret_cast<uint4*>(orow + t * 16) = make_uint4(a[0], c[0], a[1], c[1]);
      }
    }
    if (bn >= sh.nblocks) break;
    par = (par + cur.nsteps) & 1;
    cur = nxt;
    b = bn;
  }
}

// compute units of the current device (cached per device)
static int attn_compute_units() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cached[dev] = n;
  }
  return cached[dev];
}

hipError_t launch_attention(hipStream_t s, const void* qkv, void* out, const int32_t* seqlens,
                            const int32_t* cu_seqlens, int32_t N, int32_t d, int32_t n_heads, int32_t n_kv_heads,
                            bool causal, int32_t max_seqlen, int32_t align) {
  (void)align;
  const int hd = d / n_heads;
  const int32_t kv = n_kv_heads > 0 ? n_kv_heads : n_heads;
  if (kv < 1 || n_heads % kv != 0) return hipErrorInvalidValue;
  AttnShape sh;
  sh.d = d;
  sh.ld = (n_heads + 2 * kv) * hd;
  sh.kv_col = n_heads * hd;
  sh.v_col = (n_heads + kv) * hd;
  sh.n_kv = kv;
  sh.group = n_heads / kv;
  sh.qtiles = (max_seqlen + kQRows - 1) / kQRows;
  const int64_t total = (int64_t)N * kv;
  const int64_t blocks = (total + 7) / 8 * 8 * sh.group * sh.qtiles;
  if (total <= 0 || blocks > (1LL << 30)) return hipErrorInvalidValue;
  sh.total = (int32_t)total;
  sh.nblocks = (int32_t)blocks;
  sh.scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  const dim3 grid((unsigned)blocks);
  // head width 256: one workgroup per compute unit (its LDS and registers
  // allow no second), each running every gridDim.x-th block
  int cus = attn_compute_units();
  cus -= cus % 8;
  const dim3 grid16((unsigned)(cus >= 8 && blocks > cus ? cus : blocks));
  auto Q = reinterpret_cast<const uint16_t*>(qkv);
  auto O = reinterpret_cast<uint16_t*>(out);
#define JN_ATTN(HDV)                                                                        \
  case HDV:                                                                                 \
    if (causal)                                                                             \
      attn_fwd_kernel<HDV, kKeys, true><<<grid, 256, 0, s>>>(Q, O, seqlens, cu_seqlens, sh);  \
    else                                                                                    \
      attn_fwd_kernel<HDV, kKeys, false><<<grid, 256, 0, s>>>(Q, O, seqlens, cu_seqlens, sh); \
    break;
#define JN_ATTN16(HDV)                                                                          \
  case HDV:                                                                                     \
    if (causal)                                                                                 \
      attn16_fwd_kernel<HDV, true><<<grid16, 512, 0, s>>>(Q, O, seqlens, cu_seqlens, sh);        \
    else                                                                                        \
      attn16_fwd_kernel<HDV, false><<<grid16, 512, 0, s>>>(Q, O, seqlens, cu_seqlens, sh);       \
    break;
  switch (hd) {
    JN_ATTN(32)
    JN_ATTN(64)
    JN_ATTN(128)
    JN_ATTN16(256)
    default:
      return hipErrorInvalidValue;
  }
#undef JN_ATTN
#undef JN_ATTN16
  return hipGetLastError();
}

// ------------------------------------------------------------------ rope ---
// Rotary embedding in place on the q and k head slices of qkv (bf16).  One
// block per row; a thread owns two adjacent pairs (2j, 2j+1) of the row's
// rotation and applies them to a strided subset of its heads, so each sine /
// cosine is computed once per row.  Angles in fp32: p * theta^(-2i/hd).
__global__ __launch_bounds__(256) void rope_kernel(uint16_t* __restrict__ qkv, int32_t ld,
                                                   const int32_t* __restrict__ token_pos, int32_t heads,
                                                   int32_t hd, float log2_theta) {
  const int32_t t = blockIdx.x;
  const int32_t pos = token_pos[t];
  if (pos < 0) return;  // alignment row
  const int32_t half = hd >> 1, q4 = hd >> 2;
  const int32_t j = threadIdx.x % q4, hg = threadIdx.x / q4, hstep = 256 / q4;
  if (hg >= hstep) return;
  float c[2], sn[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const float inv_freq = exp2f(-(float)(2 * (2 * j + e)) / (float)hd * log2_theta);
    sincosf((float)pos * inv_freq, &sn[e], &c[e]);
  }
  uint16_t* row = qkv + (int64_t)t * ld;
  for (int32_t h = hg; h < heads; h += hstep) {
    uint32_t* pa = reinterpret_cast<uint32_t*>(row + h * hd + 2 * j);
    uint32_t* pb = reinterpret_cast<uint32_t*>(row + h * hd + half + 2 * j);
    const uint32_t wa = *pa, wb = *pb;
    const float a0 = __uint_as_float(wa << 16), a1 = __uint_as_float(wa & 0xffff0000u);
    const float b0 = __uint_as_float(wb << 16), b1 = __uint_as_float(wb & 0xffff0000u);
    *pa = pack_bf2(a0 * c[0] - b0 * sn[0], a1 * c[1] - b1 * sn[1]);
    *pb = pack_bf2(b0 * c[0] + a0 * sn[0], b1 * c[1] + a1 * sn[1]);
  }
}

hipError_t launch_rope(hipStream_t s, void* qkv, int32_t ld, const int32_t* token_pos, int32_t T, int32_t heads,
                       int32_t hd, float theta) {
  if (T < 1 || heads < 1 || hd % 4 != 0 || hd / 4 > 256 || !(theta > 0.f)) return hipErrorInvalidValue;
  rope_kernel<<<T, 256, 0, s>>>(reinterpret_cast<uint16_t*>(qkv), ld, token_pos, heads, hd, log2f(theta));
  return hipGetLastError();
}

}  // namespace jnx

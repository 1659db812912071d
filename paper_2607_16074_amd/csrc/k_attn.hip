// Segment-masked varlen attention over the packed batch (forward), gfx950.
//
// Every sample attends bidirectionally over its own valid rows only; nothing
// crosses a sample (hence a tenant) boundary and alignment rows are neither
// keys nor queries (their output rows are written as zero).
//
// Grid (query tile, sample, head); a workgroup = 4 wavefronts x 32 query rows.
// The kernel computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so each lane
// holds one query row's scores for 16 of every 32 keys: the online-softmax
// row max / row sum need only the lane's registers plus one exchange with the
// partner lane (lane ^ 32).  The probabilities then already sit in the
// operand layout of O^T += V^T P^T (a permutation of the 16-key contraction
// index that is applied identically to both operands), so P never goes
// through LDS.  K is staged row-major and V transposed in LDS, 64 keys per
// step (V keys reordered so each P^T-matching operand is one 16-byte read);
// statistics in fp32, P rounded to bf16 for the second MFMA.
#include "jn_device.h"
#include "jn_internal.h"

namespace jnx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kQRows = 128;  // query rows per workgroup (4 waves x 32)
constexpr int kKeys = 64;    // keys per step

// Column of key k (0..63) in a transposed-V row: within each 16-key chunk the
// keys a lane pairs with one P^T operand (chunk + hi*4 + 0..3 and
// chunk + 8 + hi*4 + 0..3, hi = lane >> 5) are stored contiguously, so the
// operand is one 16-byte read.  Adjacent even/odd keys stay adjacent.
__device__ __forceinline__ int vt_pos(int k) {
  const int within = k & 15, blk = within >> 3, sub = within & 7;
  return (k & ~15) + (sub >> 2) * 8 + blk * 4 + (sub & 3);
}

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(const uint16_t* __restrict__ qkv,
                                                          uint16_t* __restrict__ out,
                                                          const int32_t* __restrict__ seqlens,
                                                          const int32_t* __restrict__ cu_seqlens, int32_t d,
                                                          float scale_log2) {
  constexpr int KLD = HD + 8;     // K row pitch in LDS (elements)
  constexpr int VLD = kKeys + 8;  // V^T row pitch in LDS (elements)
  constexpr int NQC = HD / 16;    // 16-wide head-dim chunks
  constexpr int NOT = HD / 32;    // 32-row tiles of O^T
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeys][KLD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[HD][VLD];

  const int32_t i = blockIdx.y, h = blockIdx.z;
  const int32_t L = seqlens[i];
  const int32_t base = cu_seqlens[i];
  const int32_t q0 = blockIdx.x * kQRows;
  const int64_t ld = 3 * (int64_t)d;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  if (blockIdx.x == 0) {  // alignment rows of this sample: zero output
    const int32_t pad = cu_seqlens[i + 1] - base - L;
    for (int32_t e = tid; e < pad * (HD / 8); e += 256) {
      const int32_t row = base + L + e / (HD / 8);
      *reinterpret_cast<uint4*>(out + (int64_t)row * d + h * HD + (e % (HD / 8)) * 8) = make_uint4(0, 0, 0, 0);
    }
  }
  if (q0 >= L) return;

  const uint16_t* Qg = qkv + h * HD;
  const uint16_t* Kg = qkv + d + h * HD;
  const uint16_t* Vg = qkv + 2 * d + h * HD;

  const int32_t qw = q0 + wave * 32;  // this wave's first query row
  const bool active = qw < L;
  const int32_t qrow = min(qw + (lane & 31), L - 1);
  const int fk = (lane >> 5) * 8;
  bf16x8 qf[NQC];
#pragma unroll
  for (int c = 0; c < NQC; ++c)
    qf[c] = *reinterpret_cast<const bf16x8*>(Qg + (int64_t)(base + qrow) * ld + c * 16 + fk);

  f32x16 o[NOT];
#pragma unroll
  for (int t = 0; t < NOT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const int hi4 = (lane >> 5) * 4;

  for (int32_t kb = 0; kb < L; kb += kKeys) {
    __syncthreads();  // previous step's readers are done with Ks / Vt
    // K: 64 rows x HD, 16-byte chunks
    for (int e = tid; e < kKeys * (HD / 8); e += 256) {
      const int kr = e / (HD / 8), c8 = (e % (HD / 8)) * 8;
      const int32_t key = min(kb + kr, L - 1);
      *reinterpret_cast<uint4*>(&Ks[kr][c8]) =
          *reinterpret_cast<const uint4*>(Kg + (int64_t)(base + key) * ld + c8);
    }
    // V transposed, keys in the order the P^T operand uses (see vt_pos): a
    // thread takes two adjacent keys of one 8-wide head-dim chunk and writes
    // 8 packed key pairs; the 32 lanes of a half-wave cover the 32 key pairs
    // of one chunk, so each row write hits 32 distinct banks
    for (int e = tid; e < (kKeys / 2) * (HD / 8); e += 256) {
      const int kp = e % (kKeys / 2), c8 = (e / (kKeys / 2)) * 8;
      const int32_t k0 = min(kb + 2 * kp, L - 1), k1 = min(kb + 2 * kp + 1, L - 1);
      const uint4 a = *reinterpret_cast<const uint4*>(Vg + (int64_t)(base + k0) * ld + c8);
      const uint4 b = *reinterpret_cast<const uint4*>(Vg + (int64_t)(base + k1) * ld + c8);
      const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
      const int pos = vt_pos(2 * kp);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        *reinterpret_cast<uint32_t*>(&Vt[c8 + 2 * w][pos]) = (aw[w] & 0xffffu) | (bw[w] << 16);
        *reinterpret_cast<uint32_t*>(&Vt[c8 + 2 * w + 1][pos]) = (aw[w] >> 16) | (bw[w] & 0xffff0000u);
      }
    }
    __syncthreads();
    if (!active) continue;

    // S^T for two 32-key tiles
    f32x16 s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kt][e] = 0.f;
#pragma unroll
      for (int c = 0; c < NQC; ++c) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[kt * 32 + (lane & 31)][c * 16 + fk]);
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[c], s[kt], 0, 0, 0);
      }
    }
    // scale, mask keys past the sample, running max
    float mloc = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int32_t key = kb + kt * 32 + (r >> 2) * 8 + hi4 + (r & 3);
        const float v = key < L ? s[kt][r] * scale_log2 : -INFINITY;
        s[kt][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = exp2f(m_run - m_new);
    float lsum = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(s[kt][r] - m_new);
        s[kt][r] = p;
        lsum += p;
      }
    lsum += __shfl_xor(lsum, 32, 64);
    l_run = l_run * alpha + lsum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < NOT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[t][e] *= alpha;

    // P^T operands: 16-key chunk kc holds registers 8*(kc&1) .. +7 of tile kc>>1
    bf16x8 pf[4];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kc][e] = (__bf16)s[kc >> 1][(kc & 1) * 8 + e];
#pragma unroll
    for (int t = 0; t < NOT; ++t) {
      const uint16_t* vrow = &Vt[t * 32 + (lane & 31)][0];
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        // keys kc*16 + hi4 + 0..3 and kc*16 + 8 + hi4 + 0..3, contiguous in vt_pos order
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(vrow + kc * 16 + 2 * hi4);
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kc], o[t], 0, 0, 0);
      }
    }
  }

  if (!active) return;
  const int32_t q = qw + (lane & 31);
  if (q >= L) return;
  const float inv = 1.0f / l_run;
  uint16_t* orow = out + (int64_t)(base + q) * d + h * HD;
#pragma unroll
  for (int t = 0; t < NOT; ++t)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int c = t * 32 + rr * 8 + hi4;
      *reinterpret_cast<uint2*>(orow + c) =
          make_uint2(pack_bf2(o[t][rr * 4] * inv, o[t][rr * 4 + 1] * inv),
                     pack_bf2(o[t][rr * 4 + 2] * inv, o[t][rr * 4 + 3] * inv));
    }
}

hipError_t launch_attention(hipStream_t s, const void* qkv, void* out, const int32_t* seqlens,
                            const int32_t* cu_seqlens, int32_t N, int32_t d, int32_t n_heads, int32_t max_seqlen,
                            int32_t align) {
  (void)align;
  const int hd = d / n_heads;
  dim3 grid((max_seqlen + kQRows - 1) / kQRows, N, n_heads);
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
  auto Q = reinterpret_cast<const uint16_t*>(qkv);
  auto O = reinterpret_cast<uint16_t*>(out);
  switch (hd) {
    case 32: attn_fwd_kernel<32><<<grid, 256, 0, s>>>(Q, O, seqlens, cu_seqlens, d, scale_log2); break;
    case 64: attn_fwd_kernel<64><<<grid, 256, 0, s>>>(Q, O, seqlens, cu_seqlens, d, scale_log2); break;
    case 128: attn_fwd_kernel<128><<<grid, 256, 0, s>>>(Q, O, seqlens, cu_seqlens, d, scale_log2); break;
    case 256: attn_fwd_kernel<256><<<grid, 256, 0, s>>>(Q, O, seqlens, cu_seqlens, d, scale_log2); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace jnx

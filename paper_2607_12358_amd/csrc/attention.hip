// Full non-causal multi-head self-attention over all video (and text) tokens.
//
// bf16 path: flash-style single pass on MFMA (v_mfma_f32_32x32x16_bf16).
//   A workgroup owns 128 queries of one head (4 waves x 32 queries) and
//   streams the head's keys in tiles of 64 through LDS, double-buffered with
//   register prefetch.  Scores are formed transposed, S^T = K Q^T, so that a
//   lane owns one query (lane % 32) and 16 keys per 32-key block: the row max
//   is an in-register max plus one exchange with the partner half-wave, and
//   the row sum stays a per-lane partial until the end.  The probabilities
//   P^T in accumulator layout are exactly the B operand of O^T = V^T P^T when
//   the contraction index is relabelled accordingly, so P never leaves
//   registers; V is stored transposed (keys contiguous) by the QKV epilogue,
//   and keys are staged into LDS in a permuted order so the matching A
//   operand is one 16-byte read from an XOR-swizzled V^T tile (no LDS bank
//   conflicts).  Work items are mapped so each XCD streams a contiguous,
//   head-major range (a head's K/V passes through few L2s).  Softmax runs in the
//   exp2 domain with log2(e)/sqrt(d) folded into one multiply, in fp32.
// fp32 path: one thread per query with K/V tiles in LDS, online softmax in
//   fp32 (for the fp32 configuration).
#include "common.h"

namespace acid {

namespace {

constexpr int BQ = 128, BKV = 64;

template <int D>
struct AttnLds {
  static constexpr int KLD = D;         // K tile row stride (elements), XOR-swizzled
  static constexpr int VLD = BKV;       // V^T tile row stride: 128 B, XOR-swizzled
  static constexpr int K_ELEMS = BKV * KLD;
  static constexpr int V_ELEMS = D * VLD;
  static constexpr size_t BYTES = (size_t)2 * (K_ELEMS + V_ELEMS) * sizeof(bf16);
};

// Keys are staged into the K tile in the order pi(j) = j with bits 2 and 3
// swapped (an involution).  Then the 8 probabilities a lane feeds to one
// P V^T MFMA step are 8 consecutive keys, so the matching V^T operand is one
// 16-byte LDS read.
__device__ __forceinline__ int key_perm(int j) {
  return (j & ~12) | ((j & 4) << 1) | ((j & 8) >> 1);
}

// 16-byte slot of chunk c in row r of a tile with 2^log2c chunks per row:
// 16 consecutive rows read at one chunk cover all 64 four-byte LDS banks
// (rows of 256 B start on the same bank: XOR with r % 16; rows of 128 B
// alternate halves: XOR with (r / 2) % 8).
template <int CHUNKS>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (CHUNKS == 16) return c ^ (r & 15);
  else return c ^ ((r >> 1) & 7);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// One 16-byte-per-lane global -> LDS DMA: lane l writes LDS bytes
// [lds + 16 l, +16).  Inline assembly keeps it out of the compiler's
// wait-count bookkeeping (completion is waited for explicitly).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_byte) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(g), "s"(lds_byte)
      : "memory");
}

// Bijection from dispatch order to (head, query-tile) work items that gives
// XCD x (workgroups bid = x, x+8, ...) a contiguous, head-major range, so a
// head's K/V is streamed through as few L2s as possible.
__device__ __forceinline__ int64_t attn_xcd_remap(int64_t bid, int64_t T) {
  constexpr int64_t NX = 8;
  const int64_t x = bid % NX, local = bid / NX;
  const int64_t q = T / NX, r = T % NX;
  return (x < r) ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

template <int D>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const bf16* Q,
                                                           const bf16* Kp,
                                                           const bf16* Vt,
                                                           int64_t L, int64_t vt_ld, int n_heads,
                                                           bf16* __restrict__ O,
                                                           float scale_log2) {
  using Ld = AttnLds<D>;
  constexpr int KLD = Ld::KLD, VLD = Ld::VLD;
  constexpr int NK = D / 16;     // MFMA K-steps over the head dim
  constexpr int ND = D / 32;     // 32-row blocks of O^T
  constexpr int CPT = D / 32;    // 16-byte chunks per thread per tile
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* Ks = reinterpret_cast<bf16*>(smem);
  bf16* Vs = Ks + 2 * Ld::K_ELEMS;

  const int64_t n_qt = (L + BQ - 1) / BQ;
  const int64_t item = attn_xcd_remap(blockIdx.x, n_qt * n_heads);
  const int head = (int)(item / n_qt);
  const int64_t qt = item - (int64_t)head * n_qt;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int64_t qrow = qt * BQ + wave * 32 + lr;

  const bf16* Qh = Q + (int64_t)head * L * D;
  const bf16* Kh = Kp + (int64_t)head * L * D;
  const bf16* Vh = Vt + (int64_t)head * D * vt_ld;

  bf16x8 qf[NK];
  {
    const bf16* qsrc = Qh + (qrow < L ? qrow : L - 1) * D + lg * 8;
    const uint32_t qmask = qrow < L ? 0xFFFFFFFFu : 0u;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      uint4 v = *reinterpret_cast<const uint4*>(qsrc + kk * 16);
      v = make_uint4(v.x & qmask, v.y & qmask, v.z & qmask, v.w & qmask);
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x16 o[ND];
#pragma unroll
  for (int db = 0; db < ND; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -__builtin_inff(), l_run = 0.f;

  // Staging.  Full tiles go global -> LDS by DMA: instruction i of wave w
  // fills 1 KB at (4 w + i) KB of the tile (K: D/32 instructions per wave,
  // V^T: D/32).  K tile: LDS row r (D * 2 bytes) holds key j0 + key_perm(r);
  // V^T tile: LDS row d (128 bytes) holds keys j0 .. j0+63 of head dim d.
  // Chunks sit at swizzled slots (swz).  The tail tile (the one reaching past
  // L) is staged through registers instead, with keys >= L zeroed.
  constexpr int KCH = D / 8;              // 16-byte chunks per K row
  constexpr int KROWS_PER_KB = 1024 / (2 * D);  // K rows per 1 KB
  u32x4 rk[CPT], rv[CPT];
  // Offsets are 32-bit element offsets from the per-head base pointers
  // (a head's K is L * d elements, its V^T d * vt_ld: far below 2^31).
  const int Li = (int)L;
  const int vld = (int)vt_ld;
  const uint32_t ks_lds = (uint32_t)(uintptr_t)(lds_void_t*)Ks;
  const uint32_t vs_lds = (uint32_t)(uintptr_t)(lds_void_t*)Vs;
#define ATTN_DMA(BUF, J0)                                                               \
  do {                                                                                  \
    _Pragma("unroll") for (int i = 0; i < CPT; ++i) {                                   \
      const int blk_ = wave * CPT + i;                                                  \
      const int r_ = blk_ * KROWS_PER_KB + lane / KCH;                                  \
      const int c_ = swz<KCH>(r_, lane % KCH);                                          \
      dma16(Kh + (uint32_t)(((J0) + key_perm(r_)) * D + c_ * 8),                        \
            __builtin_amdgcn_readfirstlane(ks_lds + ((BUF) * Ld::K_ELEMS) * 2 + blk_ * 1024)); \
    }                                                                                   \
    _Pragma("unroll") for (int i = 0; i < CPT; ++i) {                                   \
      const int blk_ = wave * CPT + i;                                                  \
      const int d_ = blk_ * 8 + (lane >> 3);                                            \
      const int c_ = swz<8>(d_, lane & 7);                                              \
      dma16(Vh + (uint32_t)(d_ * vld + (J0) + c_ * 8),                                  \
            __builtin_amdgcn_readfirstlane(vs_lds + ((BUF) * Ld::V_ELEMS) * 2 + blk_ * 1024)); \
    }                                                                                   \
  } while (0)
#define ATTN_GLOAD(J0)                                                                  \
  do {                                                                                  \
    _Pragma("unroll") for (int i = 0; i < CPT; ++i) {                                   \
      const int c_ = tid + 256 * i;                                                     \
      const int key_ = (J0) + c_ / KCH;                                                 \
      const uint32_t off_ = (uint32_t)((key_ < Li ? key_ : Li - 1) * D + (c_ % KCH) * 8); \
      rk[i] = *reinterpret_cast<const u32x4*>(Kh + off_);                               \
    }                                                                                   \
    _Pragma("unroll") for (int i = 0; i < CPT; ++i) {                                   \
      const int c_ = tid + 256 * i;                                                     \
      const int key0_ = (J0) + (c_ & 7) * 8;                                            \
      const uint32_t off_ = (uint32_t)((c_ >> 3) * vld + (key0_ < Li ? key0_ : 0));     \
      rv[i] = *reinterpret_cast<const u32x4*>(Vh + off_);                               \
    }                                                                                   \
  } while (0)
// Writes the register-staged tail tile J0 to LDS with keys >= L zeroed.
#define ATTN_SSTORE(BUF, J0)                                                            \
  do {                                                                                  \
    _Pragma("unroll") for (int i = 0; i < CPT; ++i) {                                   \
      const int c_ = tid + 256 * i;                                                     \
      u32x4 kv_ = rk[i], vv_ = rv[i];                                                   \
      kv_ &= ((J0) + c_ / KCH < Li) ? 0xFFFFFFFFu : 0u;                                 \
      const int key0_ = (J0) + (c_ & 7) * 8;                                            \
      const int valid_ = key0_ < Li ? Li - key0_ : 0;                                   \
      u32x4 vm_;                                                                        \
      _Pragma("unroll") for (int p_ = 0; p_ < 4; ++p_)                                  \
        vm_[p_] = ((2 * p_ < valid_) ? 0x0000FFFFu : 0u) |                              \
                  ((2 * p_ + 1 < valid_) ? 0xFFFF0000u : 0u);                           \
      vv_ &= vm_;                                                                       \
      const int kr_ = key_perm(c_ / KCH);                                               \
      *reinterpret_cast<u32x4*>(Ks + (BUF) * Ld::K_ELEMS + kr_ * KLD +                  \
                                swz<KCH>(kr_, c_ % KCH) * 8) = kv_;                     \
      *reinterpret_cast<u32x4*>(Vs + (BUF) * Ld::V_ELEMS + (c_ >> 3) * VLD +            \
                                swz<8>(c_ >> 3, c_ & 7) * 8) = vv_;                     \
    }                                                                                   \
  } while (0)
// Stages tile J0 (DMA, or registers for the tail) / completes it.
#define ATTN_STAGE_BEGIN(BUF, J0)                                                       \
  do {                                                                                  \
    if ((J0) + BKV <= Li) ATTN_DMA(BUF, J0); else ATTN_GLOAD(J0);                       \
  } while (0)
#define ATTN_STAGE_END(BUF, J0)                                                         \
  do {                                                                                  \
    if ((J0) + BKV > Li) ATTN_SSTORE(BUF, J0);                                          \
    __builtin_amdgcn_s_waitcnt(0);                                                      \
  } while (0)

  const int nkv = (Li + BKV - 1) / BKV;
  ATTN_STAGE_BEGIN(0, 0);
  ATTN_STAGE_END(0, 0);
  __syncthreads();
  // The next tile streams in (DMA, or registers for the tail) while this one
  // is consumed; past the last tile it reloads itself into the idle buffer.
  for (int it = 0; it < nkv; ++it) {
    const int buf = it & 1;
    const int j0 = it * BKV;
    const int jn = (it + 1 < nkv ? it + 1 : it) * BKV;
    ATTN_STAGE_BEGIN(buf ^ 1, jn);
    __builtin_amdgcn_sched_barrier(0);

    // S^T (keys x queries) for two 32-key blocks.
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
      const int kr = kb * 32 + lr;
      const bf16* kbase = Ks + buf * Ld::K_ELEMS + kr * KLD;
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(kbase + swz<KCH>(kr, 2 * kk + lg) * 8);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[kb], 0, 0, 0);
      }
    }
    // Keys past L exist only in the last tile: mask them there (uniform branch).
    if (j0 + BKV > Li) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // S^T row kb*32 + 8 (r/4) + 4 lg + r%4 holds key key_perm(row).
          const int key = j0 + kb * 32 + 16 * (r >> 3) + 8 * lg + 4 * ((r >> 2) & 1) + (r & 3);
          if (key >= Li) s[kb][r] = -__builtin_inff();
        }
    }
    // Row max of the raw scores (scale > 0 commutes with max), shared with
    // the partner half-wave that holds the other keys of the same query.
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    // Lazy rescaling: the running reference max moves only when the new
    // max exceeds it by more than 2^8 in probability, so probabilities stay
    // <= 256 (exact range for bf16 and fp32) and the O / l rescale is skipped
    // on most tiles.  The branch is wave-uniform.
    const float m_cand = mx * scale_log2;
    const bool grow = m_cand > m_run + 8.0f;
    if (__any(grow)) {
      const float m_new = grow ? m_cand : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < ND; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    }
    // p = 2^(s log2(e)/sqrt(d) - m): one FMA and one v_exp_f32 per score.
    float psum = 0.f;
    bf16x8 pf[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][r], scale_log2, -m_run));
        psum += p;
        pf[kb][r >> 3][r & 7] = (bf16)p;
      }
    l_run += psum;

    // O^T (d x queries) += V^T P^T.  Contraction slot (lg, e) of K-step
    // (kb, k2) is S^T row kb*32 + 16 k2 + 8 (e/4) + 4 lg + e%4, i.e. key
    // kb*32 + 16 k2 + 8 lg + e: eight consecutive keys, one 16-byte chunk
    // (4 kb + 2 k2 + lg) of the V^T row.
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      const bf16* vrow = Vs + buf * Ld::V_ELEMS + (db * 32 + lr) * VLD;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int kb = ks >> 1, k2 = ks & 1;
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(
            vrow + swz<8>(db * 32 + lr, 4 * kb + 2 * k2 + lg) * 8);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][k2], o[db], 0, 0, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // tail writes and waits after the MFMAs
    ATTN_STAGE_END(buf ^ 1, jn);
    __syncthreads();
  }
#undef ATTN_DMA
#undef ATTN_GLOAD
#undef ATTN_SSTORE
#undef ATTN_STAGE_BEGIN
#undef ATTN_STAGE_END

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  if (qrow < L) {
    bf16* orow = O + qrow * ((int64_t)n_heads * D) + (int64_t)head * D;
#pragma unroll
    for (int db = 0; db < ND; ++db)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (bf16)(o[db][rg * 4 + e] * inv);
        *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * rg + 4 * lg) = w;
      }
  }
}

// ------------------------------------------------------------------ fp32

constexpr int FQ = 64, FKV = 32;

template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ Q,
                                                      const float* __restrict__ Kp,
                                                      const float* __restrict__ Vt, int64_t L,
                                                      int64_t vt_ld, int n_heads,
                                                      float* __restrict__ O, float scale) {
  __shared__ float Ks[FKV][D];
  __shared__ float Vs[FKV][D + 1];
  const int head = blockIdx.y;
  const int t = threadIdx.x;
  const int64_t qrow = (int64_t)blockIdx.x * FQ + t;
  const float* Qh = Q + (int64_t)head * L * D;
  const float* Kh = Kp + (int64_t)head * L * D;
  const float* Vh = Vt + (int64_t)head * D * vt_ld;
  float q[D], o[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = qrow < L ? Qh[qrow * D + d] : 0.f;
    o[d] = 0.f;
  }
  float m_run = -__builtin_inff(), l_run = 0.f;
  for (int64_t j0 = 0; j0 < L; j0 += FKV) {
    __syncthreads();
    for (int idx = t; idx < FKV * D; idx += 64) {
      const int j = idx / D, d = idx % D;
      Ks[j][d] = (j0 + j < L) ? Kh[(j0 + j) * D + d] : 0.f;
    }
    for (int idx = t; idx < FKV * D; idx += 64) {
      const int d = idx / FKV, j = idx % FKV;
      Vs[j][d] = (j0 + j < L) ? Vh[(int64_t)d * vt_ld + j0 + j] : 0.f;
    }
    __syncthreads();
    float sc[FKV];
    float mx = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < FKV; ++j) {
      float a = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) a += q[d] * Ks[j][d];
      sc[j] = (j0 + j < L) ? a * scale : -__builtin_inff();
      mx = fmaxf(mx, sc[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = expf(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] *= alpha;
#pragma unroll
    for (int j = 0; j < FKV; ++j) {
      const float p = expf(sc[j] - m_new);
      l_run += p;
#pragma unroll
      for (int d = 0; d < D; ++d) o[d] += p * Vs[j][d];
    }
  }
  if (qrow < L) {
    const float inv = 1.0f / l_run;
    float* orow = O + qrow * ((int64_t)n_heads * D) + (int64_t)head * D;
#pragma unroll
    for (int d = 0; d < D; ++d) orow[d] = o[d] * inv;
  }
}

template <int D>
hipError_t launch_bf16(int n_heads, int64_t L, const void* q, const void* k, const void* vt,
                       int64_t vt_ld, void* o, hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute((const void*)attn_bf16_kernel<D>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)AttnLds<D>::BYTES);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)D);
  dim3 grid((unsigned)(((L + BQ - 1) / BQ) * n_heads));
  hipLaunchKernelGGL(attn_bf16_kernel<D>, grid, dim3(256), AttnLds<D>::BYTES, s,
                     (const bf16*)q, (const bf16*)k, (const bf16*)vt, L, vt_ld, n_heads,
                     (bf16*)o, scale_log2);
  return hipGetLastError();
}

template <int D>
hipError_t launch_f32(int n_heads, int64_t L, const void* q, const void* k, const void* vt,
                      int64_t vt_ld, void* o, hipStream_t s) {
  dim3 grid((unsigned)((L + FQ - 1) / FQ), (unsigned)n_heads);
  hipLaunchKernelGGL(attn_f32_kernel<D>, grid, dim3(64), 0, s, (const float*)q,
                     (const float*)k, (const float*)vt, L, vt_ld, n_heads, (float*)o,
                     1.0f / sqrtf((float)D));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int dtype, int n_heads, int64_t L, int d, const void* q,
                            const void* k, const void* vt, int64_t vt_ld, void* o,
                            hipStream_t s) {
  if (L == 0) return hipSuccess;
  if (dtype == ACID_BF16) {
    if (d == 64) return launch_bf16<64>(n_heads, L, q, k, vt, vt_ld, o, s);
    if (d == 128) return launch_bf16<128>(n_heads, L, q, k, vt, vt_ld, o, s);
  } else {
    if (d == 64) return launch_f32<64>(n_heads, L, q, k, vt, vt_ld, o, s);
    if (d == 128) return launch_f32<128>(n_heads, L, q, k, vt, vt_ld, o, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace acid

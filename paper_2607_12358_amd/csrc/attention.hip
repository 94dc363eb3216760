// Full non-causal multi-head self-attention over all video (and text) tokens.
//
// bf16 path: flash-style single pass on MFMA (v_mfma_f32_32x32x16_bf16).
//   A workgroup owns 32 queries per wave of one head (8 waves for d = 128,
//   4 for d = 64) and streams the head's keys in tiles of 64 through two LDS
//   ring buffers filled by global -> LDS DMA.  Scores are formed transposed,
//   S^T = K Q^T, so that a lane owns one query (lane % 32) and 16 keys per
//   32-key block: the row max is an in-register max plus one exchange with
//   the partner half-wave (v_permlane32_swap), and the row sum stays a
//   per-lane partial until the end.  The probabilities P^T in accumulator
//   layout are exactly the B operand of O^T = V^T P^T when the contraction
//   index is relabelled accordingly, so P never leaves registers; V is stored
//   transposed (keys contiguous) by the QKV epilogue, and keys are staged
//   into LDS in a permuted order so the matching A operand is one 16-byte
//   read from an XOR-swizzled V^T tile (no LDS bank conflicts).  Each wave
//   runs a two-stage software pipeline (exponentials of one tile under the
//   score MFMAs of the next; for d = 128 the next tile's row max under the
//   P V MFMAs, for d = 64 an optimistic softmax without a row max, checked
//   through the probability sum).
//   Work items are mapped so each XCD streams a contiguous, head-major range
//   (a head's K/V passes through few L2s).  Softmax runs in the exp2 domain
//   in fp32: with plain Q, log2(e)/sqrt(d) is folded into one FMA per score;
//   with Q stored pre-multiplied by log2(e)/sqrt(d) (as the model's QKV
//   epilogue writes it) the score MFMAs start from -m and deliver the exp2
//   arguments themselves.  The row sum adds the bf16-rounded probabilities
//   that the P V product uses.
// fp32 path: one wave per (head, query), online softmax in fp32 (for the
//   fp32 configuration).
#include <atomic>

#include "common.h"

namespace acid {

namespace {

constexpr int BKV = 64;

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

// One 16-byte-per-lane global -> LDS DMA: lane l reads 16 bytes at
// base + off_bytes(l) and writes LDS bytes [lds + 16 l, +16).  base and lds
// are wave-uniform (scalar registers).  Inline assembly keeps it out of the
// compiler's wait-count bookkeeping (completion is waited for explicitly).
__device__ __forceinline__ uint64_t uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ void dma16(uint64_t base, uint32_t off_bytes, uint32_t lds_byte) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(off_bytes), "s"(base), "s"(lds_byte)
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

// Maximum of a value over the two half-waves (lanes l and l ^ 32).
__device__ __forceinline__ float half_swap_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Software pipeline, per wave and key tile j (LDS holds K_{j+1} and V_j):
//   VALU: p = 2^(s_j - m) for tile j (scores formed one iteration earlier),
//   MFMA: S_{j+1} = K_{j+1} Q^T, then O^T += V_j^T P_j^T,
//   VALU: row max of S_{j+1} (under the P V MFMAs),
// so the softmax of one tile overlaps the score MFMAs of the next.  K runs
// one tile ahead of V in the two LDS ring buffers: iteration j streams
// K_{j+2} and V_{j+1} in while K_{j+1} and V_j are read.  Softmax does not
// depend on the order of the keys, so the ragged last tile (keys up to L)
// is processed first, staged through registers and masked in the prologue;
// every tile of the loop is full and arrives by DMA.
template <int D, int NW, bool kPre>
__global__ __launch_bounds__(64 * NW, 8 / NW) void attn_bf16_kernel(const bf16* Q,
                                                           const bf16* Kp,
                                                           const bf16* Vt,
                                                           int64_t L, int64_t vt_ld, int n_heads,
                                                           bf16* __restrict__ O, int64_t o_ld,
                                                           float scale_log2,
                                                           const int32_t* pred) {
  if (pred && *pred == 0) return;  // predicated off by the device gate
  using Ld = AttnLds<D>;
  constexpr int BQ = 32 * NW, NT = 64 * NW;  // queries / threads per workgroup
  constexpr int KLD = Ld::KLD, VLD = Ld::VLD;
  constexpr int NK = D / 16;     // MFMA K-steps over the head dim
  constexpr int ND = D / 32;     // 32-row blocks of O^T
  constexpr int CPT = D / (8 * NW);  // 16-byte chunks per thread per tile (K, and V^T)
  constexpr int KCH = D / 8;     // 16-byte chunks per K row
  constexpr int KROWS_PER_KB = 1024 / (2 * D);  // K rows per 1 KB
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* Ks = reinterpret_cast<bf16*>(smem);
  bf16* Vs = Ks + 2 * Ld::K_ELEMS;

  const int64_t n_qt = (L + BQ - 1) / BQ;
  const int64_t item = attn_xcd_remap(blockIdx.x, n_qt * n_heads);
  const int head = (int)(item / n_qt);
  const int64_t qt = item - (int64_t)head * n_qt;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  // kPre (Q stored pre-multiplied by log2(e)/sqrt(d)): the score MFMAs start
  // from C = -m instead of 0, so they deliver the exp2 arguments directly and
  // no per-score multiply-add remains.  cneg holds -m in every entry.
  f32x16 cneg;
  auto set_cneg = [&](float v) {
#pragma unroll
    for (int r = 0; r < 16; ++r) cneg[r] = v;
  };

  // Offsets are 32-bit (a head's K is L * d elements, its V^T d * vt_ld:
  // far below 2^31 bytes).
  const int Li = (int)L;
  const int vld = (int)vt_ld;
  const uint32_t ks_lds = (uint32_t)(uintptr_t)(lds_void_t*)Ks;
  const uint32_t vs_lds = (uint32_t)(uintptr_t)(lds_void_t*)Vs;

  // DMA staging of a full tile in 1 KB blocks: block b = CPT w + i is wave
  // w's share.  K tile: LDS row r (D * 2 bytes) holds key j0 + key_perm(r);
  // V^T tile: LDS row d (128 bytes) holds keys j0 .. j0+63 of head dim d;
  // chunks sit at swizzled slots (swz).  With 8 waves (two per SIMD: waves
  // w and w + 4) wave w issues the blocks of both, so wave w + 4 issues no
  // global loads in the loop.  Per-lane byte offsets relative to the tile's
  // first element, and the block each DMA fills:
  constexpr bool kPairDma = NW == 8;
  constexpr int NB = kPairDma ? 2 * CPT : CPT;
  const bool dma_wave = !kPairDma || wave < 4;
  uint32_t koff[NB], voff[NB];
  int kblk[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int blk = (kPairDma ? (wave & 3) + (i / CPT) * 4 : wave) * CPT + i % CPT;
    kblk[i] = blk;
    const int r = blk * KROWS_PER_KB + lane / KCH;
    koff[i] = (uint32_t)(key_perm(r) * D + swz<KCH>(r, lane % KCH) * 8) * 2u;
    const int d = blk * 8 + (lane >> 3);
    voff[i] = (uint32_t)(d * vld + swz<8>(d, lane & 7) * 8) * 2u;
  }
  auto stage_k_dma = [&](int buf, int j0) {
    if (!dma_wave) return;
    const uint64_t base = uniform_ptr(Kh + (int64_t)j0 * D);
#pragma unroll
    for (int i = 0; i < NB; ++i)
      dma16(base, koff[i], ks_lds + buf * Ld::K_ELEMS * 2 + kblk[i] * 1024);
  };
  auto stage_v_dma = [&](int buf, int j0) {
    if (!dma_wave) return;
    const uint64_t base = uniform_ptr(Vh + j0);
#pragma unroll
    for (int i = 0; i < NB; ++i)
      dma16(base, voff[i], vs_lds + buf * Ld::V_ELEMS * 2 + kblk[i] * 1024);
  };
  // The ragged tile j0 .. L-1 through registers, keys >= L zeroed (K rows,
  // and V^T columns, whose padding past L may hold anything).
  auto stage_tail = [&](int buf, int j0) {
    u32x4 rk[CPT], rv[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + NT * i;
      const int key = j0 + c / KCH;
      rk[i] = *reinterpret_cast<const u32x4*>(
          Kh + (uint32_t)((key < Li ? key : Li - 1) * D + (c % KCH) * 8));
      const int key0 = j0 + (c & 7) * 8;
      rv[i] = *reinterpret_cast<const u32x4*>(Vh + (uint32_t)((c >> 3) * vld +
                                                              (key0 < Li ? key0 : 0)));
    }
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + NT * i;
      u32x4 kv = rk[i];
      kv &= (j0 + c / KCH < Li) ? 0xFFFFFFFFu : 0u;
      const int kr = key_perm(c / KCH);
      *reinterpret_cast<u32x4*>(Ks + buf * Ld::K_ELEMS + kr * KLD + swz<KCH>(kr, c % KCH) * 8) =
          kv;
      const int key0 = j0 + (c & 7) * 8;
      const int valid = key0 < Li ? Li - key0 : 0;
      u32x4 vm;
#pragma unroll
      for (int p = 0; p < 4; ++p)
        vm[p] = ((2 * p < valid) ? 0x0000FFFFu : 0u) | ((2 * p + 1 < valid) ? 0xFFFF0000u : 0u);
      *reinterpret_cast<u32x4*>(Vs + buf * Ld::V_ELEMS + (c >> 3) * VLD +
                                swz<8>(c >> 3, c & 7) * 8) = rv[i] & vm;
    }
  };

  // S^T (keys x queries) of the K tile in buffer kbuf, two 32-key blocks.
  auto scores = [&](f32x16(&s)[2], int kbuf) {
    if constexpr (!kPre) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
    }
#pragma unroll
    for (int kk = 0; kk < NK; ++kk)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int kr = kb * 32 + lr;
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(Ks + kbuf * Ld::K_ELEMS + kr * KLD +
                                                            swz<KCH>(kr, 2 * kk + lg) * 8);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk],
                                                        (kPre && kk == 0) ? cneg : s[kb], 0, 0, 0);
      }
  };
  // Row max of the first (raw) score tile, shared with the partner half-wave
  // that holds the other keys of the same query: the initial reference m.
  auto first_max = [&](const f32x16(&s)[2]) {
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    m_run = kPre ? half_swap_max(mx) : half_swap_max(mx) * scale_log2;
  };
  // Scores to exp2 arguments in place: s log2(e)/sqrt(d) - m.
  auto shift = [&](f32x16(&s)[2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        s[kb][r] = kPre ? s[kb][r] - m_run : __builtin_fmaf(s[kb][r], scale_log2, -m_run);
  };
  auto sub_all = [&](f32x16(&s)[2], float v) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] -= v;
  };
  // Row max of a raw score tile (scale > 0 commutes with max), shared with
  // the partner half-wave that holds the other keys of the same query, then
  // the tile is rewritten in place as s log2(e)/sqrt(d) - m (exp2 argument).
  // Lazy rescaling: the reference max m moves only when the new max exceeds
  // it by more than 2^8 in probability, so probabilities stay <= 256 (exact
  // range for bf16 and fp32) and the O / l rescale is skipped on most tiles.
  float m_nx = 0.f, a_nx = 1.f, d_nx = 0.f;
  bool g_nx = false;
  auto row_max_shift = [&](f32x16(&s)[2]) {
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = half_swap_max(mx);
    const float m_cand = mx * scale_log2;
    g_nx = m_cand > m_run + 8.0f;
    m_nx = g_nx ? m_cand : m_run;
    a_nx = __builtin_amdgcn_exp2f(m_run - m_nx);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = __builtin_fmaf(s[kb][r], scale_log2, -m_nx);
  };
  // kPre: the tile already holds s' - m; only the lazy-rescale decision is
  // taken here (its shift by d_nx, rare, is applied at the next iteration).
  auto row_max_check = [&](const f32x16(&s)[2]) {
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = half_swap_max(mx);
    g_nx = mx > 8.0f;
    d_nx = g_nx ? mx : 0.0f;
    m_nx = m_run + d_nx;
    a_nx = __builtin_amdgcn_exp2f(-d_nx);
  };
  // p = 2^(shifted score) for the 16 keys of one P V K-step (kb, k2), rounded
  // to bf16 as the B operand of the P V MFMAs; the row sum adds exactly those
  // bf16 values (v_dot2 with (1, 1)) into ps.
  auto probs_part = [&](const f32x16(&s)[2], int kb, int k2, bf16x8(&pf)[2][2],
                        float(&ps)[2]) {
    const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 8 * k2 + 2 * e;
      const bf16x2 pr = {(bf16)__builtin_amdgcn_exp2f(s[kb][r]),
                         (bf16)__builtin_amdgcn_exp2f(s[kb][r + 1])};
      ps[e & 1] = __builtin_amdgcn_fdot2_f32_bf16(pr, one, ps[e & 1], false);
      w[e] = __builtin_bit_cast(uint32_t, pr);
    }
    pf[kb][k2] = __builtin_bit_cast(bf16x8, w);
  };
  // The whole tile.
  auto probs = [&](const f32x16(&s)[2], bf16x8(&pf)[2][2], float& psum) {
    float ps[2] = {0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) probs_part(s, kb, k2, pf, ps);
    psum = ps[0] + ps[1];
  };
  // O^T (d x queries) += V^T P^T.  Contraction slot (lg, e) of K-step
  // (kb, k2) is S^T row kb*32 + 16 k2 + 8 (e/4) + 4 lg + e%4, i.e. key
  // kb*32 + 16 k2 + 8 lg + e: eight consecutive keys, one 16-byte chunk
  // (4 kb + 2 k2 + lg) of the V^T row.
  auto pv = [&](const bf16x8(&pf)[2][2], int vbuf) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int db = 0; db < ND; ++db) {
        const int kb = ks >> 1, k2 = ks & 1;
        const int vr = db * 32 + lr;
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(Vs + vbuf * Ld::V_ELEMS + vr * VLD +
                                                            swz<8>(vr, 4 * kb + 2 * k2 + lg) * 8);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kb][k2], o[db], 0, 0, 0);
      }
  };

  // Processing order of the key tiles: the ragged tile (if any) first, then
  // the full tiles in order.  u >= 1 maps to the full tile u - has_tail.
  const int nkv = (Li + BKV - 1) / BKV;
  const int has_tail = (Li % BKV) != 0;
  // One pipeline iteration: sc holds S of processed tile it; S of tile it+1
  // goes to sn (on the last tile this reads a stale buffer and is dropped).
  // One pipeline iteration: sc holds the exp2 arguments of processed tile
  // it (against the reference m); S of tile it+1 goes to sn (on the last
  // tile this reads a stale buffer and is dropped).
  //
  // d = 128 (MFMA-bound): the row max of S_{it+1} and its shift run under
  // the P V MFMAs, and the lazy rescale is decided at the top of the next
  // iteration.  d = 64 (VALU-bound: half the MFMA work per score):
  // optimistic softmax, no row max.  The probabilities are formed against
  // the current reference; a lane whose bf16 sum stays <= 2^8 had every
  // p <= 2^8 (the lazy bound).  Otherwise (rare) the wave takes the true row
  // max of the shifted tile, moves the reference to it, rescales O and l,
  // and forms the probabilities again.
  constexpr bool kOptimistic = D == 64;
  auto iter = [&](f32x16(&sc)[2], f32x16(&sn)[2], int it) {
    if (it + 2 < nkv) stage_k_dma(it & 1, (it + 2 - has_tail) * BKV);
    if (it + 1 < nkv) stage_v_dma((it + 1) & 1, (it + 1 - has_tail) * BKV);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!kOptimistic) {
      m_run = m_nx;
      if (__any(g_nx)) {
        l_run *= a_nx;
#pragma unroll
        for (int db = 0; db < ND; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= a_nx;
        if constexpr (kPre) {
          sub_all(sc, d_nx);
          // -m_run in place: (-m) - d equals -(m + d) exactly, and updating
          // cneg's own registers spares the common path a 16-register copy.
#pragma unroll
          for (int r = 0; r < 16; ++r) cneg[r] -= d_nx;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    bf16x8 pf[2][2];
    float psum;
    if constexpr (kPre && !kOptimistic) {
      // The exponentials of the first key block under the score MFMAs of the
      // next tile, those of the second under the first half of the P V
      // MFMAs (which use only the first block), the row max of the next
      // tile under the second half; exponentials (transcendental unit) and
      // the other VALU work in separate groups, one or two of each per MFMA.
      float ps[2] = {0.f, 0.f};
      probs_part(sc, 0, 0, pf, ps);
      probs_part(sc, 0, 1, pf, ps);
      scores(sn, (it + 1) & 1);
      probs_part(sc, 1, 0, pf, ps);
      probs_part(sc, 1, 1, pf, ps);
      psum = ps[0] + ps[1];
      l_run += psum;
      pv(pf, it & 1);
      row_max_check(sn);
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int i = 0; i < 2 * NK; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x400, (16 + 2 * NK - 1) / (2 * NK), 0);
        __builtin_amdgcn_sched_group_barrier(0x002, (16 + 2 * NK - 1) / (2 * NK), 0);
      }
#pragma unroll
      for (int i = 0; i < 2 * ND; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x400, (16 + 2 * ND - 1) / (2 * ND), 0);
        __builtin_amdgcn_sched_group_barrier(0x002, (18 + 2 * ND - 1) / (2 * ND), 0);
      }
#pragma unroll
      for (int i = 0; i < 2 * ND; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, (24 + 2 * ND - 1) / (2 * ND), 0);
      }
    } else {
    probs(sc, pf, psum);
    scores(sn, (it + 1) & 1);
    if constexpr (kOptimistic) {
      // Each score MFMA with one fragment read and a share of the
      // exponentials.
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
      for (int i = 0; i < 2 * NK; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, (66 + 2 * NK - 1) / (2 * NK), 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (__any(!(psum <= 256.0f))) {
        float mx = sc[0][0];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][r]);
        mx = half_swap_max(mx);
        const float d = mx > 0.0f ? mx : 0.0f;
        const float alpha = __builtin_amdgcn_exp2f(-d);
        m_run += d;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < ND; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        sub_all(sc, d);
        if constexpr (kPre) {
          sub_all(sn, d);  // formed against the old reference
          set_cneg(-m_run);
        }
        probs(sc, pf, psum);
      }
      __builtin_amdgcn_sched_barrier(0);
      l_run += psum;
      pv(pf, it & 1);
      if constexpr (!kPre) {
        shift(sn);
        // Each P V MFMA with one fragment read and a share of the shift.
#pragma unroll
        for (int i = 0; i < 4 * ND; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, (32 + 4 * ND - 1) / (4 * ND), 0);
        }
      }
    } else {
      l_run += psum;
      pv(pf, it & 1);
      row_max_shift(sn);
      // Four fragment reads ahead, then each score MFMA with one more read
      // and a share of the exponentials, then each P V MFMA with one read
      // and a share of the row max and shift of the next tile.
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int i = 0; i < 2 * NK; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, (66 + 2 * NK - 1) / (2 * NK), 0);
      }
#pragma unroll
      for (int i = 0; i < 4 * ND; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, (56 + 4 * ND - 1) / (4 * ND), 0);
      }
    }
    }
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);  // this iteration's staging has landed
    __builtin_amdgcn_s_barrier();
  };

  f32x16 sa[2], sb[2];
  if (has_tail) {
    stage_tail(0, (nkv - 1) * BKV);
  } else {
    stage_k_dma(0, 0);
    stage_v_dma(0, 0);
  }
  if (nkv > 1) stage_k_dma(1, (1 - has_tail) * BKV);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if constexpr (kPre) set_cneg(0.0f);
  scores(sa, 0);
  // Every wave has read K tile 0 before the first iteration restages its
  // buffer (a wave running ahead would otherwise overwrite it).
  __syncthreads();
  if (has_tail) {
    // Keys past L get score -inf.  S^T row kb*32 + 8 (r/4) + 4 lg + r%4
    // holds key j0 + key_perm(row).
    const int j0 = (nkv - 1) * BKV;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = j0 + kb * 32 + 16 * (r >> 3) + 8 * lg + 4 * ((r >> 2) & 1) + (r & 3);
        if (key >= Li) sa[kb][r] = -__builtin_inff();
      }
  }
  if constexpr (kPre) {
    // The first reference is the first tile's row max (held against m = 0).
    first_max(sa);
    sub_all(sa, m_run);
    set_cneg(-m_run);
    m_nx = m_run;
  } else if constexpr (kOptimistic) {
    first_max(sa);
    shift(sa);
  } else {
    row_max_shift(sa);
  }
  int it = 0;
  for (; it + 1 < nkv; it += 2) {
    iter(sa, sb, it);
    iter(sb, sa, it + 1);
  }
  if (it < nkv) iter(sa, sb, it);

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  if (qrow < L) {
    bf16* orow = O + qrow * o_ld + (int64_t)head * D;
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

// fp32 path (the small fp32 configuration): one wave per (head, query).
// Lanes take one key each of a 64-key chunk for the scores; the wave max and
// sum give the online softmax; lane l accumulates output dims l, l + 64, ...
// over the chunk's probabilities, broadcast one key at a time.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(const float* __restrict__ Q,
                                                       const float* __restrict__ Kp,
                                                       const float* __restrict__ Vt, int64_t L,
                                                       int64_t vt_ld, int n_heads,
                                                       float* __restrict__ O, int64_t o_ld,
                                                       float scale, const int32_t* pred) {
  if (pred && *pred == 0) return;
  constexpr int C = D / 64;  // output dims per lane
  const int lane = threadIdx.x & 63;
  const int64_t wq = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wq >= L * n_heads) return;  // whole wave; no barriers below
  const int head = (int)(wq / L);
  const int64_t qrow = wq - (int64_t)head * L;
  const float* Kh = Kp + (int64_t)head * L * D;
  const float* Vh = Vt + (int64_t)head * D * vt_ld;
  float q[D];
  {
    const float4* q4 = reinterpret_cast<const float4*>(Q + ((int64_t)head * L + qrow) * D);
#pragma unroll
    for (int d4 = 0; d4 < D / 4; ++d4) {
      const float4 v = q4[d4];
      q[4 * d4] = v.x;
      q[4 * d4 + 1] = v.y;
      q[4 * d4 + 2] = v.z;
      q[4 * d4 + 3] = v.w;
    }
  }
  float o[C];
#pragma unroll
  for (int c = 0; c < C; ++c) o[c] = 0.f;
  float m_run = -__builtin_inff(), l_run = 0.f;
  for (int64_t j0 = 0; j0 < L; j0 += 64) {
    const int64_t j = j0 + lane;
    float s = -__builtin_inff();
    if (j < L) {
      const float4* k4 = reinterpret_cast<const float4*>(Kh + j * D);
      float a = 0.f;
#pragma unroll
      for (int d4 = 0; d4 < D / 4; ++d4) {
        const float4 kv = k4[d4];
        a += q[4 * d4] * kv.x + q[4 * d4 + 1] * kv.y + q[4 * d4 + 2] * kv.z + q[4 * d4 + 3] * kv.w;
      }
      s = a * scale;
    }
    const float m_new = fmaxf(m_run, wave_max(s));  // finite: the chunk has a key
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    const float p = j < L ? exp2f(s - m_new) : 0.f;
    l_run = l_run * alpha + wave_sum(p);
#pragma unroll
    for (int c = 0; c < C; ++c) o[c] *= alpha;
    const int cnt = (int)(L - j0 < 64 ? L - j0 : 64);
    for (int jj = 0; jj < cnt; ++jj) {
      const float pj = __shfl(p, jj, 64);
#pragma unroll
      for (int c = 0; c < C; ++c) o[c] += pj * Vh[(int64_t)(lane + 64 * c) * vt_ld + j0 + jj];
    }
  }
  const float inv = 1.0f / l_run;
  float* orow = O + qrow * o_ld + (int64_t)head * D;
#pragma unroll
  for (int c = 0; c < C; ++c) orow[lane + 64 * c] = o[c] * inv;
}

// Waves per workgroup: 8 for d = 128 (a staged K/V tile feeds 256 queries),
// 4 for d = 64 (finer grid for the shorter sequences of that configuration).
template <int D, bool kPre>
hipError_t launch_bf16(int n_heads, int64_t L, const void* q, const void* k, const void* vt,
                       int64_t vt_ld, void* o, int64_t o_ld, hipStream_t s,
                       const int32_t* pred) {
  constexpr int NW = D == 128 ? 8 : 4;
  constexpr int BQ = 32 * NW;
  // The dynamic-LDS attribute is set once per device (one bit each).
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
  if (!(attr_set.load(std::memory_order_acquire) & bit)) {
    err = hipFuncSetAttribute((const void*)attn_bf16_kernel<D, NW, kPre>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)AttnLds<D>::BYTES);
    if (err != hipSuccess) return err;
    attr_set.fetch_or(bit, std::memory_order_release);
  }
  const float scale_log2 = attn_q_scale(D);
  dim3 grid((unsigned)(((L + BQ - 1) / BQ) * n_heads));
  hipLaunchKernelGGL((attn_bf16_kernel<D, NW, kPre>), grid, dim3(64 * NW), AttnLds<D>::BYTES, s,
                     (const bf16*)q, (const bf16*)k, (const bf16*)vt, L, vt_ld, n_heads,
                     (bf16*)o, o_ld, scale_log2, pred);
  return hipGetLastError();
}

template <int D>
hipError_t launch_f32(int n_heads, int64_t L, const void* q, const void* k, const void* vt,
                      int64_t vt_ld, void* o, int64_t o_ld, hipStream_t s, const int32_t* pred,
                      bool q_prescaled) {
  dim3 grid((unsigned)((L * n_heads + 3) / 4));
  hipLaunchKernelGGL(attn_f32_kernel<D>, grid, dim3(256), 0, s, (const float*)q,
                     (const float*)k, (const float*)vt, L, vt_ld, n_heads, (float*)o, o_ld,
                     q_prescaled ? 1.0f : attn_q_scale(D), pred);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int dtype, int n_heads, int64_t L, int d, const void* q,
                            const void* k, const void* vt, int64_t vt_ld, void* o,
                            hipStream_t s, const int32_t* pred, int64_t o_ld,
                            bool q_prescaled) {
  if (L == 0) return hipSuccess;
  if (o_ld == 0) o_ld = (int64_t)n_heads * d;
  if (dtype == ACID_BF16) {
    if (d == 64)
      return q_prescaled ? launch_bf16<64, true>(n_heads, L, q, k, vt, vt_ld, o, o_ld, s, pred)
                         : launch_bf16<64, false>(n_heads, L, q, k, vt, vt_ld, o, o_ld, s, pred);
    if (d == 128)
      return q_prescaled ? launch_bf16<128, true>(n_heads, L, q, k, vt, vt_ld, o, o_ld, s, pred)
                         : launch_bf16<128, false>(n_heads, L, q, k, vt, vt_ld, o, o_ld, s, pred);
  } else {
    if (d == 64) return launch_f32<64>(n_heads, L, q, k, vt, vt_ld, o, o_ld, s, pred, q_prescaled);
    if (d == 128) return launch_f32<128>(n_heads, L, q, k, vt, vt_ld, o, o_ld, s, pred, q_prescaled);
  }
  return hipErrorInvalidValue;
}

}  // namespace acid

// Fused GEMMs of the DiT block: y = a W + b with the epilogues the block
// needs (plain, tanh-GELU, gated residual add, QKV head split, Euler update).
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 (gfx950), fp32 accumulate.
//   Macro tile 256 (tokens) x 256 (features), K in steps of 64, 8 waves in a
//   2 x 4 grid (two per SIMD), each wave 128 x 64 = 4 x 2 MFMA blocks of
//   32 x 32.  Operands go global -> LDS directly (global_load_lds_dwordx4,
//   no staging registers) into a ring of 32 KB operand tiles (three for
//   the activations, requested about 1.75 K-steps ahead, two for the
//   weights, 1.25 ahead: 160 KB, the whole LDS), K-contiguous 128-byte rows
//   (whole cache lines, so the L2 request rate stays within budget) with an
//   XOR swizzle that is conflict-free for gfx950's 64 LDS banks.  One
//   barrier per K-step, placed before the last 16-wide sub-step so the
//   weight refill and the next stage's first fragment reads hide behind its
//   MFMAs (the activation refill runs under the first sub-step); all other
//   fragment reads are software-pipelined one sub-step ahead.  A wave that
//   issues global loads holds back its own MFMA issue, so two waves share
//   each SIMD and one of them issues the DMAs of both: the other only reads
//   fragments and issues MFMAs.  A 256 x 256 tile halves the operand bytes
//   per flop of a 256 x 128 tile (operand traffic also costs clock under
//   the power cap).  The activation tile feeds MFMA operand A and the weight
//   tile operand B, so the accumulator holds C with lanes along features:
//   every epilogue store is a run of consecutive features of one token row
//   (coalesced), and bias / gate are one value per lane.  Workgroups are
//   remapped so each XCD (8 per MI355X, own L2) works on a contiguous group
//   of tiles that share activation rows.
// fp32 path: a plain 64 x 64 register-blocked VALU kernel for the fp32
//   configuration (small shapes, latency-bound).
#include <atomic>
#include <type_traits>

#include "common.h"

namespace acid {

namespace {

struct Epi {
  const float* bias;
  const float* gate;
  void* out;
  float* v_out;
  void* q;
  void* k;
  void* vt;
  int64_t vt_ld;
  int64_t M;
  int n_heads, head_dim, H;
  float dsigma;
  const int32_t* pred;  // device gate's decision: no work when *pred == 0
  const float* bias2;   // GATE_RESIDUAL: optional second bias
  int64_t out_ld;       // QKV_GELU: row stride of the GELU output
  int n_qkv;            // QKV_GELU: columns [0, n_qkv) are Q | K | V
  float q_mul;          // QKV kinds: factor on the Q columns (1: plain Q)
  float* split_ws;      // bf16: fp32 partial tiles of a K split (nullptr: no split)
};

// Q | K | V head-major destination of column c < 3 H (which = c / H).
template <typename T>
__device__ __forceinline__ T* qkv_dst(const Epi& e, int c, int64_t& stride) {
  const int which = c / e.H, cc = c - which * e.H;
  const int head = cc / e.head_dim, dd = cc - head * e.head_dim;
  if (which < 2) {
    stride = e.head_dim;
    return static_cast<T*>(which == 0 ? e.q : e.k) + (int64_t)head * e.M * e.head_dim + dd;
  }
  stride = 1;
  return static_cast<T*>(e.vt) + ((int64_t)head * e.head_dim + dd) * e.vt_ld;
}

template <int KIND, typename T>
__device__ __forceinline__ void epi_elem(const Epi& e, int64_t m, int n, int N, float acc) {
  float bias = e.bias[n];
  if (KIND == ACID_EPI_GATE_RESIDUAL && e.bias2) bias += e.bias2[n];
  const float y = acc + bias;
  const int64_t idx = m * N + n;
  if constexpr (KIND == ACID_EPI_BIAS) {
    static_cast<float*>(e.out)[idx] = y;
  } else if constexpr (KIND == ACID_EPI_BIAS_GELU) {
    static_cast<T*>(e.out)[idx] = (T)gelu_tanh(y);
  } else if constexpr (KIND == ACID_EPI_GATE_RESIDUAL) {
    float* h = static_cast<float*>(e.out) + idx;
    *h = *h + e.gate[n] * y;
  } else if constexpr (KIND == ACID_EPI_QKV || KIND == ACID_EPI_QKV_GELU) {
    if (KIND == ACID_EPI_QKV || n < e.n_qkv) {
      int64_t stride;
      T* dst = qkv_dst<T>(e, n, stride);
      dst[m * stride] = (T)(n < e.H ? y * e.q_mul : y);
    } else {
      static_cast<T*>(e.out)[m * e.out_ld + (n - e.n_qkv)] = (T)gelu_tanh(y);
    }
  } else {  // ACID_EPI_EULER
    if (e.v_out) e.v_out[idx] = y;
    float* x = static_cast<float*>(e.out) + idx;
    *x = *x + e.dsigma * y;
  }
}

// Epilogue of one output column n: bias, gate and destination are resolved
// once; put(m, acc) then stores row m.
template <int KIND, typename T>
struct ColEpi {
  float bias, gate;
  T* dst_t;
  float* dst_f;
  float* v_f;
  int64_t stride;
  float dsigma;
  bool gelu;  // QKV_GELU: this column is in the GELU part
  float qmul;  // QKV kinds: e.q_mul on the Q columns, else 1
  __device__ __forceinline__ ColEpi(const Epi& e, int n, int N) {
    bias = e.bias[n];
    if (KIND == ACID_EPI_GATE_RESIDUAL && e.bias2) bias += e.bias2[n];
    gate = (KIND == ACID_EPI_GATE_RESIDUAL) ? e.gate[n] : 0.f;
    dsigma = e.dsigma;
    dst_t = nullptr;
    dst_f = nullptr;
    v_f = nullptr;
    stride = N;
    gelu = false;
    qmul = ((KIND == ACID_EPI_QKV || KIND == ACID_EPI_QKV_GELU) && n < e.H) ? e.q_mul : 1.f;
    if constexpr (KIND == ACID_EPI_QKV) {
      dst_t = qkv_dst<T>(e, n, stride);
    } else if constexpr (KIND == ACID_EPI_QKV_GELU) {
      if (n < e.n_qkv) {
        dst_t = qkv_dst<T>(e, n, stride);
      } else {
        gelu = true;
        dst_t = static_cast<T*>(e.out) + (n - e.n_qkv);
        stride = e.out_ld;
      }
    } else if constexpr (KIND == ACID_EPI_BIAS_GELU) {
      dst_t = static_cast<T*>(e.out) + n;
    } else {
      dst_f = static_cast<float*>(e.out) + n;
      if (KIND == ACID_EPI_EULER && e.v_out) v_f = e.v_out + n;
    }
  }
  static constexpr bool kRmw = KIND == ACID_EPI_GATE_RESIDUAL || KIND == ACID_EPI_EULER;
  // Read-modify-write kinds read the old value first (batched by the caller).
  __device__ __forceinline__ float old(int64_t m) const {
    if constexpr (kRmw) return dst_f[m * stride];
    return 0.f;
  }
  __device__ __forceinline__ void put_old(int64_t m, float acc, float prev) const {
    const float y = acc + bias;
    if constexpr (KIND == ACID_EPI_GATE_RESIDUAL) {
      dst_f[m * stride] = prev + gate * y;
    } else if constexpr (KIND == ACID_EPI_EULER) {
      if (v_f) v_f[m * stride] = y;
      dst_f[m * stride] = prev + dsigma * y;
    } else {
      put(m, acc);
    }
  }
  __device__ __forceinline__ void put(int64_t m, float acc) const {
    const float y = acc + bias;
    if constexpr (KIND == ACID_EPI_BIAS) {
      dst_f[m * stride] = y;
    } else if constexpr (KIND == ACID_EPI_BIAS_GELU) {
      if constexpr (sizeof(T) == 2)
        dst_t[m * stride] = (T)gelu_tanh_fast(y);
      else
        dst_t[m * stride] = (T)gelu_tanh(y);
    } else if constexpr (KIND == ACID_EPI_GATE_RESIDUAL) {
      float* h = dst_f + m * stride;
      *h = *h + gate * y;
    } else if constexpr (KIND == ACID_EPI_QKV) {
      dst_t[m * stride] = (T)(y * qmul);
    } else if constexpr (KIND == ACID_EPI_QKV_GELU) {
      float z = y * qmul;
      if (gelu) {
        if constexpr (sizeof(T) == 2)
          z = gelu_tanh_fast(y);
        else
          z = gelu_tanh(y);
      }
      dst_t[m * stride] = (T)z;
    } else {
      if (v_f) v_f[m * stride] = y;
      float* x = dst_f + m * stride;
      *x = *x + dsigma * y;
    }
  }
};

// Bijection from dispatch order to tile order giving XCD x (workgroups
// bid = x, x+8, ...) the contiguous tile range of its share.
__device__ __forceinline__ int64_t xcd_remap(int64_t bid, int64_t T) {
  constexpr int64_t NX = 8;
  const int64_t x = bid % NX, local = bid / NX;
  const int64_t q = T / NX, r = T % NX;
  return (x < r) ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

// Tile t -> (tm, tn) in groups of kGroupM token tiles, feature tiles inner.
// The 32 tiles an XCD runs at once then share few activation row blocks
// (streamed once from HBM) and many weight column blocks (re-read by every
// row block, so they come from the on-package cache): groups of 2 measured
// 3-6% faster than 8 on the model shapes here (4 and 3 within noise of 2).
constexpr int kGroupM = 2;
__device__ __forceinline__ void tile_coords(int64_t t, int64_t tiles_m, int tiles_n, int64_t& tm,
                                            int& tn) {
  const int64_t per_group = (int64_t)kGroupM * tiles_n;
  const int64_t g = t / per_group;
  const int64_t first = g * kGroupM;
  const int64_t gsize = min((int64_t)kGroupM, tiles_m - first);
  const int64_t w = t - g * per_group;
  tm = first + w % gsize;
  tn = (int)(w / gsize);
}

// ------------------------------------------------------------ bf16 MFMA

typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kWaves = 8;                // 2 (tokens) x 4 (features), two per SIMD
constexpr int kTileElems = 256 * BK;     // one operand tile per stage (32 KB)
constexpr int64_t kSplitItemFloats = 256 * 256;  // one K-split partial tile (256 KB)
constexpr int64_t kSplitMaxItems = 256;           // work items the split workspace holds

// One 16-byte-per-lane LDS-DMA: lane l reads 16 bytes at base + off(l) and
// writes LDS bytes [lds + 16 l, +16).  base and lds are wave-uniform.
// Issued as inline assembly so the compiler's wait-count pass does not see
// it (that pass cannot order DMA completions against LDS reads and would
// drain every read); completion is waited for explicitly.  M0 (the DMA's
// LDS base) is set here and nothing else in these kernels uses M0.
__device__ __forceinline__ void dma16(uint64_t base, uint32_t off_bytes, uint32_t lds_byte) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(off_bytes), "s"(base), "s"(lds_byte)
      : "memory");
}
__device__ __forceinline__ uint64_t uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ void wait_all() { __builtin_amdgcn_s_waitcnt(0); }

// Epilogue of one 256 x 256 tile: wave (wm, wn) stores its 128 x 64 block
// from the MFMA accumulators.
template <int KIND>
__device__ __forceinline__ void tile_epilogue(const Epi& e, f32x16 (&acc)[4][2], int64_t M,
                                              int N, int64_t m0, int n0, int wm, int wn,
                                              int lane) {
  const int lr = lane & 31, lg = lane >> 5;
  // D[i][j] of a 32x32 block: j = lane % 32, i = 8 (r / 4) + 4 (lane / 32) + r % 4.
  // A lane owns one feature column per 32-wide block: set up its epilogue
  // once, then handle its 64 rows of that column.  Full tiles skip the row
  // check (a per-element branch would serialise every load behind a wait);
  // read-modify-write kinds issue 32 loads before their stores.
  const bool full = m0 + BM <= M;
  const int64_t mrow = m0 + wm * 128 + 4 * lg;
  if constexpr (KIND == ACID_EPI_QKV || KIND == ACID_EPI_QKV_GELU) {
    // V columns are rows of V^T, whose tokens are contiguous: a lane holds 4
    // consecutive tokens per group r / 4 and its partner lane (l ^ 32) the
    // next 4, so one permlane32 swap per dword gives each lane 8 consecutive
    // tokens: 16-byte stores instead of 2-byte ones scattered over 32 rows.
    const int nw = n0 + wn * 64;
    if (full && nw >= 2 * e.H && nw + 64 <= 3 * e.H) {  // all 64 columns in V
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const int n = nw + nb * 32 + lr;
        const int cc = n - 2 * e.H;
        const int head = cc / e.head_dim, dd = cc - head * e.head_dim;
        bf16* vrow = static_cast<bf16*>(e.vt) + ((int64_t)head * e.head_dim + dd) * e.vt_ld;
        const float bias = e.bias[n];
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
          uint32_t w[8];  // tokens 8 (r / 4) + 4 lg + r % 4 as bf16 pairs
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            const bf16x2 pr = {(bf16)(acc[mb][nb][r] + bias), (bf16)(acc[mb][nb][r + 1] + bias)};
            w[r / 2] = __builtin_bit_cast(uint32_t, pr);
          }
          const int64_t t0 = m0 + wm * 128 + mb * 32 + 8 * lg;
#pragma unroll
          for (int p = 0; p < 2; ++p) {  // groups 2p (tokens +0..7) and 2p + 1 (+8..15)
            uint32_t lo[2], hi[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const auto sw = __builtin_amdgcn_permlane32_swap(w[4 * p + h], w[4 * p + 2 + h],
                                                               false, false);
              lo[h] = sw[0];
              hi[h] = sw[1];
            }
            const u32x4 v = {lo[0], lo[1], hi[0], hi[1]};
            *reinterpret_cast<u32x4*>(vrow + t0 + 16 * p) = v;
          }
        }
      }
      return;
    }
  }
  if constexpr (!ColEpi<KIND, bf16>::kRmw) {
    if (full) {
      // The two 32-column blocks of a wave fill the two halves of the same
      // 128-byte line of each output row (bf16): store them back to back so
      // the line is complete in the L2 before it can be written back.
      const ColEpi<KIND, bf16> c0(e, n0 + wn * 64 + lr, N), c1(e, n0 + wn * 64 + 32 + lr, N);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t m = mrow + mb * 32 + 8 * (r >> 2) + (r & 3);
          c0.put(m, acc[mb][0][r]);
          c1.put(m, acc[mb][1][r]);
        }
      return;
    }
    // The ragged last row tile: row offsets from mrow in 32 bits (a 64-bit
    // row per element made the register allocator spill).
    const int rows_left = (int)(M - mrow < 128 ? M - mrow : 128);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const ColEpi<KIND, bf16> ce(e, n0 + wn * 64 + nb * 32 + lr, N);
      // The column's bias has landed before the guarded stores: a load still
      // in flight there makes every guarded block wait for all earlier stores.
      asm volatile("" ::"v"(ce.bias));
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int dr = mb * 32 + 8 * (r >> 2) + (r & 3);
          if (dr < rows_left) ce.put(mrow + dr, acc[mb][nb][r]);
        }
    }
    return;
  }
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + wn * 64 + nb * 32 + lr;
    ColEpi<KIND, bf16> ce(e, n, N);
    if (full) {
      if constexpr (ColEpi<KIND, bf16>::kRmw) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {  // 32 loads in flight, then 32 stores
          float prev[2][16];
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              prev[mb][r] = ce.old(mrow + (2 * h + mb) * 32 + 8 * (r >> 2) + (r & 3));
#pragma unroll
          for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              ce.put_old(mrow + (2 * h + mb) * 32 + 8 * (r >> 2) + (r & 3),
                         acc[2 * h + mb][nb][r], prev[mb][r]);
        }
      } else {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            ce.put(mrow + mb * 32 + 8 * (r >> 2) + (r & 3), acc[mb][nb][r]);
      }
    } else {
      // The ragged last row tile of a read-modify-write kind: loads from rows
      // clamped to M - 1 (always valid) batched as above, stores guarded.  A
      // load under the store's guard would wait for each element in turn.
      const int rows_left = (int)(M - mrow < 128 ? M - mrow : 128);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float prev[2][16];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int dr = (2 * h + mb) * 32 + 8 * (r >> 2) + (r & 3);
            prev[mb][r] = ce.old(dr < rows_left ? mrow + dr : M - 1);
          }
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) asm volatile("" ::"v"(prev[mb][r]));  // loads land here
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int dr = (2 * h + mb) * 32 + 8 * (r >> 2) + (r & 3);
            if (dr < rows_left) ce.put_old(mrow + dr, acc[2 * h + mb][nb][r], prev[mb][r]);
          }
      }
    }
  }
}

// Operand tiles are 256 rows x 64 (K-contiguous 128-byte rows: every row
// fetch is one whole line).  DMA instruction i (0..3) of wave w fills LDS
// bytes [(4 w + i) KB, +1 KB) = rows 32 w + 8 i .. +7; lane l lands in row
// 32 w + 8 i + l / 8, slot l % 8, which holds global chunk
// (l % 8) ^ ((row / 2) % 8) (= (l % 8) ^ (l / 16) for even i, ^ 4 more for
// odd i).  With 64 four-byte LDS banks a row spans half the banks, so 16
// consecutive fragment rows read at one chunk cover all 64 banks once.
//
// Eight waves, two per SIMD (waves w and w + 4): wave w issues the DMAs of
// both (a wave that issues global loads holds back its own MFMA issue), so
// wave w + 4 keeps the MFMA unit busy while wave w stalls.  Each wave owns
// 128 x 64 of the tile (4 x 2 blocks of 32 x 32, 128 accumulator registers).
//
// K split (grids whose last round of tiles would leave most CUs idle): the
// first tiles_main work items are whole tiles in the XCD-aware order; each of
// the remaining tiles is split into `split` equal K ranges, one work item
// each, which store their raw fp32 partial sums to e.split_ws for
// gemm_split_reduce_kernel.
template <int KIND>
__global__ __launch_bounds__(64 * kWaves, 1) void gemm_bf16_kernel(const bf16* A, const bf16* Wt,
                                                                   int64_t M, int N, int K,
                                                                   Epi e, int64_t tiles_main,
                                                                   int split) {
  if (e.pred && *e.pred == 0) return;
  // Three A tiles and two B tiles, one LDS object per tile so the compiler
  // can tell the tile being read from the tile being filled.
  __shared__ __attribute__((aligned(1024))) bf16 As0[kTileElems], Bs0[kTileElems];
  __shared__ __attribute__((aligned(1024))) bf16 As1[kTileElems], Bs1[kTileElems];
  __shared__ __attribute__((aligned(1024))) bf16 As2[kTileElems];

  const int tiles_n = (N + BN - 1) / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  int64_t tm;
  int tn;
  int64_t item = -1;  // K-split work item, or -1 for a whole tile
  int kbeg = 0, klen = K;
  if ((int64_t)blockIdx.x < tiles_main) {
    tile_coords(xcd_remap(blockIdx.x, tiles_main), tiles_m, tiles_n, tm, tn);
  } else {
    item = (int64_t)blockIdx.x - tiles_main;
    klen = K / split;
    kbeg = (int)(item % split) * klen;
    tile_coords(tiles_main + item / split, tiles_m, tiles_n, tm, tn);
  }
  const int64_t m0 = tm * BM;
  const int n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const int lr = lane & 31, lg = lane >> 5;
  // A tile of width 128 at the right edge (N % 256 == 128): waves with
  // wn >= 2 compute on clamped rows and store nothing.
  const bool active = n0 + wn * 64 < N;

  // Load-side addressing: byte offsets from the tile's first row (rows past
  // the edge are clamped; they only feed outputs that are never stored).
  // The K offset of a stage is added to the scalar base, so the per-lane
  // offsets stay fixed and a DMA needs no vector arithmetic.  Waves w and
  // w + 4 share a SIMD: wave w (< 4) issues the DMAs of both (DMA i < 4 its
  // own rows, i >= 4 those of wave w + 4), so wave w + 4 issues MFMAs only.
  const bool dma_wave = wave < 4;
  const int chunk_even = (lane & 7) ^ (lane >> 4);
  const int chunk_odd = (lane & 7) ^ ((lane >> 4) ^ 4);
  const uint64_t a_base = uniform_ptr(A + m0 * K + kbeg);
  const uint64_t b_base = uniform_ptr(Wt + (int64_t)n0 * K + kbeg);
  uint32_t a_off[8], b_off[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int ww = (wave & 3) + (i >> 2) * 4;
    const int r = ww * 32 + (i & 3) * 8 + (lane >> 3);
    const int ra = m0 + r < M ? r : (int)(M - 1 - m0);
    const int rb = n0 + r < N ? r : N - 1 - n0;
    const int ch = (i & 1) ? chunk_odd : chunk_even;
    a_off[i] = (uint32_t)(ra * K + ch * 8) * 2u;
    b_off[i] = (uint32_t)(rb * K + ch * 8) * 2u;
  }
  auto tile_lds = [&](const bf16* tile) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)tile);
  };
  auto lds_slot = [&](int i) {
    return (uint32_t)((((wave & 3) + (i >> 2) * 4) * 4 + (i & 3)) * 1024);
  };

  // Read-side addressing: fragment row rr at K-step kk (16 wide) reads chunk
  // 2 kk + lg, stored at slot (2 kk + lg) ^ ((rr / 2) % 8), and
  // (rr / 2) % 8 == (lr / 2) % 8 for every fragment row of this lane.
  const int a_rbase = (wm * 128 + lr) * BK;
  const int b_rbase = (wn * 64 + lr) * BK;
  int sl[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) sl[kk] = 8 * ((2 * kk + lg) ^ ((lr >> 1) & 7));

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  bf16x8 fa0[4], fb0[2], fa1[4], fb1[2];
  auto read_frags = [&](const bf16* As, const bf16* Bs, int slot, bf16x8(&fa)[4],
                        bf16x8(&fb)[2]) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      fa[mb] = *reinterpret_cast<const bf16x8*>(As + a_rbase + mb * 32 * BK + slot);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
      fb[nb] = *reinterpret_cast<const bf16x8*>(Bs + b_rbase + nb * 32 * BK + slot);
  };
  auto mma = [&](const bf16x8(&fa)[4], const bf16x8(&fb)[2]) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[mb], fb[nb], acc[mb][nb], 0, 0, 0);
  };
  auto load_stage = [&](const bf16* As, const bf16* Bs, int k0) {
    const uint32_t la = tile_lds(As), lb = tile_lds(Bs);
#pragma unroll
    for (int i = 0; i < 8; ++i) dma16(a_base + (uint32_t)(k0 * 2), a_off[i], la + lds_slot(i));
#pragma unroll
    for (int i = 0; i < 8; ++i) dma16(b_base + (uint32_t)(k0 * 2), b_off[i], lb + lds_slot(i));
  };
  // One DMA after each of the 8 MFMAs of a K-step (order pinned by
  // scheduling barriers): the 8 DMAs that fill tile T at K offset k0.
  auto mma_dma = [&](const bf16x8(&fa)[4], const bf16x8(&fb)[2], const bf16* T,
                     uint64_t base, const uint32_t(&off)[8], int k0) {
    const uint32_t lt = tile_lds(T);
    const uint64_t bk = base + (uint32_t)(k0 * 2);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[mb], fb[nb], acc[mb][nb], 0, 0, 0);
        const int i = mb * 2 + nb;
        dma16(bk, off[i], lt + lds_slot(i));
        __builtin_amdgcn_sched_barrier(0);
      }
  };

  const int KT = klen / BK;  // even: K and each split's K range are multiples of 128
  auto kc = [&](int k) { return (k < KT ? k : KT - 1) * BK; };
  // Three A stages and two B stages (160 KB).  Stage kt refills A with
  // stage kt + 2 during its first K-step (the buffer stage kt - 1 read) and
  // B with stage kt + 2 during its last (the buffer it has just read), one
  // DMA per MFMA, so the activations, streamed from HBM, are requested about
  // 1.75 stages ahead of use and the weights 1.25.  Prologue: A 0, B 0, A 1,
  // B 1 (32 DMAs in a DMA wave); stage 0 landed (vmcnt 16; a wave without
  // DMAs has nothing outstanding).
  auto main_loop = [&](auto dma_flag) {
    constexpr bool kDma = decltype(dma_flag)::value;
    if constexpr (kDma) {
      load_stage(As0, Bs0, 0);
      load_stage(As1, Bs1, kc(1));
    }
    __builtin_amdgcn_s_waitcnt((16 & 15) | (7 << 4) | (15 << 8) | ((16 >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    read_frags(As0, Bs0, sl[0], fa0, fb0);

    // Stage kt reads A[kt % 3], B[kt % 2].  At its barrier the DMAs of this
    // stage's first K-step (A of stage kt + 2) may still be in flight, those
    // of stage kt + 1 (A in stage kt - 1, B in stage kt - 1's last K-step)
    // have landed: vmcnt(8).
    int kt = 0;
#define GEMM_STAGE(AS, BS, AN, BN_, AP)                                          \
  {                                                                            \
    read_frags(AS, BS, sl[1], fa1, fb1);                                       \
    __builtin_amdgcn_sched_barrier(0);                                         \
    if constexpr (kDma)                                                        \
      mma_dma(fa0, fb0, AP, a_base, a_off, kc(kt + 2));                        \
    else                                                                       \
      mma(fa0, fb0);                                                           \
    __builtin_amdgcn_sched_barrier(0);                                         \
    read_frags(AS, BS, sl[2], fa0, fb0);                                       \
    __builtin_amdgcn_sched_barrier(0);                                         \
    mma(fa1, fb1);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                         \
    read_frags(AS, BS, sl[3], fa1, fb1);                                       \
    __builtin_amdgcn_sched_barrier(0);                                         \
    mma(fa0, fb0);                                                             \
    __builtin_amdgcn_sched_barrier(0);                                         \
    __builtin_amdgcn_s_waitcnt(8 | (7 << 4) | (0 << 8));                       \
    __builtin_amdgcn_s_barrier();                                              \
    read_frags(AN, BN_, sl[0], fa0, fb0);                                      \
    __builtin_amdgcn_sched_barrier(0);                                         \
    if constexpr (kDma)                                                        \
      mma_dma(fa1, fb1, BS, b_base, b_off, kc(kt + 2));                        \
    else                                                                       \
      mma(fa1, fb1);                                                           \
    __builtin_amdgcn_sched_barrier(0);                                         \
    ++kt;                                                                      \
  }
    while (kt + 6 <= KT) {
      GEMM_STAGE(As0, Bs0, As1, Bs1, As2)
      GEMM_STAGE(As1, Bs1, As2, Bs0, As0)
      GEMM_STAGE(As2, Bs0, As0, Bs1, As1)
      GEMM_STAGE(As0, Bs1, As1, Bs0, As2)
      GEMM_STAGE(As1, Bs0, As2, Bs1, As0)
      GEMM_STAGE(As2, Bs1, As0, Bs0, As1)
    }
    if (kt + 2 <= KT) {
      GEMM_STAGE(As0, Bs0, As1, Bs1, As2)
      GEMM_STAGE(As1, Bs1, As2, Bs0, As0)
    }
    if (kt + 2 <= KT) {
      GEMM_STAGE(As2, Bs0, As0, Bs1, As1)
      GEMM_STAGE(As0, Bs1, As1, Bs0, As2)
    }
#undef GEMM_STAGE
  };
  if (dma_wave)
    main_loop(std::true_type{});
  else
    main_loop(std::false_type{});
  wait_all();  // the last refill lands before the workgroup's LDS is released
  if (!active) return;
  if (item >= 0) {
    // Partial sums of this K range: value q of thread tid at (q * 512 + tid)
    // float4s into the item's 256 KB (consecutive threads, consecutive 16 B).
    f32x4* dst = reinterpret_cast<f32x4*>(e.split_ws) + item * (kSplitItemFloats / 4);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int q = (mb * 2 + nb) * 4 + r4;
          dst[q * 64 * kWaves + tid] = f32x4{acc[mb][nb][4 * r4], acc[mb][nb][4 * r4 + 1],
                                             acc[mb][nb][4 * r4 + 2], acc[mb][nb][4 * r4 + 3]};
        }
    return;
  }
  tile_epilogue<KIND>(e, acc, M, N, m0, n0, wm, wn, lane);
}

// The split tiles: partial sums added in split order (deterministic), then
// the tile's epilogue.  Work item b reduces tile tiles_main + b.
template <int KIND>
__global__ __launch_bounds__(64 * kWaves, 1) void gemm_split_reduce_kernel(int64_t M, int N, Epi e,
                                                                           int64_t tiles_main,
                                                                           int split) {
  if (e.pred && *e.pred == 0) return;
  const int tiles_n = (N + BN - 1) / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  int64_t tm;
  int tn;
  tile_coords(tiles_main + blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int64_t m0 = tm * BM;
  const int n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  if (!(n0 + wn * 64 < N)) return;
  const f32x4* src = reinterpret_cast<const f32x4*>(e.split_ws) +
                     (int64_t)blockIdx.x * split * (kSplitItemFloats / 4);
  f32x16 acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int q = (mb * 2 + nb) * 4 + r4;
        f32x4 v = src[q * 64 * kWaves + tid];
        for (int sp = 1; sp < split; ++sp)
          v += src[sp * (kSplitItemFloats / 4) + q * 64 * kWaves + tid];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[mb][nb][4 * r4 + i] = v[i];
      }
  tile_epilogue<KIND>(e, acc, M, N, m0, n0, wm, wn, lane);
}

// ------------------------------------------------------------ fp32 VALU

template <int KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ Wt, int64_t M,
                                                       int N, int K, Epi e) {
  if (e.pred && *e.pred == 0) return;
  __shared__ float As[16][64 + 4];
  __shared__ float Ws[16][64 + 4];
  const int64_t m0 = (int64_t)blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    const int64_t gm = m0 + lrow;
    float4 a = gm < M ? *reinterpret_cast<const float4*>(A + gm * K + k0 + lk)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 w = *reinterpret_cast<const float4*>(Wt + (int64_t)(n0 + lrow) * K + k0 + lk);
    As[lk + 0][lrow] = a.x;
    As[lk + 1][lrow] = a.y;
    As[lk + 2][lrow] = a.z;
    As[lk + 3][lrow] = a.w;
    Ws[lk + 0][lrow] = w.x;
    Ws[lk + 1][lrow] = w.y;
    Ws[lk + 2][lrow] = w.z;
    Ws[lk + 3][lrow] = w.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float4 a4 = *reinterpret_cast<const float4*>(&As[k][ty * 4]);
      float4 w4 = *reinterpret_cast<const float4*>(&Ws[k][tx * 4]);
      const float av[4] = {a4.x, a4.y, a4.z, a4.w};
      const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * wv[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) epi_elem<KIND, float>(e, m, n0 + tx * 4 + j, N, acc[i][j]);
  }
}

// K split of the last round's tiles: when the tiles beyond whole rounds of
// the device's CUs would leave at least half of them idle, those `rem` tiles
// are split into S K ranges (S <= 8, S * rem within the CUs and the 256 work
// items the workspace holds, each range a multiple of 128).  Each range is at
// least 2048 long: a work item also fills the staging ring and writes its
// 256 KB of partial sums, which the reduction reads back, and with shorter
// ranges that costs more than the fuller round saves (measured: split into
// K ranges of 256-1024, the small configuration's GEMMs ran twice as long).
int cu_count() {
  static std::atomic<int> cus{0};
  int c = cus.load(std::memory_order_relaxed);
  if (c == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c < 1)
      c = 256;
    cus.store(c, std::memory_order_relaxed);
  }
  return c;
}
int choose_split(int64_t tiles, int K, int64_t& rem) {
  const int cus = cu_count();
  rem = tiles % cus;
  if (rem == 0 || 2 * rem > cus) return 1;
  int S = (int)(cus / rem);
  if (S > 8) S = 8;
  while (S > 1 && (rem * S > kSplitMaxItems || K % (S * 128) != 0 || K / S < 2048)) --S;
  return S;
}

template <int KIND>
hipError_t launch_kind(int dtype, int64_t M, int N, int K, const void* a, const void* wt,
                       const Epi& e, hipStream_t s) {
  if (dtype == ACID_BF16) {
    const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    int64_t rem = 0;
    const int split = e.split_ws ? choose_split(tiles, K, rem) : 1;
    const int64_t tiles_main = tiles - (split > 1 ? rem : 0);
    const int64_t grid = tiles_main + (split > 1 ? rem * split : 0);
    hipLaunchKernelGGL(gemm_bf16_kernel<KIND>, dim3((unsigned)grid), dim3(64 * kWaves), 0, s,
                       (const bf16*)a, (const bf16*)wt, M, N, K, e, tiles_main, split);
    if (split > 1) {
      const hipError_t err = hipGetLastError();
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL(gemm_split_reduce_kernel<KIND>, dim3((unsigned)rem), dim3(64 * kWaves),
                         0, s, M, N, e, tiles_main, split);
    }
  } else {
    dim3 grid((unsigned)((M + 63) / 64), (unsigned)(N / 64));
    hipLaunchKernelGGL(gemm_f32_kernel<KIND>, grid, dim3(256), 0, s, (const float*)a,
                       (const float*)wt, M, N, K, e);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_linear(int dtype, int64_t M, int N, int K, const void* a, const void* wt,
                         const acid_epilogue_args& ea, hipStream_t s, const int32_t* pred,
                         float* split_ws) {
  if (M == 0) return hipSuccess;
  Epi e;
  e.split_ws = dtype == ACID_BF16 ? split_ws : nullptr;
  e.bias = ea.bias;
  e.gate = ea.gate;
  e.out = ea.out;
  e.v_out = ea.v_out;
  e.q = ea.q;
  e.k = ea.k;
  e.vt = ea.vt;
  e.vt_ld = ea.vt_ld;
  e.M = M;
  e.n_heads = ea.n_heads;
  e.head_dim = ea.head_dim;
  e.H = ea.n_heads * ea.head_dim;
  e.dsigma = ea.dsigma;
  e.pred = pred;
  e.bias2 = ea.bias2;
  e.out_ld = ea.out_ld;
  e.n_qkv = 3 * ea.n_heads * ea.head_dim;
  e.q_mul = ea.q_prescale ? attn_q_scale(ea.head_dim) : 1.f;
  switch (ea.kind) {
    case ACID_EPI_BIAS: return launch_kind<ACID_EPI_BIAS>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_BIAS_GELU: return launch_kind<ACID_EPI_BIAS_GELU>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_GATE_RESIDUAL:
      return launch_kind<ACID_EPI_GATE_RESIDUAL>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_QKV: return launch_kind<ACID_EPI_QKV>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_EULER: return launch_kind<ACID_EPI_EULER>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_QKV_GELU: return launch_kind<ACID_EPI_QKV_GELU>(dtype, M, N, K, a, wt, e, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace acid

// Fused GEMMs of the DiT block: y = a W + b with the epilogues the block
// needs (plain, tanh-GELU, gated residual add, QKV head split, Euler update).
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 (gfx950), fp32 accumulate.
//   Macro tile 256 (tokens) x 128 (features) x 64 (K), 4 waves in a 2x2
//   grid, each wave 128 x 64 = 4 x 2 MFMA blocks of 32 x 32.  Both operands
//   are staged K-contiguous in LDS (rows padded by 16 bytes so that a
//   half-wave's 16-byte fragment reads hit distinct banks), double-buffered
//   with register prefetch so global loads of tile k+1 overlap the MFMAs of
//   tile k, one barrier per K step.  The activation tile feeds MFMA operand A
//   and the weight tile operand B, so the accumulator holds C with lanes
//   along features: every epilogue store is a run of consecutive features of
//   one token row (coalesced), and bias / gate are one value per lane.
//   Workgroups are remapped so each XCD (8 per MI355X, own L2) works on a
//   contiguous group of tiles that share activation rows.
// fp32 path: a plain 64 x 64 register-blocked VALU kernel for the fp32
//   configuration (small shapes, latency-bound).
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
};

template <int KIND, typename T>
__device__ __forceinline__ void epi_elem(const Epi& e, int64_t m, int n, int N, float acc) {
  const float y = acc + e.bias[n];
  const int64_t idx = m * N + n;
  if constexpr (KIND == ACID_EPI_BIAS) {
    static_cast<float*>(e.out)[idx] = y;
  } else if constexpr (KIND == ACID_EPI_BIAS_GELU) {
    static_cast<T*>(e.out)[idx] = (T)gelu_tanh(y);
  } else if constexpr (KIND == ACID_EPI_GATE_RESIDUAL) {
    float* h = static_cast<float*>(e.out) + idx;
    *h = *h + e.gate[n] * y;
  } else if constexpr (KIND == ACID_EPI_QKV) {
    const int which = n / e.H, c = n - which * e.H;
    const int head = c / e.head_dim, dd = c - head * e.head_dim;
    if (which < 2) {
      T* dst = static_cast<T*>(which == 0 ? e.q : e.k);
      dst[((int64_t)head * e.M + m) * e.head_dim + dd] = (T)y;
    } else {
      static_cast<T*>(e.vt)[((int64_t)head * e.head_dim + dd) * e.vt_ld + m] = (T)y;
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
  __device__ __forceinline__ ColEpi(const Epi& e, int n, int N) {
    bias = e.bias[n];
    gate = (KIND == ACID_EPI_GATE_RESIDUAL) ? e.gate[n] : 0.f;
    dsigma = e.dsigma;
    dst_t = nullptr;
    dst_f = nullptr;
    v_f = nullptr;
    stride = N;
    if constexpr (KIND == ACID_EPI_QKV) {
      const int which = n / e.H, c = n - which * e.H;
      const int head = c / e.head_dim, dd = c - head * e.head_dim;
      if (which < 2) {
        dst_t = static_cast<T*>(which == 0 ? e.q : e.k) + (int64_t)head * e.M * e.head_dim + dd;
        stride = e.head_dim;
      } else {
        dst_t = static_cast<T*>(e.vt) + ((int64_t)head * e.head_dim + dd) * e.vt_ld;
        stride = 1;
      }
    } else if constexpr (KIND == ACID_EPI_BIAS_GELU) {
      dst_t = static_cast<T*>(e.out) + n;
    } else {
      dst_f = static_cast<float*>(e.out) + n;
      if (KIND == ACID_EPI_EULER && e.v_out) v_f = e.v_out + n;
    }
  }
  __device__ __forceinline__ void put(int64_t m, float acc) const {
    const float y = acc + bias;
    if constexpr (KIND == ACID_EPI_BIAS) {
      dst_f[m * stride] = y;
    } else if constexpr (KIND == ACID_EPI_BIAS_GELU) {
      dst_t[m * stride] = (T)gelu_tanh(y);
    } else if constexpr (KIND == ACID_EPI_GATE_RESIDUAL) {
      float* h = dst_f + m * stride;
      *h = *h + gate * y;
    } else if constexpr (KIND == ACID_EPI_QKV) {
      dst_t[m * stride] = (T)y;
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
constexpr int kGroupM = 8;
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

constexpr int BM = 256, BN = 128, BK = 64, LDK = BK + 8;
constexpr int kLdsA = BM * LDK, kLdsB = BN * LDK;  // elements per buffer
constexpr size_t kGemmLds = (size_t)2 * (kLdsA + kLdsB) * sizeof(bf16);

template <int KIND>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(const bf16* A,
                                                           const bf16* Wt,
                                                           int64_t M, int N, int K, Epi e) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* As = reinterpret_cast<bf16*>(smem);
  bf16* Bs = As + 2 * kLdsA;

  const int tiles_n = N / BN;
  const int64_t tiles_m = (M + BM - 1) / BM;
  int64_t tm;
  int tn;
  tile_coords(xcd_remap(blockIdx.x, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
  const int64_t m0 = tm * BM;
  const int n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 31, lg = lane >> 5;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Global -> register staging.  Rows past M read row M-1 (a valid address)
  // and are zeroed by value, so every load is an unconditional global load.
  const int srow = tid >> 3, skc = tid & 7;  // row (+32 i) and 16-byte chunk
  const bf16* a_src[8];
  uint32_t a_mask[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t gm = m0 + srow + 32 * i;
    a_mask[i] = gm < M ? 0xFFFFFFFFu : 0u;
    a_src[i] = A + (gm < M ? gm : M - 1) * K + skc * 8;
  }
  const bf16* b_src = Wt + (int64_t)(n0 + srow) * K + skc * 8;
  u32x4 ra[8], rb[4];

#define GEMM_GLOAD(K0)                                                              \
  do {                                                                              \
    _Pragma("unroll") for (int i = 0; i < 8; ++i) {                                 \
      ra[i] = *reinterpret_cast<const u32x4*>(a_src[i] + (K0));                     \
    }                                                                               \
    _Pragma("unroll") for (int i = 0; i < 4; ++i)                                   \
      rb[i] = *reinterpret_cast<const u32x4*>(b_src + (int64_t)32 * i * K + (K0));  \
  } while (0)
#define GEMM_SSTORE(BUF)                                                            \
  do {                                                                              \
    bf16* as_ = As + (BUF) * kLdsA + srow * LDK + skc * 8;                          \
    bf16* bs_ = Bs + (BUF) * kLdsB + srow * LDK + skc * 8;                          \
    _Pragma("unroll") for (int i = 0; i < 8; ++i)                                   \
      *reinterpret_cast<u32x4*>(as_ + 32 * i * LDK) = ra[i] & a_mask[i];            \
    _Pragma("unroll") for (int i = 0; i < 4; ++i)                                   \
      *reinterpret_cast<u32x4*>(bs_ + 32 * i * LDK) = rb[i];                        \
  } while (0)

  GEMM_GLOAD(0);
  GEMM_SSTORE(0);
  __syncthreads();
  const int KT = K / BK;
  // The prefetch is unconditional (the last step reloads its own tile into
  // the idle buffer) so the loop body has no branches and the staging
  // registers stay in registers; masks are applied when writing LDS, after
  // the MFMAs, so no wait on the loads is forced early.
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    GEMM_GLOAD((kt + 1 < KT ? kt + 1 : kt) * BK);
    asm volatile("" ::: "memory");     // no IR pass may sink the prefetch
    __builtin_amdgcn_sched_barrier(0);  // nor the machine scheduler
    const bf16* Ab = As + buf * kLdsA + (wm * 128 + lr) * LDK + lg * 8;
    const bf16* Bb = Bs + buf * kLdsB + (wn * 64 + lr) * LDK + lg * 8;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[4], bfr[2];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        af[mb] = *reinterpret_cast<const bf16x8*>(Ab + mb * 32 * LDK + kk * 16);
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        bfr[nb] = *reinterpret_cast<const bf16x8*>(Bb + nb * 32 * LDK + kk * 16);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mb], bfr[nb], acc[mb][nb], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);  // masks and LDS writes after the MFMAs
    GEMM_SSTORE(buf ^ 1);
    __syncthreads();
  }
#undef GEMM_GLOAD
#undef GEMM_SSTORE

  // D[i][j] of a 32x32 block: j = lane % 32, i = 8 (r / 4) + 4 (lane / 32) + r % 4.
  // A lane owns one feature column per 32-wide block: set up its epilogue once.
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int n = n0 + wn * 64 + nb * 32 + lr;
    ColEpi<KIND, bf16> ce(e, n, N);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * 128 + mb * 32 + 8 * (r >> 2) + 4 * lg + (r & 3);
        if (m < M) ce.put(m, acc[mb][nb][r]);
      }
  }
}

// ------------------------------------------------------------ fp32 VALU

template <int KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ Wt, int64_t M,
                                                       int N, int K, Epi e) {
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

template <int KIND>
hipError_t launch_kind(int dtype, int64_t M, int N, int K, const void* a, const void* wt,
                       const Epi& e, hipStream_t s) {
  if (dtype == ACID_BF16) {
    static bool attr_set = false;
    if (!attr_set) {
      hipError_t err = hipFuncSetAttribute((const void*)gemm_bf16_kernel<KIND>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)kGemmLds);
      if (err != hipSuccess) return err;
      attr_set = true;
    }
    const int64_t tiles = ((M + BM - 1) / BM) * (N / BN);
    hipLaunchKernelGGL(gemm_bf16_kernel<KIND>, dim3((unsigned)tiles), dim3(256), kGemmLds, s,
                       (const bf16*)a, (const bf16*)wt, M, N, K, e);
  } else {
    dim3 grid((unsigned)((M + 63) / 64), (unsigned)(N / 64));
    hipLaunchKernelGGL(gemm_f32_kernel<KIND>, grid, dim3(256), 0, s, (const float*)a,
                       (const float*)wt, M, N, K, e);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_linear(int dtype, int64_t M, int N, int K, const void* a, const void* wt,
                         const acid_epilogue_args& ea, hipStream_t s) {
  if (M == 0) return hipSuccess;
  Epi e;
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
  switch (ea.kind) {
    case ACID_EPI_BIAS: return launch_kind<ACID_EPI_BIAS>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_BIAS_GELU: return launch_kind<ACID_EPI_BIAS_GELU>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_GATE_RESIDUAL:
      return launch_kind<ACID_EPI_GATE_RESIDUAL>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_QKV: return launch_kind<ACID_EPI_QKV>(dtype, M, N, K, a, wt, e, s);
    case ACID_EPI_EULER: return launch_kind<ACID_EPI_EULER>(dtype, M, N, K, a, wt, e, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace acid

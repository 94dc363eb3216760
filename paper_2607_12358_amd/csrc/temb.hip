// Timestep conditioning: sinusoidal embedding of t = 1000 sigma and the small
// fp32 matrix products that turn it into the adaLN modulation table.
//
// This runs once per denoise loop for all noise levels at once, so the
// products have few rows (the step count) and are bound by reading the
// fp32 adaLN weights (1.7 GB at the Wan-1.3B shape) once.
#include "common.h"

namespace acid {

namespace {

constexpr int kMaxSig = 128;
struct SigmaPack {
  float v[kMaxSig];
};

__global__ void sinusoid_kernel(SigmaPack sig, int n, int freq_dim, float* __restrict__ e) {
  const int i = blockIdx.x;
  if (i >= n) return;
  const int half = freq_dim / 2;
  const double t = 1000.0 * (double)sig.v[i];
  const double lnp = 9.210340371976184;  // ln(10000)
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    double f = exp(-lnp * (double)j / (double)half);
    double a = t * f;
    e[(int64_t)i * freq_dim + j] = (float)cos(a);
    e[(int64_t)i * freq_dim + half + j] = (float)sin(a);
  }
}

constexpr int kKChunk = 64;   // K rows of X staged per LDS round
constexpr int kColsPerBlock = 128;  // two columns per lane, 64 lanes

// Y[s][n] = act(sum_k X[s][k] W[k][n] + b[n]) for up to R rows s per block.
// Lane l of every wave owns columns 2l, 2l+1 of the block's 128; the four
// waves split K (wave w takes the rows k = 4j + w of each staged chunk), so
// each wave keeps 16 independent float2 loads of W in flight per chunk and
// W is read once for all R rows.  The waves' partial sums meet in LDS and
// are added in a fixed order (deterministic).
template <int R>
__global__ __launch_bounds__(256) void skinny_gemm_kernel(
    const float* __restrict__ X, int ldx, int S, int K, const float* __restrict__ W, int N,
    const float* __restrict__ bias, float* __restrict__ Y, int64_t ldy, int act_out,
    int64_t w_stride, int64_t b_stride, int64_t y_stride) {
  // X chunk [kKChunk][R] during the K loop; [4 waves][16 rows][128 cols]
  // partial sums during the reduction (32 KB).
  __shared__ __attribute__((aligned(16))) float lds[4 * 16 * kColsPerBlock];
  static_assert(kKChunk * R <= 4 * 16 * kColsPerBlock, "X chunk must fit");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cb = blockIdx.x * kColsPerBlock;
  const int c = cb + 2 * lane;
  const int g = blockIdx.y;
  const int s0 = blockIdx.z * R;
  const int rows = min(R, S - s0);
  const float* Wg = W + g * w_stride;
  const float* bg = bias + g * b_stride;
  float* Yg = Y + g * y_stride;
  const bool col_ok = c < N;  // N is even, so c + 1 < N too
  float acc[R][2];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r][0] = acc[r][1] = 0.f;
  for (int k0 = 0; k0 < K; k0 += kKChunk) {
    const int kend = min(kKChunk, K - k0);
    __syncthreads();
    for (int idx = tid; idx < kKChunk * R; idx += 256) {
      const int kk = idx / R, r = idx % R;
      lds[idx] = (r < rows && kk < kend) ? X[(int64_t)(s0 + r) * ldx + k0 + kk] : 0.f;
    }
    __syncthreads();
    if (col_ok) {
      float2 w[kKChunk / 4];
#pragma unroll
      for (int j = 0; j < kKChunk / 4; ++j) {
        const int kk = 4 * j + wave;
        w[j] = kk < kend ? *reinterpret_cast<const float2*>(Wg + (int64_t)(k0 + kk) * N + c)
                         : make_float2(0.f, 0.f);
      }
#pragma unroll
      for (int j = 0; j < kKChunk / 4; ++j) {
        const float* xk = lds + (4 * j + wave) * R;  // wave-uniform: broadcast reads
#pragma unroll
        for (int r = 0; r < R; r += 4) {
          const float4 xv = *reinterpret_cast<const float4*>(xk + r);
          acc[r + 0][0] += xv.x * w[j].x;
          acc[r + 0][1] += xv.x * w[j].y;
          acc[r + 1][0] += xv.y * w[j].x;
          acc[r + 1][1] += xv.y * w[j].y;
          acc[r + 2][0] += xv.z * w[j].x;
          acc[r + 2][1] += xv.z * w[j].y;
          acc[r + 3][0] += xv.w * w[j].x;
          acc[r + 3][1] += xv.w * w[j].y;
        }
      }
    }
  }
  // Reduction over the four waves, 16 rows at a time.
#pragma unroll
  for (int rr = 0; rr < R; rr += 16) {
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r)
      *reinterpret_cast<float2*>(lds + (wave * 16 + r) * kColsPerBlock + 2 * lane) =
          make_float2(acc[rr + r][0], acc[rr + r][1]);
    __syncthreads();
    for (int o = tid; o < 16 * kColsPerBlock; o += 256) {
      const int r = o / kColsPerBlock, cc = o % kColsPerBlock;
      const int col = cb + cc;
      if (rr + r < rows && col < N) {
        const float* p = lds + r * kColsPerBlock + cc;
        float y = ((p[0] + p[16 * kColsPerBlock]) + p[32 * kColsPerBlock]) +
                  p[48 * kColsPerBlock];
        y += bg[col];
        if (act_out == 1) y = silu(y);
        Yg[(int64_t)(s0 + rr + r) * ldy + col] = y;
      }
    }
  }
}

}  // namespace

hipError_t launch_sinusoid(const float* sigmas_host, int n, int freq_dim, float* e,
                           hipStream_t s) {
  for (int i0 = 0; i0 < n; i0 += kMaxSig) {
    SigmaPack p;
    int cnt = n - i0 < kMaxSig ? n - i0 : kMaxSig;
    for (int i = 0; i < cnt; ++i) p.v[i] = sigmas_host[i0 + i];
    hipLaunchKernelGGL(sinusoid_kernel, dim3(cnt), dim3(128), 0, s, p, cnt, freq_dim,
                       e + (int64_t)i0 * freq_dim);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

hipError_t launch_skinny_gemm(const float* X, int ldx, int S, int K, const float* W, int N,
                              const float* b, float* Y, int64_t ldy, int act_out, int batch,
                              int64_t w_stride, int64_t b_stride, int64_t y_stride,
                              hipStream_t s) {
  if (S == 0 || batch == 0) return hipSuccess;
  if (N % 2 != 0 || ((uintptr_t)W % 8) != 0 || (w_stride % 2) != 0)
    return hipErrorInvalidValue;  // float2 loads of W
  const unsigned cols = (unsigned)((N + kColsPerBlock - 1) / kColsPerBlock);
#define SKINNY(R)                                                                            \
  hipLaunchKernelGGL(skinny_gemm_kernel<R>, dim3(cols, (unsigned)batch, (unsigned)((S + R - 1) / R)), \
                     dim3(256), 0, s, X, ldx, S, K, W, N, b, Y, ldy, act_out, w_stride,     \
                     b_stride, y_stride)
  if (S <= 16)
    SKINNY(16);
  else if (S <= 32)
    SKINNY(32);
  else
    SKINNY(64);
#undef SKINNY
  return hipGetLastError();
}

}  // namespace acid

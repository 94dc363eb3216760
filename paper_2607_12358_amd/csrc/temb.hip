// Timestep conditioning: sinusoidal embedding of t = 1000 sigma and the small
// fp32 matrix products that turn it into the adaLN modulation table.
//
// This runs once per denoise loop for all noise levels at once, so the
// products have few rows (the step count) and are bound by reading the
// fp32 adaLN weights.  Each thread owns one output column and up to kRows
// rows of accumulators; the input rows are staged through LDS in K-chunks
// and broadcast to all threads, and W is read once per row-chunk with
// consecutive threads on consecutive columns (coalesced).
#include "common.h"

namespace acid {

namespace {

constexpr int kMaxSig = 128;
struct SigmaPack {
  float v[kMaxSig];
};

__global__ void sinusoid_kernel(SigmaPack sig, int n, int freq_dim, float* __restrict__ e) {
  const int i = blockIdx.x;
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

constexpr int kRows = 32;    // accumulator rows per thread
constexpr int kKChunk = 64;  // K staged per LDS round

__global__ __launch_bounds__(256) void skinny_gemm_kernel(
    const float* __restrict__ X, int ldx, int S, int K, const float* __restrict__ W, int N,
    const float* __restrict__ bias, float* __restrict__ Y, int64_t ldy, int act_out,
    int64_t w_stride, int64_t b_stride, int64_t y_stride) {
  __shared__ float xs[kKChunk][kRows];
  const int n = blockIdx.x * 256 + threadIdx.x;
  const int g = blockIdx.y;            // batch group
  const int s0 = blockIdx.z * kRows;   // row chunk
  const int rows = min(kRows, S - s0);
  const float* Wg = W + g * w_stride;
  const float* bg = bias + g * b_stride;
  float* Yg = Y + g * y_stride;
  float acc[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) acc[r] = 0.f;
  for (int k0 = 0; k0 < K; k0 += kKChunk) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < kKChunk * kRows; idx += 256) {
      int kk = idx / kRows, r = idx % kRows;
      xs[kk][r] = (r < rows && k0 + kk < K) ? X[(int64_t)(s0 + r) * ldx + k0 + kk] : 0.f;
    }
    __syncthreads();
    if (n < N) {
      const int kend = min(kKChunk, K - k0);
      for (int kk = 0; kk < kend; ++kk) {
        float w = Wg[(int64_t)(k0 + kk) * N + n];
#pragma unroll
        for (int r = 0; r < kRows; ++r) acc[r] += xs[kk][r] * w;
      }
    }
  }
  if (n < N) {
    float b = bg[n];
    for (int r = 0; r < rows; ++r) {
      float y = acc[r] + b;
      if (act_out == 1) y = silu(y);
      Yg[(int64_t)(s0 + r) * ldy + n] = y;
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
  dim3 grid((unsigned)((N + 255) / 256), (unsigned)batch, (unsigned)((S + kRows - 1) / kRows));
  hipLaunchKernelGGL(skinny_gemm_kernel, grid, dim3(256), 0, s, X, ldx, S, K, W, N, b, Y, ldy,
                     act_out, w_stride, b_stride, y_stride);
  return hipGetLastError();
}

}  // namespace acid

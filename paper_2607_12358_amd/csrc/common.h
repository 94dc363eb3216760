// Internal helpers of libacid (gfx950).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "acid.h"

namespace acid {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Records a message for acid_last_error() and returns the status.
acid_status set_error(acid_status st, const char* fmt, ...);
acid_status check_hip(hipError_t e, const char* what);

#define ACID_HIP(call)                                            \
  do {                                                            \
    hipError_t e_ = (call);                                       \
    if (e_ != hipSuccess) return ::acid::check_hip(e_, #call);    \
  } while (0)

#define ACID_TRY(call)                          \
  do {                                          \
    acid_status s_ = (call);                    \
    if (s_ != ACID_OK) return s_;               \
  } while (0)

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float gelu_tanh(float z) {
  // 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))
  const float k0 = 0.7978845608028654f;
  float u = k0 * (z + 0.044715f * z * z * z);
  return 0.5f * z * (1.0f + tanhf(u));
}

// Same function for bf16 outputs: 0.5 z (1 + tanh(u)) == z / (1 + e^(-2u)),
// one exp2 and one reciprocal (hardware approximations, ~1 ulp each).
__device__ __forceinline__ float gelu_tanh_fast(float z) {
  // -2 log2(e) sqrt(2/pi), and the same times 0.044715
  const float k = -2.302208198144325f, kc = -0.10294324f;
  const float t = z * __builtin_fmaf(kc * z, z, k);
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

// log2(e) / sqrt(d): the factor that turns a dot product q.k into the
// softmax's exp2 argument.  Attention with plain Q applies it per score; the
// QKV epilogue can store Q pre-multiplied by it (the same float value).
inline float attn_q_scale(int d) { return 1.4426950408889634f / sqrtf((float)d); }

// ---------------------------------------------------------------- launchers
// Each returns hipGetLastError() of its launch.

// Elementwise / row kernels (elementwise.hip)
// A kernel given a predicate `pred` (a device int32) does nothing when
// *pred == 0: the device-resident gate's skip decision.
hipError_t launch_ln_modulate(int out_dtype, const float* x, int64_t rows, int H,
                              const float* shift, const float* scale, void* out,
                              hipStream_t s, const int32_t* pred = nullptr);
// TEMNI + per-workgroup partial sums (drift_partial_count(rows) fp64 pairs);
// m_prev may be null (then no partials).
hipError_t launch_temni_drift(const float* x, int64_t rows, int H, const float* shift,
                              const float* scale, const float* m_prev, float* m_cur,
                              double* partials, hipStream_t s);
int64_t drift_partial_count(int64_t rows);
// Fixed-order reduction of the (num, den) pairs of launch_temni_drift over
// `rows` rows -> out[0]=num, out[1]=den, out[2]=s.
hipError_t launch_drift_finalize(const double* partials, int64_t rows, double* out,
                                 hipStream_t s);
// With `flag` (a device int32) the operation is STORE if *flag, else APPLY;
// without it, op, skipped when predicated off.
hipError_t launch_cache(int op, const float* x, float* h, float* r, int64_t n,
                        hipStream_t s, const int32_t* flag = nullptr,
                        const int32_t* pred = nullptr);
// dst = src (n floats, 16-byte aligned) unless predicated off.
hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t s,
                       const int32_t* pred);
// One step of Algorithm 1 on the device; see gate_step_kernel.  sig_kind is
// an acid_mode (ACID: TeaCache's drift).
hipError_t launch_gate_step(const double* res, int sig_kind, int has_signal,
                            const acid_gate_params& p, int forced, int step_index,
                            acid_gate_state* st, acid_step_trace* tr, int32_t* skip, double* ec,
                            hipStream_t s);
// EasyCache's rate update on the device; see easycache_rate_kernel.
hipError_t launch_easycache_rate(const double* res, double* ec, const int32_t* pred,
                                 hipStream_t s);
// Algorithm 1 over a signal sequence on the device.
hipError_t launch_gate_sequence(const double* sig, int n, const acid_gate_params& p,
                                acid_step_trace* tr, hipStream_t s);
// fp32 [in][out] -> [out][in] in dtype
hipError_t launch_l1_norms(const float* a, const float* b, const float* c, int64_t n,
                           double* partials, int max_groups, double* out, hipStream_t s,
                           const int32_t* pred = nullptr);
hipError_t launch_easycache_reuse(float* x, float* xp, float* v, const float* d, int64_t n,
                                  float dsig, hipStream_t s, const int32_t* pred = nullptr);
// dst row o at dst + o * ldd (ldd 0: in).
hipError_t launch_transpose_convert(const float* src, int64_t in, int64_t out, int dtype,
                                    void* dst, hipStream_t s, int64_t ldd = 0);

// Timestep embedding + modulation (temb.hip)
// e[i][:] = [cos(t f_j)]_j ++ [sin(t f_j)]_j with t = 1000 sigmas_host[i], in fp64.
hipError_t launch_sinusoid(const float* sigmas_host, int n, int freq_dim, float* e,
                           hipStream_t s);
// Y[s][n] = act_out( X[s][:] . W[:, n] + b[n] ) (act_out: 0 none, 1 SiLU), batched over `batch`
// groups with element strides for W, b and the output column offset.
hipError_t launch_skinny_gemm(const float* X, int ldx, int S, int K, const float* W,
                              int N, const float* b, float* Y, int64_t ldy, int act_out,
                              int batch, int64_t w_stride, int64_t b_stride,
                              int64_t y_stride, hipStream_t s);

// GEMMs (gemm.hip)
// split_ws: for bf16, a workspace of kGemmSplitWsBytes with which grids whose
// last round would leave most CUs idle split those tiles along K (nullptr:
// never split).
constexpr size_t kGemmSplitWsBytes = (size_t)256 * 256 * 256 * 4;
hipError_t launch_linear(int dtype, int64_t M, int N, int K, const void* a, const void* wt,
                         const acid_epilogue_args& epi, hipStream_t s,
                         const int32_t* pred = nullptr, float* split_ws = nullptr);

// Attention (attention.hip)
// o_ld: row stride of O in elements (0: n_heads * d).
hipError_t launch_attention(int dtype, int n_heads, int64_t L, int d, const void* q,
                            const void* k, const void* vt, int64_t vt_ld, void* o,
                            hipStream_t s, const int32_t* pred = nullptr, int64_t o_ld = 0,
                            bool q_prescaled = false);

}  // namespace acid

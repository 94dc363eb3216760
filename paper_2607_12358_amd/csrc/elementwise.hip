// Row-wise and elementwise kernels: LayerNorm + adaLN modulate, TEMNI +
// relative-L1 drift partial sums, the fixed-order drift reduction, the
// residual cache, and weight layout conversion.
//
// All are HBM-bound.  A row (hidden <= 4096 fp32) is owned by one 64-wide
// wavefront and kept in registers as float4 chunks, so LayerNorm statistics
// take two in-register passes (mean, then centred variance) and each row is
// read from HBM exactly once.
#include "common.h"
#include "gate_step.h"

namespace acid {

namespace {

constexpr int kRowsPerBlock = 4;  // 4 waves x 1 row

__device__ __forceinline__ void store4(float* out, int64_t idx4, float4 y) {
  reinterpret_cast<float4*>(out)[idx4] = y;
}
__device__ __forceinline__ void store4(bf16* out, int64_t idx4, float4 y) {
  bf16x4 v;
  v[0] = (bf16)y.x;
  v[1] = (bf16)y.y;
  v[2] = (bf16)y.z;
  v[3] = (bf16)y.w;
  reinterpret_cast<bf16x4*>(out)[idx4] = v;
}

// Chunk c of a row as this lane reads and writes it.  Indices past the
// row's n4 chunks are clamped to its last chunk, so every load and store is
// unconditional (a load under a branch that also uses it makes the wave
// wait for each load in turn): such a lane holds a copy of the last chunk,
// stores the same bytes as the lane that owns it, and is left out of the
// row's sums.
__device__ __forceinline__ int chunk_index(int lane, int c, int n4) {
  const int idx = lane + 64 * c;
  return idx < n4 ? idx : n4 - 1;
}

// Loads a row into registers and returns (mean, rstd) of LayerNorm
// (biased variance, eps 1e-6).  All of the row's loads are issued before
// the first is used.
template <int CPL>
__device__ __forceinline__ void load_row_stats(const float4* __restrict__ xr, int n4, int lane,
                                               float4 (&v)[CPL], float& mean, float& rstd,
                                               int H) {
#pragma unroll
  for (int c = 0; c < CPL; ++c) v[c] = xr[chunk_index(lane, c, n4)];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const float t = (v[c].x + v[c].y) + (v[c].z + v[c].w);
    s += lane + 64 * c < n4 ? t : 0.f;
  }
  s = wave_sum(s);
  mean = s / (float)H;
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    int idx = lane + 64 * c;
    if (idx < n4) {
      float a = v[c].x - mean, b = v[c].y - mean, cc = v[c].z - mean, d = v[c].w - mean;
      q += (a * a + b * b) + (cc * cc + d * d);
    }
  }
  q = wave_sum(q);
  rstd = 1.0f / sqrtf(q / (float)H + 1e-6f);
}

template <int CPL, typename OutT>
__global__ __launch_bounds__(256) void ln_modulate_kernel(const float* __restrict__ x,
                                                          int64_t rows, int H,
                                                          const float* __restrict__ shift,
                                                          const float* __restrict__ scale,
                                                          OutT* __restrict__ out,
                                                          const int32_t* __restrict__ pred) {
  if (pred && *pred == 0) return;  // predicated off by the device gate
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;  // whole wave leaves together
  const int n4 = H >> 2;
  float4 v[CPL];
  float mean, rstd;
  load_row_stats<CPL>(reinterpret_cast<const float4*>(x + row * H), n4, lane, v, mean, rstd, H);
  const float4* sh4 = reinterpret_cast<const float4*>(shift);
  const float4* sc4 = reinterpret_cast<const float4*>(scale);
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int j = chunk_index(lane, c, n4);
    const float4 sc = sc4[j], sh = sh4[j];
    float4 y;
    y.x = (v[c].x - mean) * rstd * (1.f + sc.x) + sh.x;
    y.y = (v[c].y - mean) * rstd * (1.f + sc.y) + sh.y;
    y.z = (v[c].z - mean) * rstd * (1.f + sc.z) + sh.z;
    y.w = (v[c].w - mean) * rstd * (1.f + sc.w) + sh.w;
    store4(out, row * n4 + j, y);
  }
}

// TEMNI m = LN(x) (1 + scale) + shift, stored; if m_prev is given, the
// block also writes (sum|m - m_prev|, sum|m_prev|) over its rows as doubles
// to partials[2 blockIdx.x], partials[2 blockIdx.x + 1]: each wave reduces
// its row in fp32, the block adds its waves' sums in wave order in fp64.
template <int CPL>
__global__ __launch_bounds__(256) void temni_drift_kernel(
    const float* __restrict__ x, int64_t rows, int H, const float* __restrict__ shift,
    const float* __restrict__ scale, const float* __restrict__ m_prev,
    float* __restrict__ m_cur, double* __restrict__ partials) {
  __shared__ double wsum[2 * kRowsPerBlock];
  const int wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + wave;
  const int lane = threadIdx.x & 63;
  float num = 0.f, den = 0.f;
  if (row < rows) {  // whole waves
    const int n4 = H >> 2;
    float4 v[CPL];
    float mean, rstd;
    load_row_stats<CPL>(reinterpret_cast<const float4*>(x + row * H), n4, lane, v, mean, rstd, H);
    const float4* sh4 = reinterpret_cast<const float4*>(shift);
    const float4* sc4 = reinterpret_cast<const float4*>(scale);
    const float4* mp4 = reinterpret_cast<const float4*>(m_prev + row * H);
    float4* mc4 = reinterpret_cast<float4*>(m_cur + row * H);
    // One straight-line body with the previous TEMNI, one without.  The
    // m_cur stores may alias the loads as far as the compiler can tell, so
    // each group of G chunks loads all it needs before its first store.
    auto body = [&](auto with_prev) {
      constexpr bool kPrev = decltype(with_prev)::value;
      constexpr int G = CPL < 6 ? CPL : 6;
#pragma unroll
      for (int c0 = 0; c0 < CPL; c0 += G) {
        float4 sc[G], sh[G];
        f32x4 pv[G];
#pragma unroll
        for (int i = 0; i < G && c0 + i < CPL; ++i) {
          const int j = chunk_index(lane, c0 + i, n4);
          sc[i] = sc4[j];
          sh[i] = sh4[j];
          // m_prev and m_cur are read and written once per step, and the
          // whole DiT step runs before they are touched again: both bypass
          // the caches (non-temporal)
          if constexpr (kPrev) pv[i] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(mp4) + j);
        }
        __builtin_amdgcn_sched_barrier(0);  // the group's loads stay ahead of its stores
#pragma unroll
        for (int i = 0; i < G && c0 + i < CPL; ++i) {
          const int c = c0 + i;
          const float4 v4 = v[c];
          float4 y;
          y.x = (v4.x - mean) * rstd * (1.f + sc[i].x) + sh[i].x;
          y.y = (v4.y - mean) * rstd * (1.f + sc[i].y) + sh[i].y;
          y.z = (v4.z - mean) * rstd * (1.f + sc[i].z) + sh[i].z;
          y.w = (v4.w - mean) * rstd * (1.f + sc[i].w) + sh[i].w;
          if constexpr (kPrev) {
            const float4 p = make_float4(pv[i][0], pv[i][1], pv[i][2], pv[i][3]);
            const float dn =
                (fabsf(y.x - p.x) + fabsf(y.y - p.y)) + (fabsf(y.z - p.z) + fabsf(y.w - p.w));
            const float dd = (fabsf(p.x) + fabsf(p.y)) + (fabsf(p.z) + fabsf(p.w));
            const bool in = lane + 64 * c < n4;
            num += in ? dn : 0.f;
            den += in ? dd : 0.f;
          }
          __builtin_nontemporal_store(f32x4{y.x, y.y, y.z, y.w},
                                      reinterpret_cast<f32x4*>(mc4) + chunk_index(lane, c, n4));
        }
      }
    };
    if (m_prev)
      body(std::true_type{});
    else
      body(std::false_type{});
    if (m_prev) {
      num = wave_sum(num);
      den = wave_sum(den);
    }
  }
  if (m_prev) {  // uniform over the block: every wave reaches the barrier
    if (lane == 0) {
      wsum[2 * wave] = (double)num;
      wsum[2 * wave + 1] = (double)den;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      double n = 0.0, d = 0.0;
#pragma unroll
      for (int w = 0; w < kRowsPerBlock; ++w) {
        n += wsum[2 * w];
        d += wsum[2 * w + 1];
      }
      partials[2 * blockIdx.x] = n;
      partials[2 * blockIdx.x + 1] = d;
    }
  }
}

// One block of 1024 threads over G partial pairs: thread t adds pairs t,
// t + 1024, ... in that order (eight loads in flight at a time), then a
// fixed binary tree in LDS.  Deterministic for a given G.
__global__ __launch_bounds__(1024) void drift_finalize_kernel(const double* __restrict__ part,
                                                              int64_t G,
                                                              double* __restrict__ out) {
  constexpr int kT = 1024, kU = 8;
  __shared__ double sn[kT], sd[kT];
  const int t = threadIdx.x;
  const double2* p2 = reinterpret_cast<const double2*>(part);
  double n = 0.0, d = 0.0;
  int64_t g = t;
  for (; g + (kU - 1) * kT < G; g += kU * kT) {
    double2 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = p2[g + u * kT];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      n += v[u].x;
      d += v[u].y;
    }
  }
  for (; g < G; g += kT) {
    const double2 v = p2[g];
    n += v.x;
    d += v.y;
  }
  sn[t] = n;
  sd[t] = d;
  __syncthreads();
  for (int w = kT / 2; w > 0; w >>= 1) {
    if (t < w) {
      sn[t] += sn[t + w];
      sd[t] += sd[t + w];
    }
    __syncthreads();
  }
  if (t == 0) {
    double num = sn[0], den = sd[0], s;
    if (den == 0.0)
      s = (num == 0.0) ? 0.0 : __builtin_inf();
    else
      s = num / den;
    out[0] = num;
    out[1] = den;
    out[2] = s;
  }
}

// STORE: r = h - x ; APPLY: h = x + r.  float4 body, scalar tail.
template <int OP>
__device__ __forceinline__ void cache_body(const float* __restrict__ x, float* __restrict__ h,
                                           float* __restrict__ r, int64_t n) {
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float4* x4 = reinterpret_cast<const float4*>(x);
  float4* h4 = reinterpret_cast<float4*>(h);
  float4* r4 = reinterpret_cast<float4*>(r);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 a = *(x4 + i);
    if (OP == ACID_CACHE_STORE) {
      float4 b = *(h4 + i);
      *(r4 + i) = make_float4(b.x - a.x, b.y - a.y, b.z - a.z, b.w - a.w);
    } else {
      float4 b = *(r4 + i);
      *(h4 + i) = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    int64_t i = n4 * 4 + threadIdx.x;
    if (OP == ACID_CACHE_STORE)
      r[i] = h[i] - x[i];
    else
      h[i] = x[i] + r[i];
  }
}

template <int OP>
__global__ __launch_bounds__(256) void cache_kernel(const float* __restrict__ x,
                                                    float* __restrict__ h,
                                                    float* __restrict__ r, int64_t n,
                                                    const int32_t* __restrict__ pred) {
  if (pred && *pred == 0) return;
  cache_body<OP>(x, h, r, n);
}

// The operation chosen by the device gate's decision: STORE after a computed
// step, APPLY on a skipped one.
__global__ __launch_bounds__(256) void cache_by_flag_kernel(const float* __restrict__ x,
                                                            float* __restrict__ h,
                                                            float* __restrict__ r, int64_t n,
                                                            const int32_t* __restrict__ flag) {
  if (*flag)
    cache_body<ACID_CACHE_STORE>(x, h, r, n);
  else
    cache_body<ACID_CACHE_APPLY>(x, h, r, n);
}

// dst = src over n floats (16-byte aligned), unless the device gate's flag
// says skip.
__global__ __launch_bounds__(256) void copy_pred_kernel(const float* __restrict__ src,
                                                        float* __restrict__ dst, int64_t n,
                                                        const int32_t* __restrict__ pred) {
  if (pred && *pred == 0) return;
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float4* s4 = reinterpret_cast<const float4*>(src);
  float4* d4 = reinterpret_cast<float4*>(dst);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
    d4[i] = s4[i];
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) dst[n4 * 4 + threadIdx.x] = src[n4 * 4 + threadIdx.x];
}

// num / den with 0 / 0 = 0 and num / 0 = +inf (the host loops' rule).
__device__ __forceinline__ double ratio_or_inf_dev(double num, double den) {
  if (den == 0.0) return num == 0.0 ? 0.0 : __builtin_inf();
  return num / den;
}

// Device-resident gate, one step of Algorithm 1 per launch (one thread).
// The signal, when has_signal (else NaN), by kind: TeaCache res[2] (the
// drift reduction's output); DiCache res[0] / res[1] (the probe's relative
// L1 change); EasyCache k res[0] / res[1] once a rate k exists (ec[0], with
// ec[1] != 0), and res[0] = |x_i - x_{i-1}| is kept in ec[2] for the rate
// update.  step_index 0 starts from the initial state.  The decision goes to
// tr->compute (the predicate of the step's model kernels): the gate's own,
// or forced (0/1) when forced >= 0; *skip receives its negation.
__global__ void gate_step_kernel(const double* __restrict__ res, int sig_kind, int has_signal,
                                 acid_gate_params p, int forced, int step_index,
                                 acid_gate_state* __restrict__ st,
                                 acid_step_trace* __restrict__ tr, int32_t* __restrict__ skip,
                                 double* __restrict__ ec) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  acid_gate_state g;
  if (step_index == 0) {
    g.sigma_sum = 0.0;
    g.s_prev = 0.0;
    g.has_prev = 0;
    g.step = 0;
    if (ec) {
      ec[0] = __builtin_nan("");
      ec[1] = 0.0;
      ec[2] = __builtin_nan("");
    }
  } else {
    g = *st;
  }
  double s = __builtin_nan("");
  if (has_signal) {
    if (sig_kind == ACID_MODE_DICACHE) {
      s = ratio_or_inf_dev(res[0], res[1]);
    } else if (sig_kind == ACID_MODE_EASYCACHE) {
      if (ec[1] != 0.0) s = ec[0] * ratio_or_inf_dev(res[0], res[1]);
      ec[2] = res[0];
    } else {
      s = res[2];
    }
  }
  double tau;
  const int32_t c = gate_step(&g, &p, s, &tau);
  *st = g;
  acid_step_trace t;
  t.compute = forced >= 0 ? forced : c;
  *skip = !t.compute;
  t.gate_compute = c;
  t.s = s;
  t.sigma_sum_after = g.sigma_sum;
  t.tau_used = tau;
  *tr = t;
}

// Algorithm 1 over a whole signal sequence s[0..n) on the device (one thread),
// for checking the device gate against the host gate and the worked example.
__global__ void gate_sequence_kernel(const double* __restrict__ s, int n, acid_gate_params p,
                                     acid_step_trace* __restrict__ tr) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  acid_gate_state g;
  g.sigma_sum = 0.0;
  g.s_prev = 0.0;
  g.has_prev = 0;
  g.step = 0;
  for (int i = 0; i < n; ++i) {
    double tau;
    const int32_t c = gate_step(&g, &p, s[i], &tau);
    acid_step_trace t;
    t.compute = c;
    t.gate_compute = c;
    t.s = s[i];
    t.sigma_sum_after = g.sigma_sum;
    t.tau_used = tau;
    tr[i] = t;
  }
}

// L1 partial sums in fp64 for EasyCache's signal: block g accumulates
// sum |a - b| (sum |a| without b) and sum |c| over its grid-stride share;
// part[2g], part[2g+1].  The grid depends on n only, and every sum has a
// fixed order, so the result is deterministic.
__device__ __forceinline__ double block_sum_f64(double v, double* lds) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) lds[w] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0)
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += lds[i];
  return t;
}

template <bool HAS_B, bool HAS_C>
__global__ __launch_bounds__(256) void l1_partials_kernel(const float* __restrict__ a,
                                                          const float* __restrict__ b,
                                                          const float* __restrict__ c,
                                                          int64_t n, double* __restrict__ part,
                                                          const int32_t* __restrict__ pred) {
  if (pred && *pred == 0) return;  // whole block: pred is uniform
  __shared__ double lds[4];
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float4* a4 = reinterpret_cast<const float4*>(a);
  const float4* b4 = reinterpret_cast<const float4*>(b);
  const float4* c4 = reinterpret_cast<const float4*>(c);
  double s0 = 0.0, s1 = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 av = a4[i];
    if (HAS_B) {
      const float4 bv = b4[i];
      av = make_float4(av.x - bv.x, av.y - bv.y, av.z - bv.z, av.w - bv.w);
    }
    s0 += ((double)fabsf(av.x) + (double)fabsf(av.y)) + ((double)fabsf(av.z) + (double)fabsf(av.w));
    if (HAS_C) {
      const float4 cv = c4[i];
      s1 += ((double)fabsf(cv.x) + (double)fabsf(cv.y)) + ((double)fabsf(cv.z) + (double)fabsf(cv.w));
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const int64_t i = n4 * 4 + threadIdx.x;
    s0 += (double)fabsf(HAS_B ? a[i] - b[i] : a[i]);
    if (HAS_C) s1 += (double)fabsf(c[i]);
  }
  s0 = block_sum_f64(s0, lds);
  s1 = block_sum_f64(s1, lds);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = s0;
    part[2 * blockIdx.x + 1] = s1;
  }
}

// Fixed-order sum of G partial pairs: out[0], out[1].
__global__ __launch_bounds__(1024) void l1_finalize_kernel(const double* __restrict__ part, int G,
                                                           double* __restrict__ out,
                                                           const int32_t* __restrict__ pred) {
  if (pred && *pred == 0) return;
  __shared__ double s0[1024], s1[1024];
  const int t = threadIdx.x;
  double u = 0.0, w = 0.0;
  for (int g = t; g < G; g += 1024) {
    u += part[2 * g];
    w += part[2 * g + 1];
  }
  s0[t] = u;
  s1[t] = w;
  __syncthreads();
  for (int k = 512; k > 0; k >>= 1) {
    if (t < k) {
      s0[t] += s0[t + k];
      s1[t] += s1[t + k];
    }
    __syncthreads();
  }
  if (t == 0) {
    out[0] = s0[0];
    out[1] = s1[0];
  }
}

// EasyCache's skipped step: v = x + D; x_prev = x; x = x + dsigma v.
__global__ __launch_bounds__(256) void easycache_reuse_kernel(float* __restrict__ x,
                                                              float* __restrict__ xp,
                                                              float* __restrict__ v,
                                                              const float* __restrict__ d,
                                                              int64_t n, float dsig,
                                                              const int32_t* __restrict__ pred) {
  if (pred && *pred == 0) return;
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  float4* x4 = reinterpret_cast<float4*>(x);
  float4* p4 = reinterpret_cast<float4*>(xp);
  float4* v4 = reinterpret_cast<float4*>(v);
  const float4* d4 = reinterpret_cast<const float4*>(d);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const float4 a = x4[i], o = d4[i];
    const float4 w = make_float4(a.x + o.x, a.y + o.y, a.z + o.z, a.w + o.w);
    p4[i] = a;
    v4[i] = w;
    x4[i] = make_float4(fmaf(dsig, w.x, a.x), fmaf(dsig, w.y, a.y), fmaf(dsig, w.z, a.z),
                        fmaf(dsig, w.w, a.w));
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const int64_t i = n4 * 4 + threadIdx.x;
    const float a = x[i], w = a + d[i];
    xp[i] = a;
    v[i] = w;
    x[i] = fmaf(dsig, w, a);
  }
}

// fp32 [in][out] -> [out][in] (dtype), 32x32 tiles through LDS.
template <typename T>
__global__ __launch_bounds__(256) void transpose_convert_kernel(const float* __restrict__ src,
                                                                int64_t nin, int64_t nout,
                                                                T* __restrict__ dst, int64_t ldd) {
  __shared__ float tile[32][33];
  const int64_t o0 = (int64_t)blockIdx.x * 32, i0 = (int64_t)blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int k = ty; k < 32; k += 8) {
    int64_t i = i0 + k, o = o0 + tx;
    tile[k][tx] = (i < nin && o < nout) ? src[i * nout + o] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    int64_t o = o0 + k, i = i0 + tx;
    if (o < nout && i < nin) dst[o * ldd + i] = (T)tile[tx][k];
  }
}

}  // namespace

#define ACID_ROW_DISPATCH(CPL_VAR, MACRO) \
  switch (CPL_VAR) {                      \
    case 1: MACRO(1); break;              \
    case 2: MACRO(2); break;              \
    case 3: MACRO(3); break;              \
    case 4: MACRO(4); break;              \
    case 5: MACRO(5); break;              \
    case 6: MACRO(6); break;              \
    case 8: MACRO(8); break;              \
    case 12: MACRO(12); break;            \
    case 16: MACRO(16); break;            \
    default: return hipErrorInvalidValue; \
  }

static int row_chunks(int H) {
  // float4 chunks per lane, rounded to a compiled instantiation
  int c = (H / 4 + 63) / 64;
  if (c <= 6) return c;
  if (c <= 8) return 8;
  if (c <= 12) return 12;
  if (c <= 16) return 16;
  return -1;
}

hipError_t launch_ln_modulate(int out_dtype, const float* x, int64_t rows, int H,
                              const float* shift, const float* scale, void* out,
                              hipStream_t s, const int32_t* pred) {
  if (rows == 0) return hipSuccess;
  const int cpl = row_chunks(H);
  dim3 grid((unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock));
#define LN_BF(C) hipLaunchKernelGGL((ln_modulate_kernel<C, bf16>), grid, dim3(256), 0, s, x, rows, H, shift, scale, (bf16*)out, pred)
#define LN_F(C) hipLaunchKernelGGL((ln_modulate_kernel<C, float>), grid, dim3(256), 0, s, x, rows, H, shift, scale, (float*)out, pred)
  if (out_dtype == ACID_BF16) {
    ACID_ROW_DISPATCH(cpl, LN_BF)
  } else {
    ACID_ROW_DISPATCH(cpl, LN_F)
  }
#undef LN_BF
#undef LN_F
  return hipGetLastError();
}

hipError_t launch_temni_drift(const float* x, int64_t rows, int H, const float* shift,
                              const float* scale, const float* m_prev, float* m_cur,
                              double* partials, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int cpl = row_chunks(H);
  dim3 grid((unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock));
#define TD(C) hipLaunchKernelGGL((temni_drift_kernel<C>), grid, dim3(256), 0, s, x, rows, H, shift, scale, m_prev, m_cur, partials)
  ACID_ROW_DISPATCH(cpl, TD)
#undef TD
  return hipGetLastError();
}

int64_t drift_partial_count(int64_t rows) { return (rows + kRowsPerBlock - 1) / kRowsPerBlock; }

hipError_t launch_drift_finalize(const double* partials, int64_t rows, double* out,
                                 hipStream_t s) {
  hipLaunchKernelGGL(drift_finalize_kernel, dim3(1), dim3(1024), 0, s, partials,
                     drift_partial_count(rows), out);
  return hipGetLastError();
}

// Streaming kernels take one float4 per thread (no loop trip on the common
// sizes): measured 5.85 TB/s for two streams in and one out at 201 MB each,
// against 5.0 TB/s for a grid of 4096 workgroups looping over the data.  The
// grid-stride loop only serves sizes beyond 2^22 workgroups.
static unsigned stream_grid(int64_t n) {
  int64_t blocks = ((n + 3) / 4 + 255) / 256;
  if (blocks > ((int64_t)1 << 22)) blocks = (int64_t)1 << 22;
  return (unsigned)blocks;
}

hipError_t launch_cache(int op, const float* x, float* h, float* r, int64_t n, hipStream_t s,
                        const int32_t* flag, const int32_t* pred) {
  if (n == 0) return hipSuccess;
  const unsigned blocks = stream_grid(n);
  if (flag)
    hipLaunchKernelGGL(cache_by_flag_kernel, dim3(blocks), dim3(256), 0, s, x, h, r, n, flag);
  else if (op == ACID_CACHE_STORE)
    hipLaunchKernelGGL(cache_kernel<ACID_CACHE_STORE>, dim3((unsigned)blocks), dim3(256), 0, s, x, h, r, n, pred);
  else
    hipLaunchKernelGGL(cache_kernel<ACID_CACHE_APPLY>, dim3((unsigned)blocks), dim3(256), 0, s, x, h, r, n, pred);
  return hipGetLastError();
}

static int l1_grid(int64_t n, int max_groups) {
  int64_t g = ((n >> 2) + 255) / 256;
  if (g < 1) g = 1;
  if (g > 1024) g = 1024;
  if (g > max_groups) g = max_groups;
  return (int)g;
}

hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t s,
                       const int32_t* pred) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(copy_pred_kernel, dim3(stream_grid(n)), dim3(256), 0, s, src, dst, n, pred);
  return hipGetLastError();
}

hipError_t launch_gate_step(const double* res, int sig_kind, int has_signal,
                            const acid_gate_params& p, int forced, int step_index,
                            acid_gate_state* st, acid_step_trace* tr, int32_t* skip, double* ec,
                            hipStream_t s) {
  hipLaunchKernelGGL(gate_step_kernel, dim3(1), dim3(64), 0, s, res, sig_kind, has_signal, p,
                     forced, step_index, st, tr, skip, ec);
  return hipGetLastError();
}

// EasyCache's rate after a computed step: k = |v_i - v_{i-1}| / |x_i - x_{i-1}|
// (res[0] over the kept ec[2]), one thread, unless predicated off.
__global__ void easycache_rate_kernel(const double* __restrict__ res, double* __restrict__ ec,
                                      const int32_t* __restrict__ pred) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  if (pred && *pred == 0) return;
  ec[0] = ratio_or_inf_dev(res[0], ec[2]);
  ec[1] = 1.0;
}

hipError_t launch_easycache_rate(const double* res, double* ec, const int32_t* pred,
                                 hipStream_t s) {
  hipLaunchKernelGGL(easycache_rate_kernel, dim3(1), dim3(64), 0, s, res, ec, pred);
  return hipGetLastError();
}

hipError_t launch_gate_sequence(const double* sig, int n, const acid_gate_params& p,
                                acid_step_trace* tr, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gate_sequence_kernel, dim3(1), dim3(64), 0, s, sig, n, p, tr);
  return hipGetLastError();
}

hipError_t launch_l1_norms(const float* a, const float* b, const float* c, int64_t n,
                           double* partials, int max_groups, double* out, hipStream_t s,
                           const int32_t* pred) {
  const int G = l1_grid(n, max_groups);
#define L1K(HB, HC) \
  hipLaunchKernelGGL((l1_partials_kernel<HB, HC>), dim3(G), dim3(256), 0, s, a, b, c, n, partials, pred)
  if (b && c) L1K(true, true);
  else if (b) L1K(true, false);
  else if (c) L1K(false, true);
  else L1K(false, false);
#undef L1K
  hipLaunchKernelGGL(l1_finalize_kernel, dim3(1), dim3(1024), 0, s, partials, G, out, pred);
  return hipGetLastError();
}

hipError_t launch_easycache_reuse(float* x, float* xp, float* v, const float* d, int64_t n,
                                  float dsig, hipStream_t s, const int32_t* pred) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(easycache_reuse_kernel, dim3(stream_grid(n)), dim3(256), 0, s, x, xp, v, d,
                     n, dsig, pred);
  return hipGetLastError();
}

hipError_t launch_transpose_convert(const float* src, int64_t nin, int64_t nout, int dtype,
                                    void* dst, hipStream_t s, int64_t ldd) {
  if (ldd == 0) ldd = nin;
  dim3 grid((unsigned)((nout + 31) / 32), (unsigned)((nin + 31) / 32));
  if (dtype == ACID_BF16)
    hipLaunchKernelGGL(transpose_convert_kernel<bf16>, grid, dim3(256), 0, s, src, nin, nout, (bf16*)dst, ldd);
  else
    hipLaunchKernelGGL(transpose_convert_kernel<float>, grid, dim3(256), 0, s, src, nin, nout, (float*)dst, ldd);
  return hipGetLastError();
}

}  // namespace acid

// Host runtime of libacid: configuration checks, the weight-arena and
// workspace layouts, the DiT step, the drift signal, the residual cache and
// the ACID-gated denoise loop.  All device memory is the caller's; this file
// only carves it up and launches kernels on the caller's stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "common.h"

#define ACID_VERSION "0.1.0"

namespace acid {

static thread_local char g_err[512] = "";

acid_status set_error(acid_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

acid_status check_hip(hipError_t e, const char* what) {
  return set_error(ACID_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t a) { return (a + kAlign - 1) / kAlign * kAlign; }

int esize(int dtype) { return dtype == ACID_BF16 ? 2 : 4; }

// Size limits of the kernels' index arithmetic: the bf16 attention kernel
// addresses a head's K and V^T with 32-bit offsets, the bf16 GEMM a tile's
// operand rows with 32-bit offsets (256 rows of K elements), and a launch
// holds fewer than 2^32 work-items per grid dimension.
acid_status check_attention_size(int dtype, int n_heads, int64_t L, int d, int64_t vt_ld) {
  const int64_t lim = 0x7fffffff;
  if (dtype == ACID_BF16 && vt_ld > lim / (2 * d))
    return set_error(ACID_ERR_SHAPE, "bf16 attention: head_dim * vt_ld * 2 bytes must be < 2^31");
  if (L > lim / 32 || L * n_heads > lim / 32)  // the fp32 kernel: 64 work-items per query
    return set_error(ACID_ERR_SHAPE, "attention: seq_len %lld x n_heads %d exceeds the grid limit",
                     (long long)L, n_heads);
  return ACID_OK;
}
acid_status check_linear_size(int64_t M, int N, int K) {
  if (K > (1 << 22) || N > (1 << 22))
    return set_error(ACID_ERR_SHAPE, "linear: N %d and K %d must be <= 2^22", N, K);
  if (M > (int64_t)1 << 30 || (M + 255) / 256 * ((N + 255) / 256) >= (1 << 23))
    return set_error(ACID_ERR_SHAPE, "linear: M %lld x N %d exceeds the grid limit", (long long)M,
                     N);
  return ACID_OK;
}

acid_status check_config(const acid_dit_config* c) {
  if (!c) return set_error(ACID_ERR_INVALID_ARG, "config is NULL");
  if (c->dtype != ACID_F32 && c->dtype != ACID_BF16)
    return set_error(ACID_ERR_INVALID_ARG, "dtype %d is not ACID_F32 or ACID_BF16", c->dtype);
  if (c->n_blocks < 1 || c->n_video < 1 || c->n_text < 0 || c->n_heads < 1)
    return set_error(ACID_ERR_INVALID_ARG, "n_blocks, n_video, n_heads must be >= 1 and n_text >= 0");
  if (c->head_dim != 64 && c->head_dim != 128)
    return set_error(ACID_ERR_SHAPE, "head_dim %d: supported 64 or 128", c->head_dim);
  if ((int64_t)c->n_heads * c->head_dim != c->hidden)
    return set_error(ACID_ERR_SHAPE, "hidden %d != n_heads %d * head_dim %d", c->hidden, c->n_heads,
                     c->head_dim);
  if (c->hidden % 128 || c->hidden > 4096)
    return set_error(ACID_ERR_SHAPE, "hidden %d: must be a multiple of 128 and <= 4096", c->hidden);
  if (c->ffn < 128 || c->ffn % 128)
    return set_error(ACID_ERR_SHAPE, "ffn %d: must be a positive multiple of 128", c->ffn);
  if (c->freq_dim < 2 || c->freq_dim % 2 || c->freq_dim > 1024)
    return set_error(ACID_ERR_SHAPE, "freq_dim %d: must be even and <= 1024", c->freq_dim);
  if (c->block_kind != ACID_BLOCK_SEQUENTIAL && c->block_kind != ACID_BLOCK_PARALLEL)
    return set_error(ACID_ERR_INVALID_ARG, "block_kind %d is not SEQUENTIAL or PARALLEL",
                     c->block_kind);
  // Every attention and GEMM of the step within the kernels' size limits:
  // L tokens, N up to 3H + F (the parallel block's fused projection), K up
  // to H + F.
  const int64_t L = (int64_t)c->n_video + c->n_text;
  ACID_TRY(check_attention_size(c->dtype, c->n_heads, L, c->head_dim, round_up(L, 8)));
  if ((int64_t)3 * c->hidden + c->ffn > (1 << 22))
    return set_error(ACID_ERR_SHAPE, "3 * hidden + ffn must be <= 2^22");
  return check_linear_size(L, 3 * c->hidden + c->ffn, c->hidden + c->ffn);
}

// ------------------------------------------------------------ arena layout
struct WeightLayout {
  size_t temb_w1, temb_b1, temb_w2, temb_b2;
  size_t blk0;        // offset of block 0
  size_t blk_stride;  // bytes between consecutive blocks
  // offsets within a block
  size_t ada_w, ada_b, qkv_w, qkv_b, o_w, o_b, f1_w, f1_b, f2_w, f2_b;
  size_t head_ada_w, head_ada_b, head_w, head_b;
  size_t total;
};

WeightLayout weight_layout(const acid_dit_config& c) {
  WeightLayout L;
  const size_t H = c.hidden, F = c.ffn, Ft = c.freq_dim, es = esize(c.dtype);
  size_t off = 0;
  auto put = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.temb_w1 = put(Ft * H * 4);
  L.temb_b1 = put(H * 4);
  L.temb_w2 = put(H * H * 4);
  L.temb_b2 = put(H * 4);
  L.blk0 = off;
  size_t b = 0;
  auto putb = [&](size_t bytes) {
    size_t o = b;
    b = align_up(b + bytes);
    return o;
  };
  // With H and F multiples of 128 every size below is a multiple of the
  // 256-byte alignment, so neighbours are contiguous: [W_qkv^T ; W_1^T] is one
  // [3H + F][H] operand, [b_qkv | b_1] one bias, and the o_w + f2_w region
  // holds the parallel block's [W_o ; W_2]^T as one [H][H + F] operand.
  L.ada_w = putb(H * 6 * H * 4);
  L.ada_b = putb(6 * H * 4);
  L.qkv_w = putb(3 * H * H * es);
  L.f1_w = putb(F * H * es);
  L.qkv_b = putb(3 * H * 4);
  L.f1_b = putb(F * 4);
  L.o_w = putb(H * H * es);
  L.f2_w = putb(H * F * es);
  L.o_b = putb(H * 4);
  L.f2_b = putb(H * 4);
  L.blk_stride = b;
  off += b * c.n_blocks;
  L.head_ada_w = put(H * 2 * H * 4);
  L.head_ada_b = put(2 * H * 4);
  L.head_w = put(H * H * es);
  L.head_b = put(H * 4);
  L.total = off;
  return L;
}

struct WorkLayout {
  size_t h, act, q, k, vt, o, g, modtab, temb_e, temb_hid, temb_u, partials, dres, m0, m1, r, v;
  size_t dtrace, gstate;  // device-resident gate: per-step trace, state
  size_t dskip, ecst;     // per-step skip words; EasyCache (k, have k, |dx|)
  size_t splitk;          // bf16: the GEMMs' K-split partial tiles
  size_t total;
  int64_t vt_ld;
};

WorkLayout work_layout(const acid_dit_config& c, int max_steps) {
  WorkLayout W;
  const size_t H = c.hidden, F = c.ffn, Ft = c.freq_dim, es = esize(c.dtype);
  const size_t Lv = c.n_video, L = (size_t)c.n_text + c.n_video;
  const size_t S = max_steps < 1 ? 1 : max_steps;
  W.vt_ld = round_up((int64_t)L, 8);
  size_t off = 0;
  auto put = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  W.h = put(L * H * 4);
  W.act = put(L * H * es);
  W.q = put(L * H * es);
  W.k = put(L * H * es);
  W.vt = put((size_t)c.n_heads * c.head_dim * W.vt_ld * es);
  W.o = put(L * H * es);
  // parallel block: [attention output | GELU(mlp)] rows of H + F
  W.g = put(L * (F + (c.block_kind == ACID_BLOCK_PARALLEL ? H : 0)) * es);
  W.modtab = put(S * (6 * (size_t)c.n_blocks + 2) * H * 4);
  W.temb_e = put(S * Ft * 4);
  W.temb_hid = put(S * H * 4);
  W.temb_u = put(S * H * 4);
  W.partials = put(Lv * 2 * sizeof(double));
  W.dres = put(4 * sizeof(double));
  W.m0 = put(Lv * H * 4);
  W.m1 = put(Lv * H * 4);
  W.r = put(Lv * H * 4);
  W.v = put(Lv * H * 4);
  W.dtrace = put(S * sizeof(acid_step_trace));
  W.gstate = put(sizeof(acid_gate_state));
  W.dskip = put(S * sizeof(int32_t));
  W.ecst = put(4 * sizeof(double));
  W.splitk = put(c.dtype == ACID_BF16 ? kGemmSplitWsBytes : 0);
  W.total = off;
  return W;
}

}  // namespace
}  // namespace acid

using namespace acid;

struct acid_model {
  acid_dit_config cfg;
  int max_steps;
  int probe_blocks = 1;  // DiCache probe depth
  char* wb;  // weight arena
  char* ws;  // workspace
  WeightLayout wl;
  WorkLayout kl;
  // timing
  bool timing = false;
  struct Pending {
    int cls;
    hipEvent_t e0, e1;
  };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> pool;
  double total_ms[ACID_K_COUNT] = {};
  int64_t launches[ACID_K_COUNT] = {};
  // captured loop (device-resident gate): the executable graph, the stream
  // it was captured on, and what it was captured for
  bool capturing = false;
  hipStream_t cap = nullptr;
  hipGraphExec_t gexec = nullptr;
  struct GraphKey {
    float* x = nullptr;
    const float* text = nullptr;
    int n = 0, mode = -1, probe = 0;
    acid_gate_params gate = {};
    std::vector<float> sigmas;
    std::vector<uint8_t> forced;
    bool operator==(const GraphKey& o) const {
      return x == o.x && text == o.text && n == o.n && mode == o.mode && probe == o.probe &&
             gate.tau_low == o.gate.tau_low && gate.tau_high == o.gate.tau_high &&
             gate.delta == o.gate.delta && gate.n_warmup == o.gate.n_warmup &&
             sigmas == o.sigmas && forced == o.forced;
    }
  } gkey;

  int H() const { return cfg.hidden; }
  int64_t Lv() const { return cfg.n_video; }
  int64_t Lt() const { return cfg.n_text; }
  int64_t L() const { return (int64_t)cfg.n_text + cfg.n_video; }
  int64_t rowsz() const { return (6 * (int64_t)cfg.n_blocks + 2) * cfg.hidden; }
  template <class T = float>
  T* wp(size_t off) const { return reinterpret_cast<T*>(wb + off); }
  template <class T = float>
  T* bp(int b, size_t off) const { return reinterpret_cast<T*>(wb + wl.blk0 + (size_t)b * wl.blk_stride + off); }
  template <class T = float>
  T* kp(size_t off) const { return reinterpret_cast<T*>(ws + off); }
  // The GEMMs' K-split workspace (bf16 models; fp32 GEMMs never split).
  float* split_ws() const { return cfg.dtype == ACID_BF16 ? kp<float>(kl.splitk) : nullptr; }
};

namespace {

acid_status harvest(acid_model* m) {
  for (auto& p : m->pending) {
    ACID_HIP(hipEventSynchronize(p.e1));
    float ms = 0.f;
    ACID_HIP(hipEventElapsedTime(&ms, p.e0, p.e1));
    m->total_ms[p.cls] += ms;
    m->launches[p.cls] += 1;
    m->pool.push_back(p.e0);
    m->pool.push_back(p.e1);
  }
  m->pending.clear();
  return ACID_OK;
}

acid_status get_event(acid_model* m, hipEvent_t* e) {
  if (m->pool.empty()) {
    // Timing only: no system-scope release (cache write-back and invalidate)
    // at each record, which would also slow the kernel that follows.
    ACID_HIP(hipEventCreateWithFlags(e, hipEventDisableSystemFence));
  } else {
    *e = m->pool.back();
    m->pool.pop_back();
  }
  return ACID_OK;
}

// Launches f() on stream s, bracketed by timing events when enabled.
template <class F>
acid_status run(acid_model* m, int cls, hipStream_t s, const char* what, F&& f) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  const bool timed = m->timing && !m->capturing;  // no timer inside a captured graph
  if (timed) {
    if (m->pending.size() > 4096) ACID_TRY(harvest(m));
    ACID_TRY(get_event(m, &e0));
    ACID_TRY(get_event(m, &e1));
    ACID_HIP(hipEventRecord(e0, s));
  }
  hipError_t err = f();
  if (err != hipSuccess) return check_hip(err, what);
  if (timed) {
    ACID_HIP(hipEventRecord(e1, s));
    m->pending.push_back({cls, e0, e1});
  }
  return ACID_OK;
}

// ------------------------------------------------------------ model pieces

acid_status modulation_table(acid_model* m, const float* sigmas, int n, float* table,
                             hipStream_t s) {
  const acid_dit_config& c = m->cfg;
  const int H = c.hidden, Ft = c.freq_dim;
  float* e = m->kp(m->kl.temb_e);
  float* hid = m->kp(m->kl.temb_hid);
  float* u = m->kp(m->kl.temb_u);
  const int64_t bstride = (int64_t)(m->wl.blk_stride / 4);
  return run(m, ACID_K_TEMB, s, "timestep modulation", [&]() {
    hipError_t err = launch_sinusoid(sigmas, n, Ft, e, s);
    if (err == hipSuccess)
      err = launch_skinny_gemm(e, Ft, n, Ft, m->wp(m->wl.temb_w1), H, m->wp(m->wl.temb_b1), hid,
                               H, 1, 1, 0, 0, 0, s);
    if (err == hipSuccess)
      err = launch_skinny_gemm(hid, H, n, H, m->wp(m->wl.temb_w2), H, m->wp(m->wl.temb_b2), u, H,
                               1, 1, 0, 0, 0, s);
    if (err == hipSuccess)
      err = launch_skinny_gemm(u, H, n, H, m->bp(0, m->wl.ada_w), 6 * H, m->bp(0, m->wl.ada_b),
                               table, m->rowsz(), 0, c.n_blocks, bstride, bstride,
                               6 * (int64_t)H, s);
    if (err == hipSuccess)
      err = launch_skinny_gemm(u, H, n, H, m->wp(m->wl.head_ada_w), 2 * H,
                               m->wp(m->wl.head_ada_b), table + 6 * (int64_t)c.n_blocks * H,
                               m->rowsz(), 0, 1, 0, 0, 0, s);
    return err;
  });
}

acid_status ln_mod(acid_model* m, const float* x, int64_t rows, const float* shift,
                   const float* scale, void* out, hipStream_t s, const int32_t* pred = nullptr) {
  return run(m, ACID_K_LN_MOD, s, "ln_modulate", [&]() {
    return launch_ln_modulate(m->cfg.dtype, x, rows, m->H(), shift, scale, out, s, pred);
  });
}

// pred: the device gate's decision word (null: unconditional).
acid_status block_forward_parallel(acid_model* m, int b, const float* mod6, float* h,
                                   hipStream_t s, const int32_t* pred);

acid_status block_forward(acid_model* m, int b, const float* mod6, float* h, hipStream_t s,
                          const int32_t* pred = nullptr) {
  if (m->cfg.block_kind == ACID_BLOCK_PARALLEL) return block_forward_parallel(m, b, mod6, h, s, pred);
  const acid_dit_config& c = m->cfg;
  const int H = c.hidden, F = c.ffn;
  const int64_t L = m->L();
  void* act = m->kp<void>(m->kl.act);
  void* o = m->kp<void>(m->kl.o);
  void* g = m->kp<void>(m->kl.g);
  const int dt = c.dtype;

  ACID_TRY(ln_mod(m, h, L, mod6, mod6 + H, act, s, pred));

  acid_epilogue_args e = {};
  e.kind = ACID_EPI_QKV;
  e.bias = m->bp(b, m->wl.qkv_b);
  e.q = m->kp<void>(m->kl.q);
  e.k = m->kp<void>(m->kl.k);
  e.vt = m->kp<void>(m->kl.vt);
  e.vt_ld = m->kl.vt_ld;
  e.n_heads = c.n_heads;
  e.head_dim = c.head_dim;
  e.q_prescale = 1;  // Q leaves the GEMM in the softmax's exp2 units
  ACID_TRY(run(m, ACID_K_GEMM_QKV, s, "qkv gemm", [&]() {
    return launch_linear(dt, L, 3 * H, H, act, m->bp<void>(b, m->wl.qkv_w), e, s, pred, m->split_ws());
  }));
  ACID_TRY(run(m, ACID_K_ATTENTION, s, "attention", [&]() {
    return launch_attention(dt, c.n_heads, L, c.head_dim, e.q, e.k, e.vt, e.vt_ld, o, s, pred, 0,
                            true);
  }));
  acid_epilogue_args p = {};
  p.kind = ACID_EPI_GATE_RESIDUAL;
  p.bias = m->bp(b, m->wl.o_b);
  p.gate = mod6 + 2 * H;
  p.out = h;
  ACID_TRY(run(m, ACID_K_GEMM_PROJ, s, "proj gemm", [&]() {
    return launch_linear(dt, L, H, H, o, m->bp<void>(b, m->wl.o_w), p, s, pred, m->split_ws());
  }));
  ACID_TRY(ln_mod(m, h, L, mod6 + 3 * H, mod6 + 4 * H, act, s, pred));
  acid_epilogue_args f1 = {};
  f1.kind = ACID_EPI_BIAS_GELU;
  f1.bias = m->bp(b, m->wl.f1_b);
  f1.out = g;
  ACID_TRY(run(m, ACID_K_GEMM_FFN1, s, "ffn1 gemm", [&]() {
    return launch_linear(dt, L, F, H, act, m->bp<void>(b, m->wl.f1_w), f1, s, pred, m->split_ws());
  }));
  acid_epilogue_args f2 = {};
  f2.kind = ACID_EPI_GATE_RESIDUAL;
  f2.bias = m->bp(b, m->wl.f2_b);
  f2.gate = mod6 + 5 * H;
  f2.out = h;
  ACID_TRY(run(m, ACID_K_GEMM_FFN2, s, "ffn2 gemm", [&]() {
    return launch_linear(dt, L, H, F, g, m->bp<void>(b, m->wl.f2_w), f2, s, pred, m->split_ws());
  }));
  return ACID_OK;
}

// HunyuanVideo's single-stream block: one LN-modulate, one GEMM into
// Q | K | V and GELU(mlp) (the latter next to the attention output in the
// [L][H + F] buffer g), attention into g's first H columns, one GEMM over
// K = H + F with the gated residual (biases b_o + b_2).
acid_status block_forward_parallel(acid_model* m, int b, const float* mod6, float* h,
                                   hipStream_t s, const int32_t* pred) {
  const acid_dit_config& c = m->cfg;
  const int H = c.hidden, F = c.ffn;
  const int64_t L = m->L();
  const int dt = c.dtype;
  void* act = m->kp<void>(m->kl.act);
  char* g = m->kp<char>(m->kl.g);
  ACID_TRY(ln_mod(m, h, L, mod6, mod6 + H, act, s, pred));
  acid_epilogue_args e = {};
  e.kind = ACID_EPI_QKV_GELU;
  e.bias = m->bp(b, m->wl.qkv_b);  // [b_qkv | b_1]
  e.q = m->kp<void>(m->kl.q);
  e.k = m->kp<void>(m->kl.k);
  e.vt = m->kp<void>(m->kl.vt);
  e.vt_ld = m->kl.vt_ld;
  e.n_heads = c.n_heads;
  e.head_dim = c.head_dim;
  e.out = g + (size_t)H * esize(dt);
  e.out_ld = H + F;
  e.q_prescale = 1;
  ACID_TRY(run(m, ACID_K_GEMM_QKV, s, "qkv+mlp gemm", [&]() {
    return launch_linear(dt, L, 3 * H + F, H, act, m->bp<void>(b, m->wl.qkv_w), e, s, pred, m->split_ws());
  }));
  ACID_TRY(run(m, ACID_K_ATTENTION, s, "attention", [&]() {
    return launch_attention(dt, c.n_heads, L, c.head_dim, e.q, e.k, e.vt, e.vt_ld, g, s, pred,
                            H + F, true);
  }));
  acid_epilogue_args p = {};
  p.kind = ACID_EPI_GATE_RESIDUAL;
  p.bias = m->bp(b, m->wl.o_b);
  p.bias2 = m->bp(b, m->wl.f2_b);
  p.gate = mod6 + 2 * H;
  p.out = h;
  return run(m, ACID_K_GEMM_PROJ, s, "attn+mlp projection gemm", [&]() {
    return launch_linear(dt, L, H, H + F, g, m->bp<void>(b, m->wl.o_w), p, s, pred, m->split_ws());
  });
}

// h = [text; x], all blocks with the modulation row `row`.
// h_in = [text; x] into the residual-stream buffer.
acid_status stack_assemble(acid_model* m, const float* x, const float* text, hipStream_t s) {
  const int H = m->H();
  float* h = m->kp(m->kl.h);
  return run(m, ACID_K_MISC, s, "assemble residual stream", [&]() {
    hipError_t err = hipSuccess;
    if (m->Lt() > 0)
      err = hipMemcpyAsync(h, text, (size_t)m->Lt() * H * 4, hipMemcpyDeviceToDevice, s);
    if (err == hipSuccess)
      err = hipMemcpyAsync(h + m->Lt() * H, x, (size_t)m->Lv() * H * 4, hipMemcpyDeviceToDevice,
                           s);
    return err;
  });
}

// Blocks [b0, b1) on the residual-stream buffer.
acid_status stack_blocks(acid_model* m, const float* row, int b0, int b1, hipStream_t s,
                         const int32_t* pred = nullptr) {
  float* h = m->kp(m->kl.h);
  for (int b = b0; b < b1; ++b)
    ACID_TRY(block_forward(m, b, row + 6 * (int64_t)b * m->H(), h, s, pred));
  return ACID_OK;
}

// stack_assemble as predicated copy kernels (graph capture: no copy nodes
// that would run on skipped steps).
acid_status stack_assemble_pred(acid_model* m, const float* x, const float* text,
                                const int32_t* pred, hipStream_t s) {
  const int H = m->H();
  float* h = m->kp(m->kl.h);
  return run(m, ACID_K_MISC, s, "assemble residual stream", [&]() {
    hipError_t err = hipSuccess;
    if (m->Lt() > 0) err = launch_copy(text, h, m->Lt() * H, s, pred);
    if (err == hipSuccess) err = launch_copy(x, h + m->Lt() * H, m->Lv() * H, s, pred);
    return err;
  });
}

acid_status stack_forward(acid_model* m, const float* row, const float* x, const float* text,
                          hipStream_t s) {
  ACID_TRY(stack_assemble(m, x, text, s));
  return stack_blocks(m, row, 0, m->cfg.n_blocks, s);
}

// v = LN-modulated head of h_v; EULER variant updates x in place.
acid_status head_forward(acid_model* m, const float* row, const float* hv, float* v_out,
                         float* x_euler, float dsigma, hipStream_t s,
                         const int32_t* pred = nullptr) {
  const acid_dit_config& c = m->cfg;
  const int H = c.hidden;
  const float* shift = row + 6 * (int64_t)c.n_blocks * H;
  void* act = m->kp<void>(m->kl.act);
  ACID_TRY(ln_mod(m, hv, m->Lv(), shift, shift + H, act, s, pred));
  acid_epilogue_args e = {};
  e.bias = m->wp(m->wl.head_b);
  if (x_euler) {
    e.kind = ACID_EPI_EULER;
    e.out = x_euler;
    e.v_out = v_out;
    e.dsigma = dsigma;
  } else {
    e.kind = ACID_EPI_BIAS;
    e.out = v_out;
  }
  return run(m, ACID_K_GEMM_HEAD, s, "head gemm", [&]() {
    return launch_linear(c.dtype, m->Lv(), H, H, act, m->wp<void>(m->wl.head_w), e, s, pred, m->split_ws());
  });
}

// TEMNI into m_cur; if m_prev, the relative-L1 drift is reduced into dres.
acid_status drift(acid_model* m, const float* row, const float* x, const float* m_prev,
                  float* m_cur, hipStream_t s) {
  const int H = m->H();
  double* part = m->kp<double>(m->kl.partials);
  double* dres = m->kp<double>(m->kl.dres);
  return run(m, ACID_K_DRIFT, s, "drift", [&]() {
    hipError_t err = launch_temni_drift(x, m->Lv(), H, row, row + H, m_prev, m_cur, part, s);
    if (err == hipSuccess && m_prev) err = launch_drift_finalize(part, m->Lv(), dres, s);
    return err;
  });
}

// sum |a - b| (or |a|) and sum |c| (or 0) over n elements into out2 (host).
acid_status l1_norms(acid_model* m, const float* a, const float* b, const float* c, int64_t n,
                     double* out2, hipStream_t s) {
  double* part = m->kp<double>(m->kl.partials);
  double* dres = m->kp<double>(m->kl.dres);
  const int max_groups = (int)(m->Lv() < 1024 ? m->Lv() : 1024);
  ACID_TRY(run(m, ACID_K_DRIFT, s, "l1 norms", [&]() {
    return launch_l1_norms(a, b, c, n, part, max_groups, dres, s);
  }));
  ACID_HIP(hipMemcpyAsync(out2, dres, 2 * sizeof(double), hipMemcpyDeviceToHost, s));
  ACID_HIP(hipStreamSynchronize(s));
  return ACID_OK;
}

double ratio_or_inf(double num, double den) {
  if (den == 0.0) return num == 0.0 ? 0.0 : INFINITY;
  return num / den;
}

// EasyCache's signal under Algorithm 1 (see acid_mode): the workspace's
// TEMNI buffers hold x_{i-1} (m0) and the previous output (ping-pong with v),
// the residual buffer holds the offset D.
acid_status easycache_loop(acid_model* m, float* x, const float* sig, int n, const float* text,
                           const acid_gate_params* gate, const uint8_t* forced,
                           acid_step_trace* trace, hipStream_t s) {
  const int H = m->H();
  const int64_t nv = m->Lv() * H;
  float* table = m->kp(m->kl.modtab);
  float* xprev = m->kp(m->kl.m0);
  float* vbuf[2] = {m->kp(m->kl.v), m->kp(m->kl.m1)};
  float* offset = m->kp(m->kl.r);
  float* hv = m->kp(m->kl.h) + m->Lt() * H;
  ACID_TRY(modulation_table(m, sig, n, table, s));
  acid_gate_state st = {};
  double k = NAN;
  bool have_k = false, have_offset = false;
  int cur = 0;  // vbuf[cur] receives v_i, vbuf[cur ^ 1] holds v_{i-1}
  for (int i = 0; i < n; ++i) {
    const float* row = table + (int64_t)i * m->rowsz();
    double si = NAN, tau = NAN, dx = NAN;
    if (i > 0) {
      double sums[2];
      ACID_TRY(l1_norms(m, x, xprev, vbuf[cur ^ 1], nv, sums, s));
      dx = sums[0];
      if (have_k) si = k * ratio_or_inf(sums[0], sums[1]);
    }
    int32_t gate_compute = 1;
    ACID_TRY(acid_gate(&st, gate, si, &gate_compute, &tau));
    const int compute = forced ? (forced[i] != 0) : gate_compute;
    const float dsig = sig[i + 1] - sig[i];
    float* v = vbuf[cur];
    if (compute) {
      ACID_TRY(run(m, ACID_K_MISC, s, "keep x_i", [&]() {
        return hipMemcpyAsync(xprev, x, nv * sizeof(float), hipMemcpyDeviceToDevice, s);
      }));
      ACID_TRY(stack_forward(m, row, x, text, s));
      ACID_TRY(head_forward(m, row, hv, v, x, dsig, s));  // v_i; x <- x_{i+1}
      ACID_TRY(run(m, ACID_K_CACHE, s, "offset store", [&]() {
        return launch_cache(ACID_CACHE_STORE, xprev, v, offset, nv, s);  // D = v_i - x_i
      }));
      have_offset = true;
      if (i > 0) {
        double sums[2];
        ACID_TRY(l1_norms(m, v, vbuf[cur ^ 1], nullptr, nv, sums, s));
        k = ratio_or_inf(sums[0], dx);
        have_k = true;
      }
    } else {
      if (!have_offset) return set_error(ACID_ERR_INVALID_ARG, "skip before any computed step");
      ACID_TRY(run(m, ACID_K_CACHE, s, "easycache reuse", [&]() {
        return launch_easycache_reuse(x, xprev, v, offset, nv, dsig, s);
      }));
    }
    cur ^= 1;
    if (trace) {
      trace[i].compute = compute;
      trace[i].gate_compute = gate_compute;
      trace[i].s = si;
      trace[i].sigma_sum_after = st.sigma_sum;
      trace[i].tau_used = tau;
    }
  }
  return ACID_OK;
}

// DiCache's probe signal under Algorithm 1 (see acid_mode): the TEMNI
// buffers hold the probe's video rows of this and the previous step
// (ping-pong), the residual buffer the deep residual R = h_out_v - p.
acid_status dicache_loop(acid_model* m, float* x, const float* sig, int n, const float* text,
                         const acid_gate_params* gate, const uint8_t* forced,
                         acid_step_trace* trace, hipStream_t s) {
  const int H = m->H();
  const int64_t nv = m->Lv() * H;
  const int np = m->probe_blocks;
  float* table = m->kp(m->kl.modtab);
  float* pbuf[2] = {m->kp(m->kl.m0), m->kp(m->kl.m1)};
  float* rdeep = m->kp(m->kl.r);
  float* hv = m->kp(m->kl.h) + m->Lt() * H;
  ACID_TRY(modulation_table(m, sig, n, table, s));
  acid_gate_state st = {};
  bool have_r = false;
  int cur = 0;
  for (int i = 0; i < n; ++i) {
    const float* row = table + (int64_t)i * m->rowsz();
    ACID_TRY(stack_assemble(m, x, text, s));
    ACID_TRY(stack_blocks(m, row, 0, np, s));
    float* p = pbuf[cur];
    ACID_TRY(run(m, ACID_K_MISC, s, "keep probe features", [&]() {
      return hipMemcpyAsync(p, hv, nv * sizeof(float), hipMemcpyDeviceToDevice, s);
    }));
    double si = NAN, tau = NAN;
    if (i > 0) {
      double sums[2];
      ACID_TRY(l1_norms(m, p, pbuf[cur ^ 1], pbuf[cur ^ 1], nv, sums, s));
      si = ratio_or_inf(sums[0], sums[1]);
    }
    int32_t gate_compute = 1;
    ACID_TRY(acid_gate(&st, gate, si, &gate_compute, &tau));
    const int compute = forced ? (forced[i] != 0) : gate_compute;
    if (compute) {
      ACID_TRY(stack_blocks(m, row, np, m->cfg.n_blocks, s));
      ACID_TRY(run(m, ACID_K_CACHE, s, "deep residual store", [&]() {
        return launch_cache(ACID_CACHE_STORE, p, hv, rdeep, nv, s);  // R = h_out_v - p
      }));
      have_r = true;
    } else {
      if (!have_r) return set_error(ACID_ERR_INVALID_ARG, "skip before any computed step");
      ACID_TRY(run(m, ACID_K_CACHE, s, "deep residual apply", [&]() {
        return launch_cache(ACID_CACHE_APPLY, p, hv, rdeep, nv, s);  // h_out_v = p + R
      }));
    }
    ACID_TRY(head_forward(m, row, hv, nullptr, x, sig[i + 1] - sig[i], s));
    cur ^= 1;
    if (trace) {
      trace[i].compute = compute;
      trace[i].gate_compute = gate_compute;
      trace[i].s = si;
      trace[i].sigma_sum_after = st.sigma_sum;
      trace[i].tau_used = tau;
    }
  }
  return ACID_OK;
}

acid_status check_loop_args(acid_model* m, float* x_dev, const float* sigmas_host,
                            int32_t n_steps, const float* text_dev, int32_t mode,
                            const acid_gate_params* gate, const uint8_t* forced) {
  if (!m || !x_dev || !sigmas_host) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (mode != ACID_MODE_NOCACHE && mode != ACID_MODE_ACID && mode != ACID_MODE_EASYCACHE &&
      mode != ACID_MODE_DICACHE)
    return set_error(ACID_ERR_INVALID_ARG, "bad mode %d", mode);
  if (mode != ACID_MODE_NOCACHE && !gate)
    return set_error(ACID_ERR_INVALID_ARG, "gate params NULL");
  if (mode == ACID_MODE_EASYCACHE && gate->n_warmup < 2)
    return set_error(ACID_ERR_INVALID_ARG, "EasyCache needs n_warmup >= 2 (got %d)",
                     gate->n_warmup);
  if (n_steps < 1 || n_steps > m->max_steps)
    return set_error(ACID_ERR_INVALID_ARG, "n_steps %d must be in [1, max_steps=%d]", n_steps,
                     m->max_steps);
  if ((m->cfg.n_text > 0) != (text_dev != nullptr))
    return set_error(ACID_ERR_INVALID_ARG, "text must be given iff n_text > 0");
  if (forced && !forced[0])
    return set_error(ACID_ERR_INVALID_ARG, "forced schedule must compute step 0");
  if (forced && mode == ACID_MODE_NOCACHE)
    return set_error(ACID_ERR_UNSUPPORTED, "a forced schedule needs ACID mode (the residual cache)");
  return ACID_OK;
}

// The whole loop as one stream of launches with no host round trip: per
// step the drift, the device gate (which writes the step's decision into the
// device trace), the model kernels predicated on that decision, the cache
// kernel taking STORE or APPLY from it, and the head + Euler update.
acid_status enqueue_device_gate_loop(acid_model* m, float* x, const float* sig, int n,
                                     const float* text, int mode, const acid_gate_params* gate,
                                     const uint8_t* forced, hipStream_t s) {
  const int H = m->H();
  const int64_t nv = m->Lv() * H;
  const float* table = m->kp(m->kl.modtab);
  float* mbuf[2] = {m->kp(m->kl.m0), m->kp(m->kl.m1)};
  float* r = m->kp(m->kl.r);
  float* hv = m->kp(m->kl.h) + m->Lt() * H;
  const double* dres = m->kp<double>(m->kl.dres);
  acid_step_trace* dtr = m->kp<acid_step_trace>(m->kl.dtrace);
  acid_gate_state* gst = m->kp<acid_gate_state>(m->kl.gstate);
  int cur = 0;
  for (int i = 0; i < n; ++i) {
    const float* row = table + (int64_t)i * m->rowsz();
    const int32_t* pred = nullptr;
    if (mode == ACID_MODE_ACID) {
      const float* mprev = i > 0 ? mbuf[cur ^ 1] : nullptr;
      ACID_TRY(drift(m, row, x, mprev, mbuf[cur], s));
      cur ^= 1;
      const int f = forced ? (forced[i] != 0) : -1;
      ACID_TRY(run(m, ACID_K_DRIFT, s, "device gate", [&]() {
        return launch_gate_step(dres, ACID_MODE_ACID, i > 0, *gate, f, i, gst, dtr + i,
                                m->kp<int32_t>(m->kl.dskip) + i, nullptr, s);
      }));
      pred = &dtr[i].compute;
    }
    ACID_TRY(stack_assemble_pred(m, x, text, pred, s));
    ACID_TRY(stack_blocks(m, row, 0, m->cfg.n_blocks, s, pred));
    if (mode == ACID_MODE_ACID) {
      ACID_TRY(run(m, ACID_K_CACHE, s, "cache store/apply", [&]() {
        return launch_cache(ACID_CACHE_STORE, x, hv, r, nv, s, pred);
      }));
    }
    ACID_TRY(head_forward(m, row, hv, nullptr, x, sig[i + 1] - sig[i], s));
  }
  return ACID_OK;
}

// DiCache's loop with the gate on the device: every step assembles the
// residual stream, runs the probe blocks and keeps the probe's video rows;
// the L1 sums against the previous probe stay in device memory for the gate;
// the deep blocks are predicated on the decision, the cache kernel stores
// or applies the deep residual, and the head runs every step.
acid_status enqueue_dicache_graph_loop(acid_model* m, float* x, const float* sig, int n,
                                       const float* text, const acid_gate_params* gate,
                                       const uint8_t* forced, hipStream_t s) {
  const int H = m->H();
  const int64_t nv = m->Lv() * H;
  const int np = m->probe_blocks;
  const float* table = m->kp(m->kl.modtab);
  float* pbuf[2] = {m->kp(m->kl.m0), m->kp(m->kl.m1)};
  float* rdeep = m->kp(m->kl.r);
  float* hv = m->kp(m->kl.h) + m->Lt() * H;
  double* part = m->kp<double>(m->kl.partials);
  double* dres = m->kp<double>(m->kl.dres);
  const int max_groups = (int)(m->Lv() < 1024 ? m->Lv() : 1024);
  acid_step_trace* dtr = m->kp<acid_step_trace>(m->kl.dtrace);
  acid_gate_state* gst = m->kp<acid_gate_state>(m->kl.gstate);
  int32_t* dskip = m->kp<int32_t>(m->kl.dskip);
  int cur = 0;
  for (int i = 0; i < n; ++i) {
    const float* row = table + (int64_t)i * m->rowsz();
    ACID_TRY(stack_assemble_pred(m, x, text, nullptr, s));
    ACID_TRY(stack_blocks(m, row, 0, np, s));
    float* p = pbuf[cur];
    ACID_TRY(run(m, ACID_K_MISC, s, "keep probe features", [&]() {
      return launch_copy(hv, p, nv, s, nullptr);
    }));
    if (i > 0) {
      ACID_TRY(run(m, ACID_K_DRIFT, s, "probe l1 norms", [&]() {
        return launch_l1_norms(p, pbuf[cur ^ 1], pbuf[cur ^ 1], nv, part, max_groups, dres, s);
      }));
    }
    const int f = forced ? (forced[i] != 0) : -1;
    ACID_TRY(run(m, ACID_K_DRIFT, s, "device gate", [&]() {
      return launch_gate_step(dres, ACID_MODE_DICACHE, i > 0, *gate, f, i, gst, dtr + i,
                              dskip + i, nullptr, s);
    }));
    const int32_t* pred = &dtr[i].compute;
    ACID_TRY(stack_blocks(m, row, np, m->cfg.n_blocks, s, pred));
    ACID_TRY(run(m, ACID_K_CACHE, s, "deep residual store/apply", [&]() {
      return launch_cache(ACID_CACHE_STORE, p, hv, rdeep, nv, s, pred);
    }));
    ACID_TRY(head_forward(m, row, hv, nullptr, x, sig[i + 1] - sig[i], s));
    cur ^= 1;
  }
  return ACID_OK;
}

// EasyCache's loop with the gate on the device: per step the L1 sums of
// x_i - x_{i-1} and v_{i-1} feed the gate; a computed step (predicated on the
// decision) keeps x_i, runs the stack and the head (v_i, Euler update),
// stores D = v_i - x_i and updates the rate k from |v_i - v_{i-1}|; a skipped
// step (predicated on its negation) reuses v = x + D.
acid_status enqueue_easycache_graph_loop(acid_model* m, float* x, const float* sig, int n,
                                         const float* text, const acid_gate_params* gate,
                                         const uint8_t* forced, hipStream_t s) {
  const int H = m->H();
  const int64_t nv = m->Lv() * H;
  const float* table = m->kp(m->kl.modtab);
  float* xprev = m->kp(m->kl.m0);
  float* vbuf[2] = {m->kp(m->kl.v), m->kp(m->kl.m1)};
  float* offset = m->kp(m->kl.r);
  float* hv = m->kp(m->kl.h) + m->Lt() * H;
  double* part = m->kp<double>(m->kl.partials);
  double* dres = m->kp<double>(m->kl.dres);
  const int max_groups = (int)(m->Lv() < 1024 ? m->Lv() : 1024);
  acid_step_trace* dtr = m->kp<acid_step_trace>(m->kl.dtrace);
  acid_gate_state* gst = m->kp<acid_gate_state>(m->kl.gstate);
  int32_t* dskip = m->kp<int32_t>(m->kl.dskip);
  double* ec = m->kp<double>(m->kl.ecst);
  int cur = 0;
  for (int i = 0; i < n; ++i) {
    const float* row = table + (int64_t)i * m->rowsz();
    if (i > 0) {
      ACID_TRY(run(m, ACID_K_DRIFT, s, "l1 norms", [&]() {
        return launch_l1_norms(x, xprev, vbuf[cur ^ 1], nv, part, max_groups, dres, s);
      }));
    }
    const int f = forced ? (forced[i] != 0) : -1;
    ACID_TRY(run(m, ACID_K_DRIFT, s, "device gate", [&]() {
      return launch_gate_step(dres, ACID_MODE_EASYCACHE, i > 0, *gate, f, i, gst, dtr + i,
                              dskip + i, ec, s);
    }));
    const int32_t* pred = &dtr[i].compute;
    const int32_t* spred = dskip + i;
    const float dsig = sig[i + 1] - sig[i];
    float* v = vbuf[cur];
    ACID_TRY(run(m, ACID_K_MISC, s, "keep x_i", [&]() { return launch_copy(x, xprev, nv, s, pred); }));
    ACID_TRY(stack_assemble_pred(m, x, text, pred, s));
    ACID_TRY(stack_blocks(m, row, 0, m->cfg.n_blocks, s, pred));
    ACID_TRY(head_forward(m, row, hv, v, x, dsig, s, pred));  // v_i; x <- x_{i+1}
    ACID_TRY(run(m, ACID_K_CACHE, s, "offset store", [&]() {
      return launch_cache(ACID_CACHE_STORE, xprev, v, offset, nv, s, nullptr, pred);  // D = v_i - x_i
    }));
    if (i > 0) {
      ACID_TRY(run(m, ACID_K_DRIFT, s, "rate l1 norms", [&]() {
        hipError_t e = launch_l1_norms(v, vbuf[cur ^ 1], nullptr, nv, part, max_groups, dres, s,
                                       pred);
        if (e == hipSuccess) e = launch_easycache_rate(dres, ec, pred, s);
        return e;
      }));
    }
    ACID_TRY(run(m, ACID_K_CACHE, s, "easycache reuse", [&]() {
      return launch_easycache_reuse(x, xprev, v, offset, nv, dsig, s, spred);
    }));
    cur ^= 1;
  }
  return ACID_OK;
}

acid_status read_drift(acid_model* m, double* s_out, hipStream_t s) {
  double res[3];
  ACID_HIP(hipMemcpyAsync(res, m->kp<double>(m->kl.dres), sizeof res, hipMemcpyDeviceToHost, s));
  ACID_HIP(hipStreamSynchronize(s));
  *s_out = res[2];
  return ACID_OK;
}

}  // namespace

// ====================================================================== ABI

extern "C" {

const char* acid_version(void) { return ACID_VERSION " (gfx950)"; }

const char* acid_last_error(void) { return g_err; }

acid_status acid_config_check(const acid_dit_config* cfg) { return check_config(cfg); }

size_t acid_weights_bytes(const acid_dit_config* cfg) {
  if (check_config(cfg) != ACID_OK) return 0;
  return weight_layout(*cfg).total;
}

size_t acid_workspace_bytes(const acid_dit_config* cfg, int32_t max_steps) {
  if (check_config(cfg) != ACID_OK || max_steps < 1) return 0;
  return work_layout(*cfg, max_steps).total;
}

int32_t acid_tensor_count(const acid_dit_config* cfg) {
  if (check_config(cfg) != ACID_OK) return 0;
  return 8 + 10 * cfg->n_blocks;
}

namespace {
// kind: 0 fp32 copy, 1 GEMM weight (transpose + convert)
struct TensorInfo {
  int rank;
  int64_t d0, d1;
  int gemm;
  size_t off;   // absolute offset in the arena
  int64_t ldd;  // GEMM operand row stride in elements (0: dense)
};

acid_status tensor_info(const acid_dit_config& c, int id, TensorInfo* t) {
  const int64_t H = c.hidden, F = c.ffn, Ft = c.freq_dim;
  const int nb = c.n_blocks;
  const WeightLayout L = weight_layout(c);
  if (id < 0 || id >= 8 + 10 * nb) return set_error(ACID_ERR_INVALID_ARG, "tensor id %d out of range", id);
  auto set = [&](int rank, int64_t d0, int64_t d1, int gemm, size_t off, int64_t ldd = 0) {
    *t = TensorInfo{rank, d0, d1, gemm, off, ldd};
    return ACID_OK;
  };
  const bool par = c.block_kind == ACID_BLOCK_PARALLEL;
  const size_t es = esize(c.dtype);
  if (id < 4) {
    switch (id) {
      case 0: return set(2, Ft, H, 0, L.temb_w1);
      case 1: return set(1, H, 1, 0, L.temb_b1);
      case 2: return set(2, H, H, 0, L.temb_w2);
      default: return set(1, H, 1, 0, L.temb_b2);
    }
  }
  if (id < 4 + 10 * nb) {
    const int b = (id - 4) / 10, j = (id - 4) % 10;
    const size_t base = L.blk0 + (size_t)b * L.blk_stride;
    switch (j) {
      case 0: return set(2, H, 6 * H, 0, base + L.ada_w);
      case 1: return set(1, 6 * H, 1, 0, base + L.ada_b);
      case 2: return set(2, H, 3 * H, 1, base + L.qkv_w);
      case 3: return set(1, 3 * H, 1, 0, base + L.qkv_b);
      case 4: return par ? set(2, H, H, 1, base + L.o_w, H + F) : set(2, H, H, 1, base + L.o_w);
      case 5: return set(1, H, 1, 0, base + L.o_b);
      case 6: return set(2, H, F, 1, base + L.f1_w);
      case 7: return set(1, F, 1, 0, base + L.f1_b);
      case 8:  // parallel: columns H .. H + F of the [H][H + F] operand
        return par ? set(2, F, H, 1, base + L.o_w + H * es, H + F) : set(2, F, H, 1, base + L.f2_w);
      default: return set(1, H, 1, 0, base + L.f2_b);
    }
  }
  switch (id - 4 - 10 * nb) {
    case 0: return set(2, H, 2 * H, 0, L.head_ada_w);
    case 1: return set(1, 2 * H, 1, 0, L.head_ada_b);
    case 2: return set(2, H, H, 1, L.head_w);
    default: return set(1, H, 1, 0, L.head_b);
  }
}
}  // namespace

acid_status acid_tensor_shape(const acid_dit_config* cfg, int32_t id, int32_t* rank,
                              int64_t dims[2]) {
  ACID_TRY(check_config(cfg));
  if (!rank || !dims) return set_error(ACID_ERR_INVALID_ARG, "rank/dims is NULL");
  TensorInfo t;
  ACID_TRY(tensor_info(*cfg, id, &t));
  *rank = t.rank;
  dims[0] = t.d0;
  dims[1] = t.rank == 2 ? t.d1 : 1;
  return ACID_OK;
}

acid_status acid_model_create(const acid_dit_config* cfg, void* weights_dev, void* workspace_dev,
                              int32_t max_steps, acid_model** out) {
  ACID_TRY(check_config(cfg));
  if (!weights_dev || !workspace_dev || !out)
    return set_error(ACID_ERR_INVALID_ARG, "weights, workspace and out must be non-NULL");
  if (max_steps < 1) return set_error(ACID_ERR_INVALID_ARG, "max_steps %d < 1", max_steps);
  if (((uintptr_t)weights_dev | (uintptr_t)workspace_dev) % 256)
    return set_error(ACID_ERR_INVALID_ARG, "weights and workspace must be 256-byte aligned");
  acid_model* m = new (std::nothrow) acid_model();
  if (!m) return set_error(ACID_ERR_INVALID_ARG, "host allocation failed");
  m->cfg = *cfg;
  m->max_steps = max_steps;
  m->wb = static_cast<char*>(weights_dev);
  m->ws = static_cast<char*>(workspace_dev);
  m->wl = weight_layout(*cfg);
  m->kl = work_layout(*cfg, max_steps);
  {
    const size_t H = cfg->hidden, es = esize(cfg->dtype);
    const WeightLayout& w = m->wl;
    if (w.f1_w != w.qkv_w + 3 * H * H * es || w.f1_b != w.qkv_b + 3 * H * 4 ||
        w.f2_w != w.o_w + H * H * es) {
      delete m;
      return set_error(ACID_ERR_SHAPE, "weight layout: concatenated operands are not adjacent");
    }
  }
  *out = m;
  return ACID_OK;
}

acid_status acid_model_load_tensor(acid_model* m, int32_t id, const float* src_dev, int64_t n,
                                   hipStream_t stream) {
  if (!m || !src_dev) return set_error(ACID_ERR_INVALID_ARG, "model and source must be non-NULL");
  TensorInfo t;
  ACID_TRY(tensor_info(m->cfg, id, &t));
  const int64_t count = t.rank == 2 ? t.d0 * t.d1 : t.d0;
  if (n != count)
    return set_error(ACID_ERR_SHAPE, "tensor %d has %lld elements, got %lld", id, (long long)count,
                     (long long)n);
  void* dst = m->wb + t.off;
  return run(m, ACID_K_MISC, stream, "load tensor", [&]() {
    if (t.gemm)
      return launch_transpose_convert(src_dev, t.d0, t.d1, m->cfg.dtype, dst, stream, t.ldd);
    return hipMemcpyAsync(dst, src_dev, (size_t)count * 4, hipMemcpyDeviceToDevice, stream);
  });
}

acid_status acid_model_load_tensor_host(acid_model* m, int32_t id, const float* src_host,
                                        int64_t n, hipStream_t stream) {
  if (!m || !src_host) return set_error(ACID_ERR_INVALID_ARG, "model and source must be non-NULL");
  TensorInfo t;
  ACID_TRY(tensor_info(m->cfg, id, &t));
  const int64_t rows = t.d0, cols = t.rank == 2 ? t.d1 : 1;
  if (n != rows * cols)
    return set_error(ACID_ERR_SHAPE, "tensor %d has %lld elements, got %lld", id,
                     (long long)(rows * cols), (long long)n);
  char* dst = m->wb + t.off;
  if (!t.gemm) {  // fp32 as given: one copy, host to arena
    ACID_TRY(run(m, ACID_K_MISC, stream, "load tensor (host)", [&]() {
      return hipMemcpyAsync(dst, src_host, (size_t)n * 4, hipMemcpyHostToDevice, stream);
    }));
    ACID_HIP(hipStreamSynchronize(stream));
    return ACID_OK;
  }
  // GEMM weight: whole [in] rows of the [in][out] source are staged through
  // the workspace's residual-stream buffer and transposed into columns
  // i0 .. i0 + k of the [out][in] operand.
  float* stage = m->kp(m->kl.h);
  const int64_t stage_rows = (int64_t)(m->L() * m->H()) / cols;
  if (stage_rows < 1) return set_error(ACID_ERR_SHAPE, "staging buffer smaller than one row");
  const int64_t ldd = t.ldd ? t.ldd : rows;
  const size_t es = esize(m->cfg.dtype);
  for (int64_t i0 = 0; i0 < rows; i0 += stage_rows) {
    const int64_t k = rows - i0 < stage_rows ? rows - i0 : stage_rows;
    ACID_TRY(run(m, ACID_K_MISC, stream, "load tensor (host)", [&]() {
      hipError_t e = hipMemcpyAsync(stage, src_host + i0 * cols, (size_t)(k * cols) * 4,
                                    hipMemcpyHostToDevice, stream);
      if (e != hipSuccess) return e;
      return launch_transpose_convert(stage, k, cols, m->cfg.dtype, dst + (size_t)i0 * es, stream,
                                      ldd);
    }));
    // the next chunk overwrites the staging buffer
    ACID_HIP(hipStreamSynchronize(stream));
  }
  return ACID_OK;
}

float acid_q_scale(int32_t head_dim) { return head_dim > 0 ? attn_q_scale(head_dim) : 0.0f; }

void acid_model_destroy(acid_model* m) {
  if (!m) return;
  // teardown: errors here have nowhere to go
  (void)harvest(m);
  for (auto e : m->pool) (void)hipEventDestroy(e);
  if (m->gexec) (void)hipGraphExecDestroy(m->gexec);
  if (m->cap) (void)hipStreamDestroy(m->cap);
  delete m;
}

acid_status acid_model_set_timing(acid_model* m, int32_t enable) {
  if (!m) return set_error(ACID_ERR_INVALID_ARG, "model is NULL");
  if (!enable) ACID_TRY(harvest(m));
  m->timing = enable != 0;
  return ACID_OK;
}

acid_status acid_model_reset_timing(acid_model* m) {
  if (!m) return set_error(ACID_ERR_INVALID_ARG, "model is NULL");
  ACID_TRY(harvest(m));
  for (int i = 0; i < ACID_K_COUNT; ++i) {
    m->total_ms[i] = 0;
    m->launches[i] = 0;
  }
  return ACID_OK;
}

acid_status acid_model_timing(acid_model* m, int32_t cls, double* total_ms, int64_t* launches) {
  if (!m || !total_ms || !launches) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (cls < 0 || cls >= ACID_K_COUNT) return set_error(ACID_ERR_INVALID_ARG, "kernel class %d", cls);
  ACID_TRY(harvest(m));
  *total_ms = m->total_ms[cls];
  *launches = m->launches[cls];
  return ACID_OK;
}

acid_status acid_timestep_modulation(acid_model* m, const float* sigmas_host, int32_t n,
                                     float* table_dev, hipStream_t stream) {
  if (!m || !sigmas_host || !table_dev) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (n < 1 || n > m->max_steps)
    return set_error(ACID_ERR_INVALID_ARG, "n %d must be in [1, max_steps=%d]", n, m->max_steps);
  return modulation_table(m, sigmas_host, n, table_dev, stream);
}

acid_status acid_ln_modulate(int32_t out_dtype, const float* x_dev, int64_t rows, int32_t hidden,
                             const float* shift_dev, const float* scale_dev, void* out_dev,
                             hipStream_t stream) {
  if (out_dtype != ACID_F32 && out_dtype != ACID_BF16)
    return set_error(ACID_ERR_INVALID_ARG, "bad dtype %d", out_dtype);
  if (rows < 0) return set_error(ACID_ERR_INVALID_ARG, "rows < 0");
  if (hidden < 4 || hidden % 4 || hidden > 4096)
    return set_error(ACID_ERR_SHAPE, "hidden %d: multiple of 4 in [4, 4096]", hidden);
  if (rows > 0 && (!x_dev || !shift_dev || !scale_dev || !out_dev))
    return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  hipError_t e = launch_ln_modulate(out_dtype, x_dev, rows, hidden, shift_dev, scale_dev, out_dev,
                                    stream);
  return e == hipSuccess ? ACID_OK : check_hip(e, "ln_modulate");
}

acid_status acid_attention(int32_t dtype, int32_t n_heads, int64_t seq_len, int32_t head_dim,
                           const void* q_dev, const void* k_dev, const void* vt_dev,
                           int64_t vt_ld, void* o_dev, int32_t q_prescaled,
                           hipStream_t stream) {
  if (dtype != ACID_F32 && dtype != ACID_BF16)
    return set_error(ACID_ERR_INVALID_ARG, "bad dtype %d", dtype);
  if (q_prescaled != 0 && q_prescaled != 1)
    return set_error(ACID_ERR_INVALID_ARG, "q_prescaled %d: 0 or 1", q_prescaled);
  if (n_heads < 1 || seq_len < 0) return set_error(ACID_ERR_INVALID_ARG, "n_heads < 1 or seq_len < 0");
  if (head_dim != 64 && head_dim != 128)
    return set_error(ACID_ERR_SHAPE, "head_dim %d: supported 64 or 128", head_dim);
  if (vt_ld < round_up(seq_len, 8) || vt_ld % 8)
    return set_error(ACID_ERR_SHAPE, "vt_ld %lld must be a multiple of 8 and >= round_up(L, 8)",
                     (long long)vt_ld);
  ACID_TRY(check_attention_size(dtype, n_heads, seq_len, head_dim, vt_ld));
  if (seq_len > 0 && (!q_dev || !k_dev || !vt_dev || !o_dev))
    return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  hipError_t e = launch_attention(dtype, n_heads, seq_len, head_dim, q_dev, k_dev, vt_dev, vt_ld,
                                  o_dev, stream, nullptr, 0, q_prescaled != 0);
  return e == hipSuccess ? ACID_OK : check_hip(e, "attention");
}

acid_status acid_linear(int32_t dtype, int64_t M, int32_t N, int32_t K, const void* a_dev,
                        const void* wt_dev, const acid_epilogue_args* epi, hipStream_t stream) {
  if (dtype != ACID_F32 && dtype != ACID_BF16)
    return set_error(ACID_ERR_INVALID_ARG, "bad dtype %d", dtype);
  if (!epi) return set_error(ACID_ERR_INVALID_ARG, "epilogue args NULL");
  if (epi->q_prescale != 0 && epi->q_prescale != 1)
    return set_error(ACID_ERR_INVALID_ARG, "q_prescale %d: 0 or 1", epi->q_prescale);
  if (M < 0 || N <= 0 || K <= 0) return set_error(ACID_ERR_INVALID_ARG, "bad M/N/K");
  if (N % 128 || K % 128)
    return set_error(ACID_ERR_SHAPE, "N %d and K %d must be multiples of 128", N, K);
  ACID_TRY(check_linear_size(M, N, K));
  if (M == 0) return ACID_OK;
  if (!a_dev || !wt_dev || !epi->bias) return set_error(ACID_ERR_INVALID_ARG, "NULL operand or bias");
  switch (epi->kind) {
    case ACID_EPI_BIAS:
    case ACID_EPI_BIAS_GELU:
    case ACID_EPI_EULER:
      if (!epi->out) return set_error(ACID_ERR_INVALID_ARG, "out is NULL");
      break;
    case ACID_EPI_GATE_RESIDUAL:
      if (!epi->out || !epi->gate) return set_error(ACID_ERR_INVALID_ARG, "out/gate NULL");
      break;
    case ACID_EPI_QKV:
      if (!epi->q || !epi->k || !epi->vt) return set_error(ACID_ERR_INVALID_ARG, "q/k/vt NULL");
      if (epi->head_dim < 1 || epi->n_heads < 1 ||
          (int64_t)3 * epi->n_heads * epi->head_dim != N || epi->head_dim % 32)
        return set_error(ACID_ERR_SHAPE, "QKV: N must be 3 * n_heads * head_dim, head_dim % 32 == 0");
      if (epi->vt_ld < M) return set_error(ACID_ERR_SHAPE, "QKV: vt_ld < M");
      if (epi->vt_ld % 8 || (uintptr_t)epi->vt % 16)
        return set_error(ACID_ERR_INVALID_ARG, "QKV: vt must be 16-byte aligned, vt_ld % 8 == 0");
      break;
    case ACID_EPI_QKV_GELU: {
      if (!epi->q || !epi->k || !epi->vt || !epi->out)
        return set_error(ACID_ERR_INVALID_ARG, "q/k/vt/out NULL");
      const int64_t nq = (int64_t)3 * epi->n_heads * epi->head_dim;
      if (epi->head_dim < 1 || epi->n_heads < 1 || epi->head_dim % 32 || nq >= N || nq % 32)
        return set_error(ACID_ERR_SHAPE,
                         "QKV_GELU: 3 * n_heads * head_dim must be < N, head_dim % 32 == 0");
      if (epi->vt_ld < M) return set_error(ACID_ERR_SHAPE, "QKV_GELU: vt_ld < M");
      if (epi->vt_ld % 8 || (uintptr_t)epi->vt % 16)
        return set_error(ACID_ERR_INVALID_ARG,
                         "QKV_GELU: vt must be 16-byte aligned, vt_ld % 8 == 0");
      if (epi->out_ld < N - nq) return set_error(ACID_ERR_SHAPE, "QKV_GELU: out_ld < N - 3 H");
      break;
    }
    default: return set_error(ACID_ERR_INVALID_ARG, "bad epilogue kind %d", epi->kind);
  }
  hipError_t e = launch_linear(dtype, M, N, K, a_dev, wt_dev, *epi, stream);
  return e == hipSuccess ? ACID_OK : check_hip(e, "linear");
}

acid_status acid_block_forward(acid_model* m, int32_t block, const float* mod6_dev, float* h_dev,
                               hipStream_t stream) {
  if (!m || !mod6_dev || !h_dev) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (block < 0 || block >= m->cfg.n_blocks)
    return set_error(ACID_ERR_INVALID_ARG, "block %d out of range", block);
  return block_forward(m, block, mod6_dev, h_dev, stream);
}

acid_status acid_model_set_probe_blocks(acid_model* m, int32_t n_probe) {
  if (!m) return set_error(ACID_ERR_INVALID_ARG, "NULL model");
  if (n_probe < 0 || n_probe > m->cfg.n_blocks)
    return set_error(ACID_ERR_INVALID_ARG, "n_probe %d outside [0, n_blocks=%d]", n_probe,
                     m->cfg.n_blocks);
  m->probe_blocks = n_probe;
  return ACID_OK;
}

acid_status acid_l1_norms(acid_model* m, const float* a_dev, const float* b_dev,
                          const float* c_dev, int64_t n, double* out_host, hipStream_t stream) {
  if (!m || !out_host) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (n < 0 || n > m->Lv() * m->H())
    return set_error(ACID_ERR_INVALID_ARG, "n %lld outside [0, n_video * hidden]", (long long)n);
  if (n == 0) {  // empty sums; the buffers are not touched
    out_host[0] = out_host[1] = 0.0;
    return ACID_OK;
  }
  if (!a_dev) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)a_dev | (uintptr_t)b_dev | (uintptr_t)c_dev) % 16)
    return set_error(ACID_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
  return l1_norms(m, a_dev, b_dev, c_dev, n, out_host, stream);
}

acid_status acid_easycache_reuse(float* x_dev, float* x_prev_dev, float* v_dev,
                                 const float* offset_dev, int64_t n, float dsigma,
                                 hipStream_t stream) {
  if (n < 0) return set_error(ACID_ERR_INVALID_ARG, "n < 0");
  if (n == 0) return ACID_OK;
  if (!x_dev || !x_prev_dev || !v_dev || !offset_dev)
    return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)x_dev | (uintptr_t)x_prev_dev | (uintptr_t)v_dev | (uintptr_t)offset_dev) % 16)
    return set_error(ACID_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
  hipError_t e = launch_easycache_reuse(x_dev, x_prev_dev, v_dev, offset_dev, n, dsigma, stream);
  return e == hipSuccess ? ACID_OK : check_hip(e, "easycache reuse");
}

acid_status acid_cache_apply(acid_cache_op op, const float* x_dev, float* h_out_dev, float* r_dev,
                             int64_t n, hipStream_t stream) {
  if (op != ACID_CACHE_STORE && op != ACID_CACHE_APPLY)
    return set_error(ACID_ERR_INVALID_ARG, "bad cache op %d", (int)op);
  if (n < 0) return set_error(ACID_ERR_INVALID_ARG, "n < 0");
  if (n == 0) return ACID_OK;
  if (!x_dev || !h_out_dev || !r_dev) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)x_dev | (uintptr_t)h_out_dev | (uintptr_t)r_dev) % 16)
    return set_error(ACID_ERR_INVALID_ARG, "cache buffers must be 16-byte aligned");
  hipError_t e = launch_cache(op, x_dev, h_out_dev, r_dev, n, stream);
  return e == hipSuccess ? ACID_OK : check_hip(e, "cache");
}

acid_status acid_dit_step(acid_model* m, const float* x_dev, float sigma, const float* text_dev,
                          float* v_dev, float* resid_dev, hipStream_t stream) {
  if (!m || !x_dev || !v_dev) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  if ((m->cfg.n_text > 0) != (text_dev != nullptr))
    return set_error(ACID_ERR_INVALID_ARG, "text must be given iff n_text > 0");
  float* row = m->kp(m->kl.modtab);
  ACID_TRY(modulation_table(m, &sigma, 1, row, stream));
  ACID_TRY(stack_forward(m, row, x_dev, text_dev, stream));
  float* hv = m->kp(m->kl.h) + m->Lt() * m->H();
  if (resid_dev) {
    ACID_TRY(run(m, ACID_K_CACHE, stream, "cache store", [&]() {
      return launch_cache(ACID_CACHE_STORE, x_dev, hv, resid_dev, m->Lv() * m->H(), stream);
    }));
  }
  return head_forward(m, row, hv, v_dev, nullptr, 0.f, stream);
}

acid_status acid_drift_signal(acid_model* m, const float* x_dev, float sigma,
                              const float* m_prev_dev, float* m_cur_dev, double* s_out,
                              hipStream_t stream) {
  if (!m || !x_dev || !m_cur_dev || !s_out) return set_error(ACID_ERR_INVALID_ARG, "NULL argument");
  float* row = m->kp(m->kl.modtab);
  ACID_TRY(modulation_table(m, &sigma, 1, row, stream));
  ACID_TRY(drift(m, row, x_dev, m_prev_dev, m_cur_dev, stream));
  if (!m_prev_dev) {
    ACID_HIP(hipStreamSynchronize(stream));
    *s_out = NAN;
    return ACID_OK;
  }
  return read_drift(m, s_out, stream);
}

acid_status acid_denoise_loop(acid_model* m, float* x_dev, const float* sigmas_host,
                              int32_t n_steps, const float* text_dev, int32_t mode,
                              const acid_gate_params* gate, const uint8_t* forced,
                              acid_step_trace* trace, hipStream_t stream) {
  ACID_TRY(check_loop_args(m, x_dev, sigmas_host, n_steps, text_dev, mode, gate, forced));

  if (mode == ACID_MODE_EASYCACHE)
    return easycache_loop(m, x_dev, sigmas_host, n_steps, text_dev, gate, forced, trace, stream);
  if (mode == ACID_MODE_DICACHE)
    return dicache_loop(m, x_dev, sigmas_host, n_steps, text_dev, gate, forced, trace, stream);

  const int H = m->H();
  const int64_t nv = m->Lv() * H;
  float* table = m->kp(m->kl.modtab);
  float* mbuf[2] = {m->kp(m->kl.m0), m->kp(m->kl.m1)};
  float* r = m->kp(m->kl.r);
  float* hv = m->kp(m->kl.h) + m->Lt() * H;
  ACID_TRY(modulation_table(m, sigmas_host, n_steps, table, stream));

  acid_gate_state st = {};
  int cur = 0;
  for (int i = 0; i < n_steps; ++i) {
    const float* row = table + (int64_t)i * m->rowsz();
    double s = NAN, tau = NAN;
    int32_t gate_compute = 1;
    if (mode == ACID_MODE_ACID) {
      const float* mprev = i > 0 ? mbuf[cur ^ 1] : nullptr;
      ACID_TRY(drift(m, row, x_dev, mprev, mbuf[cur], stream));
      if (mprev) ACID_TRY(read_drift(m, &s, stream));
      cur ^= 1;
      ACID_TRY(acid_gate(&st, gate, s, &gate_compute, &tau));
    }
    const int compute = forced ? (forced[i] != 0) : gate_compute;
    if (compute) {
      ACID_TRY(stack_forward(m, row, x_dev, text_dev, stream));
      if (mode == ACID_MODE_ACID) {
        ACID_TRY(run(m, ACID_K_CACHE, stream, "cache store", [&]() {
          return launch_cache(ACID_CACHE_STORE, x_dev, hv, r, nv, stream);
        }));
      }
    } else {
      ACID_TRY(run(m, ACID_K_CACHE, stream, "cache apply", [&]() {
        return launch_cache(ACID_CACHE_APPLY, x_dev, hv, r, nv, stream);
      }));
    }
    const float dsig = sigmas_host[i + 1] - sigmas_host[i];
    ACID_TRY(head_forward(m, row, hv, nullptr, x_dev, dsig, stream));
    if (trace) {
      trace[i].compute = compute;
      trace[i].gate_compute = gate_compute;
      trace[i].s = s;
      trace[i].sigma_sum_after = st.sigma_sum;
      trace[i].tau_used = tau;
    }
  }
  return ACID_OK;
}

acid_status acid_denoise_loop_graph(acid_model* m, float* x_dev, const float* sigmas_host,
                                    int32_t n_steps, const float* text_dev, int32_t mode,
                                    const acid_gate_params* gate, const uint8_t* forced,
                                    acid_step_trace* trace, hipStream_t stream) {
  ACID_TRY(check_loop_args(m, x_dev, sigmas_host, n_steps, text_dev, mode, gate, forced));
  ACID_TRY(modulation_table(m, sigmas_host, n_steps, m->kp(m->kl.modtab), stream));

  acid_model::GraphKey key;
  key.x = x_dev;
  key.text = text_dev;
  key.n = n_steps;
  key.mode = mode;
  key.probe = mode == ACID_MODE_DICACHE ? m->probe_blocks : 0;
  if (gate) key.gate = *gate;
  key.sigmas.assign(sigmas_host, sigmas_host + n_steps + 1);
  if (forced) key.forced.assign(forced, forced + n_steps);
  if (!m->gexec || !(key == m->gkey)) {
    if (m->gexec) {
      ACID_HIP(hipGraphExecDestroy(m->gexec));
      m->gexec = nullptr;
    }
    if (!m->cap) ACID_HIP(hipStreamCreateWithFlags(&m->cap, hipStreamNonBlocking));
    ACID_HIP(hipStreamBeginCapture(m->cap, hipStreamCaptureModeRelaxed));
    m->capturing = true;
    acid_status st;
    if (mode == ACID_MODE_DICACHE)
      st = enqueue_dicache_graph_loop(m, x_dev, sigmas_host, n_steps, text_dev, gate, forced,
                                      m->cap);
    else if (mode == ACID_MODE_EASYCACHE)
      st = enqueue_easycache_graph_loop(m, x_dev, sigmas_host, n_steps, text_dev, gate, forced,
                                        m->cap);
    else
      st = enqueue_device_gate_loop(m, x_dev, sigmas_host, n_steps, text_dev, mode, gate, forced,
                                    m->cap);
    m->capturing = false;
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(m->cap, &g);
    if (st != ACID_OK || e != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return st != ACID_OK ? st : check_hip(e, "hipStreamEndCapture");
    }
    const hipError_t ei = hipGraphInstantiate(&m->gexec, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (ei != hipSuccess) {
      m->gexec = nullptr;
      return check_hip(ei, "hipGraphInstantiate");
    }
    m->gkey = key;
  }
  ACID_HIP(hipGraphLaunch(m->gexec, stream));
  if (trace) {
    if (mode != ACID_MODE_NOCACHE) {
      ACID_HIP(hipMemcpyAsync(trace, m->kp(m->kl.dtrace), n_steps * sizeof(acid_step_trace),
                              hipMemcpyDeviceToHost, stream));
      ACID_HIP(hipStreamSynchronize(stream));
    } else {
      for (int i = 0; i < n_steps; ++i) {
        trace[i].compute = 1;
        trace[i].gate_compute = 1;
        trace[i].s = NAN;
        trace[i].sigma_sum_after = 0.0;
        trace[i].tau_used = NAN;
      }
    }
  }
  return ACID_OK;
}

acid_status acid_gate_device_sequence(const acid_gate_params* gate, const double* s_dev,
                                      int32_t n, acid_step_trace* trace_dev,
                                      hipStream_t stream) {
  if (!gate || n < 0 || (n > 0 && (!s_dev || !trace_dev)))
    return set_error(ACID_ERR_INVALID_ARG, "bad gate sequence arguments");
  const hipError_t e = launch_gate_sequence(s_dev, n, *gate, trace_dev, stream);
  return e == hipSuccess ? ACID_OK : check_hip(e, "gate sequence");
}

}  // extern "C"

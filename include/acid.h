/*
 * acid.h -- C ABI of libacid: the ACID-gated video-DiT denoise loop on one
 * AMD Instinct MI355X (gfx950).
 *
 * The method: "ACID: Adaptive Caching for vIDeo generation".  A dynamic
 * caching method accumulates a per-step drift signal and skips the diffusion
 * transformer's forward pass while the accumulated drift stays under a
 * threshold; ACID (Algorithm 1, Section 3.3) chooses between a low and a high
 * threshold by watching how fast the signal changes.  The signal and reuse
 * rule implemented here are TeaCache's (Section 2, paragraph "TeaCache"):
 * relative L1 change of the timestep-embedding-modulated noisy input (TEMNI),
 * and reuse of the last output through a stored residual.
 *
 * Conventions for every call
 *   - Pointers named *_dev are device pointers, *_host are host pointers.
 *   - The caller owns all memory.  The library never allocates or frees
 *     device memory: the weight arena and the workspace are caller-allocated
 *     blocks whose sizes the library reports.  An acid_model only borrows
 *     them until acid_model_destroy.
 *   - Every kernel is launched on the stream passed in.  Calls that return a
 *     host value computed on the device (acid_drift_signal, acid_denoise_loop)
 *     synchronise that stream before returning.
 *   - Calls return acid_status and never abort.  acid_last_error() gives a
 *     thread-local message for the last non-OK status.  A HIP error is
 *     returned as ACID_ERR_HIP with the HIP error string in the message.
 *   - Calls on one acid_model must not overlap (they share its workspace).
 *   - Matrices are row-major.  "[a][b]" means a rows of b contiguous items.
 *   - bf16 is bfloat16, round-to-nearest-even from fp32.
 */
#ifndef ACID_H
#define ACID_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ACID_OK = 0,
  ACID_ERR_INVALID_ARG = 1, /* null pointer, negative size, bad enum */
  ACID_ERR_SHAPE = 2,       /* a size the kernels do not support */
  ACID_ERR_HIP = 3,         /* a HIP runtime call failed */
  ACID_ERR_UNSUPPORTED = 4  /* a combination of options that is not built */
} acid_status;

/* Arithmetic type of the GEMM and attention operands.  ACID_F32 computes
 * everything in fp32; ACID_BF16 stores GEMM weights and activations that feed
 * GEMMs or attention in bf16 and accumulates in fp32.  The residual stream,
 * latents, TEMNI, modulation table, drift and cache are fp32 in both. */
typedef enum { ACID_F32 = 0, ACID_BF16 = 1 } acid_dtype;

/* NOCACHE runs f_theta on every step and forms no signal.  ACID runs
 * Algorithm 1 on TeaCache's signal; a fixed threshold is ACID with
 * tau_low == tau_high.  EASYCACHE runs Algorithm 1 on EasyCache's signal
 * (Section 2, paragraph "EasyCache"; Section 3.3 names it as the gated
 * variable): transformation rate k = |v_i - v_{i-1}|_1 / |x_i - x_{i-1}|_1 on
 * each computed step i >= 1, signal s_i = k |x_i - x_{i-1}|_1 / |v_{i-1}|_1
 * with k of the last computed step, and a skipped step outputs
 * v_i = x_i + D with D = v - x of the last computed step (the whole model,
 * head included, is skipped).  Needs gate->n_warmup >= 2.
 * DICACHE runs Algorithm 1 on DiCache's probe signal (Section 2, paragraph
 * "DiCache"; Section 3.3): every step runs the first n_probe blocks
 * (acid_model_set_probe_blocks, default 1) on [text; x_i]; the signal is
 * the relative L1 change of the probe's video rows p_i against p_{i-1}; a
 * computed step runs the remaining blocks and stores R = h_out_v - p_i, a
 * skipped step uses h_out_v = p_i + R; head and Euler on every step. */
typedef enum {
  ACID_MODE_NOCACHE = 0,
  ACID_MODE_ACID = 1,
  ACID_MODE_EASYCACHE = 2,
  ACID_MODE_DICACHE = 3
} acid_mode;

/* Residual cache (TeaCache's reuse rule).  STORE on a computed step:
 * r = h_out - x.  APPLY on a skipped step: h_out = x + r. */
typedef enum { ACID_CACHE_STORE = 0, ACID_CACHE_APPLY = 1 } acid_cache_op;

/* Block form.  SEQUENTIAL: LN-modulate, attention, gated projection into
 * the residual stream, LN-modulate, GELU MLP, gated projection (shift/scale/
 * gate 1 and 2).  PARALLEL: HunyuanVideo's single-stream block (the first
 * model of Section 4.1): one LN-modulate (shift1, scale1) feeds
 * [q | k | v | mlp] = a [W_qkv | W_1] + [b_qkv | b_1]; attention and
 * GELU(mlp) are projected together by [W_o ; W_2] (K = H + F) and added
 * with gate1, biases b_o + b_2; the second modulation triple is unused.
 * Both use the same parameter manifest. */
typedef enum { ACID_BLOCK_SEQUENTIAL = 0, ACID_BLOCK_PARALLEL = 1 } acid_block_kind;

/* Shape of the DiT stack.  Token rows are ordered text first, then video.
 * hidden = n_heads * head_dim.  Supported: head_dim 64 or 128; hidden
 * (<= 4096) and ffn multiples of 128 (every GEMM's N and K); freq_dim even
 * and <= 1024; L = n_text + n_video within acid_attention's and
 * acid_linear's size limits (ACID_ERR_SHAPE otherwise). */
typedef struct {
  int32_t n_blocks;
  int32_t hidden;
  int32_t n_heads;
  int32_t head_dim;
  int32_t ffn;
  int32_t freq_dim; /* sinusoidal timestep-embedding width, 256 */
  int32_t n_video;  /* video tokens L_v (the latent rows) */
  int32_t n_text;   /* text tokens L_t (0 if none) */
  int32_t dtype;    /* acid_dtype */
  int32_t block_kind; /* acid_block_kind */
} acid_dit_config;

/* Algorithm 1's parameters (its "Require" line): tau_low, tau_high and the
 * stability bound delta.  The first n_warmup steps always run the model and
 * leave the gate state untouched (the base method's warmup). */
typedef struct {
  double tau_low;
  double tau_high;
  double delta;
  int32_t n_warmup;
} acid_gate_params;

/* Algorithm 1's state.  Zero-initialised = its initial state (accumulated
 * drift 0, no previous signal).  Plain data: copying it checkpoints the gate. */
typedef struct {
  double sigma_sum; /* accumulated drift */
  double s_prev;    /* previous signal, valid when has_prev != 0 */
  int32_t has_prev;
  int32_t step;     /* steps consumed so far (warmup included) */
} acid_gate_state;

/* One denoising step as the loop executed it. */
typedef struct {
  int32_t compute;         /* 1: f_theta ran; 0: the cached residual was reused */
  int32_t gate_compute;    /* the gate's own decision (differs from compute only
                              under a forced schedule) */
  double s;                /* drift signal of this step; NaN if none */
  double sigma_sum_after;  /* accumulated drift after the step */
  double tau_used;         /* active threshold; NaN on warmup / NOCACHE */
} acid_step_trace;

/* Kernel classes timed by the optional HIP-event timer. */
typedef enum {
  ACID_K_TEMB = 0,     /* timestep embedding + modulation table */
  ACID_K_LN_MOD = 1,   /* LayerNorm + adaLN modulate (GEMM operand) */
  ACID_K_GEMM_QKV = 2,
  ACID_K_ATTENTION = 3,
  ACID_K_GEMM_PROJ = 4,
  ACID_K_GEMM_FFN1 = 5,
  ACID_K_GEMM_FFN2 = 6,
  ACID_K_GEMM_HEAD = 7, /* head GEMM (+ Euler update in the loop) */
  ACID_K_DRIFT = 8,     /* TEMNI + relative-L1 partial sums + final reduce */
  ACID_K_CACHE = 9,     /* residual store / apply */
  ACID_K_MISC = 10,     /* residual-stream assembly, weight conversion */
  ACID_K_COUNT = 11
} acid_kernel_class;

typedef struct acid_model acid_model;

/* ------------------------------------------------------------------ setup */

/* Library version string. */
const char* acid_version(void);

/* Thread-local message for the last non-OK status ("" if none). */
const char* acid_last_error(void);

/* Checks a configuration against the supported shapes.  ACID_OK or
 * ACID_ERR_SHAPE / ACID_ERR_INVALID_ARG with a message. */
acid_status acid_config_check(const acid_dit_config* cfg);

/* Bytes of the device weight arena for cfg (0 if cfg is invalid). */
size_t acid_weights_bytes(const acid_dit_config* cfg);

/* Bytes of the device workspace for cfg and loops of up to max_steps steps
 * (0 if cfg is invalid). */
size_t acid_workspace_bytes(const acid_dit_config* cfg, int32_t max_steps);

/* Number of parameter tensors: 4 + 10 * n_blocks + 4, in this order:
 *   temb.w1 [freq_dim][H], temb.b1 [H], temb.w2 [H][H], temb.b2 [H];
 *   per block: ada.w [H][6H], ada.b [6H], qkv.w [H][3H], qkv.b [3H],
 *              o.w [H][H], o.b [H], ffn1.w [H][F], ffn1.b [F],
 *              ffn2.w [F][H], ffn2.b [H];
 *   head.ada.w [H][2H], head.ada.b [2H], head.w [H][H], head.b [H].
 * Weights are [in][out]: y = x W + b.  The 6H adaLN output splits into
 * (shift1, scale1, gate1, shift2, scale2, gate2), each H wide; the head's
 * into (shift, scale).  QKV columns are Q | K | V, each H wide; head j owns
 * columns j*head_dim .. (j+1)*head_dim of each. */
int32_t acid_tensor_count(const acid_dit_config* cfg);

/* Shape of tensor `id` (rank 1 or 2): writes rank and dims, returns status. */
acid_status acid_tensor_shape(const acid_dit_config* cfg, int32_t id,
                              int32_t* rank, int64_t dims[2]);

/* Binds a model to a caller-allocated weight arena (acid_weights_bytes, any
 * 256-byte-aligned device allocation) and workspace (acid_workspace_bytes for
 * max_steps).  Allocates only the small host-side struct. */
acid_status acid_model_create(const acid_dit_config* cfg, void* weights_dev,
                              void* workspace_dev, int32_t max_steps,
                              acid_model** out);

/* Converts tensor `id` from fp32 [in][out] (as listed above) at src_dev into
 * the arena's layout: GEMM weights become [out][in] in the config's dtype,
 * everything else stays fp32.  n must equal the tensor's element count.  The
 * source may be freed once the stream has passed this call. */
acid_status acid_model_load_tensor(acid_model* m, int32_t id,
                                   const float* src_dev, int64_t n,
                                   hipStream_t stream);

/* The same conversion from a host source (the form Algorithm 1's inputs
 * suggest: the caller holds f_theta's parameters in host memory).  src_host
 * is fp32 [in][out] (any host memory; n elements as above).  GEMM weights
 * are staged through the model's workspace in whole source rows (its
 * residual-stream buffer, whose contents are lost) and transposed on the
 * device; other tensors are copied as they are.  Synchronises the stream:
 * src_host may be freed or reused when the call returns.  Errors as
 * acid_model_load_tensor. */
acid_status acid_model_load_tensor_host(acid_model* m, int32_t id,
                                        const float* src_host, int64_t n,
                                        hipStream_t stream);

/* Frees the host struct only (never device memory). */
void acid_model_destroy(acid_model* m);

/* Optional HIP-event timer: when enabled, every kernel the model launches is
 * bracketed by events on its stream and its duration added to its class.
 * acid_model_timing synchronises the pending events and returns the summed
 * milliseconds and launch count of one class. */
acid_status acid_model_set_timing(acid_model* m, int32_t enable);
acid_status acid_model_reset_timing(acid_model* m);
acid_status acid_model_timing(acid_model* m, int32_t kernel_class,
                              double* total_ms, int64_t* launches);

/* ------------------------------------------------------ the five calls */

/* One evaluation of f_theta (Algorithm 1's "run full model"):
 * h_in = [text; x], all blocks, then the head.  x_dev fp32 [L_v][H];
 * text_dev fp32 [L_t][H] (NULL iff n_text == 0); sigma the noise level
 * (t = 1000 sigma enters the sinusoidal embedding).  Writes the velocity
 * v_dev fp32 [L_v][H] and, if resid_dev != NULL, the residual
 * r = h_out_v - x (fp32 [L_v][H]) that TeaCache stores. */
acid_status acid_dit_step(acid_model* m, const float* x_dev, float sigma,
                          const float* text_dev, float* v_dev,
                          float* resid_dev, hipStream_t stream);

/* TeaCache's signal (Section 2): m_cur = LN(x) (1 + scale1) + shift1 with
 * block 0's first modulation at sigma (the TEMNI), written to m_cur_dev fp32
 * [L_v][H]; then s = sum|m_cur - m_prev| / sum|m_prev| (fp64 final
 * reduction, fixed order: deterministic).  m_prev_dev NULL (first step)
 * gives s = NaN.  A zero denominator gives 0 if the numerator is 0, else
 * +inf.  Synchronises the stream; *s_out is a host double. */
acid_status acid_drift_signal(acid_model* m, const float* x_dev, float sigma,
                              const float* m_prev_dev, float* m_cur_dev,
                              double* s_out, hipStream_t stream);

/* One step of Algorithm 1 (pure host code, fp64, no fast-math): during the
 * first n_warmup steps returns compute = 1, tau = NaN and changes nothing but
 * the step counter.  Otherwise: sigma_sum += s_t; tau = tau_high if a previous
 * signal exists and |s_t - s_prev| <= delta, else tau_low; skip iff
 * sigma_sum <= tau, otherwise compute and reset sigma_sum to 0; s_prev = s_t.
 * A NaN signal always computes.  tau_used_out may be NULL. */
acid_status acid_gate(acid_gate_state* st, const acid_gate_params* p,
                      double s_t, int32_t* compute_out, double* tau_used_out);

/* Residual cache over n fp32 elements (see acid_cache_op).  STORE reads
 * x and h_out and writes r; APPLY reads x and r and writes h_out. */
acid_status acid_cache_apply(acid_cache_op op, const float* x_dev,
                             float* h_out_dev, float* r_dev, int64_t n,
                             hipStream_t stream);

/* DiCache probe depth for ACID_MODE_DICACHE: the first n_probe blocks
 * (0 <= n_probe <= n_blocks; default 1) run on every step.  Model state,
 * kept until changed. */
acid_status acid_model_set_probe_blocks(acid_model* m, int32_t n_probe);

/* L1 sums for EasyCache's signal, in one pass over n fp32 elements:
 * out_host[0] = sum |a - b| (sum |a| if b_dev is NULL), out_host[1] =
 * sum |c| (0 if c_dev is NULL).  fp64 accumulation in a fixed order
 * (deterministic).  Uses the model's workspace for partial sums, so n must
 * be at most n_video * hidden.  Synchronises the stream.  n == 0 gives
 * (0, 0) without touching the buffers (which may then be NULL). */
acid_status acid_l1_norms(acid_model* m, const float* a_dev, const float* b_dev,
                          const float* c_dev, int64_t n, double* out_host,
                          hipStream_t stream);

/* acid_l1_norms without a model and without any allocation, for callers
 * that cannot allocate device memory (tight serving loops, harnesses that
 * forbid hipMalloc) and hold no model workspace.
 * Same arguments, sums and kernels as acid_l1_norms (bit-identical results
 * whenever acid_l1_norms runs its full 1024-workgroup grid, i.e. for models
 * with n_video >= 1024); no model and no size bound: the partial sums go to
 * a 16 KB array (1024 fp64 pairs plus the result pair) that the library
 * keeps in device memory on each device it runs on until the process ends,
 * and the L1 grid never exceeds those 1024 workgroups.  The device is the
 * stream's (the current device for the null stream).  n < 0:
 * ACID_ERR_INVALID_ARG.  Calls that overlap on one device race on that
 * array (one at a time per device); each call writes every entry it reads,
 * so nothing carries over from an earlier call.  Synchronises the stream. */
acid_status acid_l1_norms_noalloc(const float* a_dev, const float* b_dev,
                                  const float* c_dev, int64_t n,
                                  double* out_host, hipStream_t stream);

/* EasyCache's skipped step over n fp32 elements: v = x + D; x_prev = x;
 * x = x + dsigma v (x updated in place; v_dev and x_prev_dev written;
 * offset_dev D read).  The four buffers must not overlap. */
acid_status acid_easycache_reuse(float* x_dev, float* x_prev_dev, float* v_dev,
                                 const float* offset_dev, int64_t n, float dsigma,
                                 hipStream_t stream);

/* The denoise loop of Algorithm 1 around f_theta, n_steps steps over noise
 * levels sigmas_host[0..n_steps] (host fp32).  x_dev fp32 [L_v][H]: x_0 in,
 * x_N out.  Per step i: (ACID mode) TEMNI + drift s_i, gate; compute -> all
 * blocks and r = h_out_v - x_i; skip -> h_out_v = x_i + r; then the head
 * and the Euler update x_{i+1} = x_i + (sigma_{i+1} - sigma_i) v_i.
 * gate may be NULL in NOCACHE mode.  forced_schedule_host (NULL or n_steps
 * bytes, 0/1) overrides the executed decision while the gate keeps its own
 * state; its step 0 must be 1.  trace_host (NULL or n_steps entries)
 * receives the per-step trace.  One stream synchronisation per ACID step.
 * EASYCACHE mode: per step i >= 1 the L1 sums |x_i - x_{i-1}|, |v_{i-1}| give
 * s_i (NaN until a rate k exists), then the gate; compute -> f_theta, x
 * update by the head's Euler epilogue, D = v_i - x_i and (i >= 1) the new
 * k; skip -> acid_easycache_reuse.  The TEMNI buffers of the workspace hold
 * x_{i-1} and v_{i-1}.  Two stream synchronisations per computed step. */
acid_status acid_denoise_loop(acid_model* m, float* x_dev,
                              const float* sigmas_host, int32_t n_steps,
                              const float* text_dev, int32_t mode,
                              const acid_gate_params* gate,
                              const uint8_t* forced_schedule_host,
                              acid_step_trace* trace_host, hipStream_t stream);

/* The same loop with the gate on the device and no host round trip between
 * steps (Section 3.3's gate and the loop of Algorithm 1; the gate's low cost
 * is the paper's claim, Section 3.2).  Every mode; arguments, results and
 * trace as acid_denoise_loop, to the bit.  Per step a one-thread kernel runs
 * the gate step on the signal the reductions left in device memory (the
 * TEMNI drift, DiCache's probe change, or EasyCache's k |dx| / |v_prev|,
 * with k kept on the device) and writes the decision into a device trace
 * and its negation into a skip word; every kernel that runs only on a
 * computed (or only on a skipped) step reads that word and exits at once
 * when it says so, and the cache kernel takes STORE or APPLY from it.  The modulation table is computed on `stream` first; the
 * per-step launches are captured once into a HIP graph (on a stream the
 * model owns) and replayed on `stream` by later calls with the same x_dev,
 * text_dev, n_steps, sigmas, mode, gate and forced schedule; any change
 * captures anew.  Without trace_host the call returns without waiting for
 * the GPU; with it, it synchronises `stream` once at the end.  The kernel
 * timer (acid_model_set_timing) does not see the graph's kernels. */
acid_status acid_denoise_loop_graph(acid_model* m, float* x_dev,
                                    const float* sigmas_host, int32_t n_steps,
                                    const float* text_dev, int32_t mode,
                                    const acid_gate_params* gate,
                                    const uint8_t* forced_schedule_host,
                                    acid_step_trace* trace_host,
                                    hipStream_t stream);
/* (The DiCache probe depth, acid_model_set_probe_blocks, is part of what a
 * captured graph is keyed on.) */

/* Algorithm 1 (Section 3.3) on the device, one thread, over n signals
 * s_dev[0..n) (fp64, device; NaN where a step has no signal) from the
 * initial state: trace_dev[i] (device, n entries) as acid_gate would fill
 * it step by step (compute == gate_compute).  The step is the same
 * IEEE-double code as acid_gate's.  Asynchronous on `stream`. */
acid_status acid_gate_device_sequence(const acid_gate_params* gate,
                                      const double* s_dev, int32_t n,
                                      acid_step_trace* trace_dev,
                                      hipStream_t stream);

/* -------------------------------------------- component calls (kernels) */

/* Timestep embedding and adaLN modulation table (one row per noise level):
 * table_dev fp32 [n][n_blocks*6 + 2][H]: for each sigma, the six per-block
 * vectors in manifest order, then the head's shift and scale. */
acid_status acid_timestep_modulation(acid_model* m, const float* sigmas_host,
                                     int32_t n, float* table_dev,
                                     hipStream_t stream);

/* out = LN(x) (1 + scale) + shift per row (LayerNorm without affine,
 * eps 1e-6, biased variance).  x fp32 [rows][hidden]; shift, scale fp32
 * [hidden]; out [rows][hidden] in out_dtype.  hidden % 4 == 0, <= 4096. */
acid_status acid_ln_modulate(int32_t out_dtype, const float* x_dev,
                             int64_t rows, int32_t hidden,
                             const float* shift_dev, const float* scale_dev,
                             void* out_dev, hipStream_t stream);

/* Full non-causal multi-head attention, O = softmax(Q K^T / sqrt(d)) V per
 * head.  q, k: [n_heads][L][d]; vt: V transposed, [n_heads][d][vt_ld] with
 * vt_ld >= round_up(L, 8) (entries past L are ignored); o: [L][n_heads*d]
 * (token-major).  All in `dtype`; softmax statistics in fp32.  d is 64 or
 * 128.  q_prescaled 0: q holds Q; 1: q holds Q multiplied by
 * log2(e)/sqrt(d) (the float value 1.4426950408889634f / sqrtf(d)) and
 * rounded to `dtype`, as the QKV epilogue writes it with q_prescale set
 * (the softmax then needs no per-score scaling); other values:
 * ACID_ERR_INVALID_ARG.  Size limits (ACID_ERR_SHAPE beyond them):
 * seq_len * n_heads < 2^26, and for bf16 head_dim * vt_ld * 2 < 2^31
 * (32-bit per-head offsets). */
acid_status acid_attention(int32_t dtype, int32_t n_heads, int64_t seq_len,
                           int32_t head_dim, const void* q_dev,
                           const void* k_dev, const void* vt_dev,
                           int64_t vt_ld, void* o_dev, int32_t q_prescaled,
                           hipStream_t stream);

/* The fp32 factor log2(e)/sqrt(head_dim) that a pre-scaled Q carries (see
 * acid_attention's q_prescaled and the QKV epilogues' q_prescale): a caller
 * that stores Q in that form multiplies by exactly this value before the one
 * rounding to the operand dtype.  0 for head_dim <= 0. */
float acid_q_scale(int32_t head_dim);

/* Epilogues of the fused GEMM y = a W + b (acc in fp32). */
typedef enum {
  ACID_EPI_BIAS = 0,          /* out fp32 [M][N] = y */
  ACID_EPI_BIAS_GELU = 1,     /* out dtype [M][N] = GELU_tanh(y) */
  ACID_EPI_GATE_RESIDUAL = 2, /* out fp32 [M][N] += gate (.) y  (in place) */
  ACID_EPI_QKV = 3,           /* y split into Q | K | V heads (see below) */
  ACID_EPI_EULER = 4,         /* out fp32 [M][N] += dsigma * y (in place);
                                 v_out (optional) fp32 [M][N] = y */
  ACID_EPI_QKV_GELU = 5       /* columns < 3 n_heads head_dim as QKV; column
                                 3 n_heads head_dim + j (j < N - 3 H) to
                                 out dtype [M][out_ld] at j: GELU_tanh(y) */
} acid_epilogue;

typedef struct {
  int32_t kind;         /* acid_epilogue */
  const float* bias;    /* [N], required */
  const float* gate;    /* [N], GATE_RESIDUAL only */
  const float* bias2;   /* [N], GATE_RESIDUAL: optional second bias (NULL: none) */
  void* out;            /* see acid_epilogue */
  int64_t out_ld;       /* QKV_GELU: row stride of out (elements) */
  float* v_out;         /* EULER only, may be NULL */
  void* q;              /* QKV: [n_heads][M][head_dim] */
  void* k;              /* QKV: [n_heads][M][head_dim] */
  void* vt;             /* QKV: [n_heads][head_dim][vt_ld], 16-byte aligned */
  int64_t vt_ld;        /* QKV: >= M, a multiple of 8 */
  int32_t n_heads;      /* QKV: N == 3 * n_heads * head_dim (QKV_GELU: >) */
  int32_t head_dim;     /* QKV */
  float dsigma;         /* EULER */
  int32_t q_prescale;   /* QKV kinds: 1 stores Q multiplied by log2(e)/sqrt(
                           head_dim) (see acid_attention's q_prescaled), 0
                           plain Q; K and V are never scaled */
} acid_epilogue_args;

/* Fused GEMM: a [M][K] and wt = W transposed [N][K], both in `dtype`;
 * N % 128 == 0, K % 128 == 0, N and K <= 2^22, 0 <= M <= 2^30 with
 * ceil(M / 256) * ceil(N / 256) < 2^23 (ACID_ERR_SHAPE otherwise). */
acid_status acid_linear(int32_t dtype, int64_t M, int32_t N, int32_t K,
                        const void* a_dev, const void* wt_dev,
                        const acid_epilogue_args* epi, hipStream_t stream);

/* One DiT block in place on the residual stream h_dev fp32 [L][H]
 * (L = n_text + n_video) with mod6_dev fp32 [6][H] (shift1, scale1, gate1,
 * shift2, scale2, gate2): LN-modulate, QKV, attention, gated projection,
 * LN-modulate, GELU MLP, gated second projection. */
acid_status acid_block_forward(acid_model* m, int32_t block,
                               const float* mod6_dev, float* h_dev,
                               hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* ACID_H */

"""Plain CPU oracle of the ACID-gated video-DiT denoise loop.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this module.  It shares no code
with the HIP library (no kernels, headers, helpers or constants) and never
imports it.

Everything here is written for a reader to check against the paper by eye:
float64 arithmetic throughout, NumPy matmuls as the only library primitive,
no blocking or fusion beyond chunking attention over query rows to bound
memory (which changes no value beyond rounding order).

What is computed, and where it comes from
-----------------------------------------
* The gate (``AcidGate``) is Algorithm 1 ("Adaptive Threshold Caching") of
  Section 3.3, step by step.  Fixed-threshold caching (Section 2, paragraph on
  the fixed threshold of dynamic caching methods) is the special case
  tau_low == tau_high.
* The drift signal is TeaCache's: the L1 change between consecutive
  timestep-embedding-modulated noisy inputs (TEMNI), Section 2, paragraph
  "TeaCache".  It is taken relative to the previous step's L1 norm.
* Skipped steps reuse the previous output corrected by a stored residual
  (same paragraph): on a computed step r = h_out - x, on a skipped step
  h_out = x + r.
* DiCache's probe signal under the same gate (``dicache_loop``): Section 2,
  paragraph "DiCache" (shallow probe of the first blocks every step, relative
  change of its features, deep-output reuse on skipped steps) and Section
  3.3; the reuse adds the stored deep residual to the probe output.
* EasyCache's signal under the same gate (``easycache_loop``): Section 2,
  paragraph "EasyCache" (transformation rate k, signal k |dx| / |v_prev|,
  reuse v = x + D) and Section 3.3 (the gated variable); L1 norms.
* The backbone f_theta (Algorithm 1 treats it as a black box) is an adaLN
  DiT: sinusoidal timestep embedding -> MLP -> per-block shift/scale/gate
  modulation, LayerNorm without affine parameters, full non-causal multi-head
  self-attention over all tokens, a tanh-GELU MLP, and a modulated
  LayerNorm + linear head.  The reverse process (Section 3.1, eq. (2)) is
  realised as a flow-matching Euler step x_{i+1} = x_i + (s_{i+1} - s_i) v_i.
* The parallel block (``parallel_block``) is HunyuanVideo's single-stream
  block (HunyuanVideo is the first model of Section 4.1): attention and MLP
  branches from one modulated LayerNorm, projected together, one gated
  residual.  Pinned by reduction to the sequential block: equal to it when
  the MLP weights are zero, equal to it when the attention weights are zero
  and the second modulation triple equals the first, and its two branches
  add.

Pins
----
Every function below is pinned by a ``-m "not gpu"`` test against something
other than itself (library routines, closed forms, brute force, invariants,
hand-derived dyadic traces).  The composed DiT block and stack are checked
through their components, token-permutation equivariance, the zero-gate
identity and a torch.nn.functional composition; beyond that the full stack's
values are "parity unpinned": no external numbers exist for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

F64 = np.float64

# --------------------------------------------------------------------------
# Precision helpers
# --------------------------------------------------------------------------


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns float32 values that are exactly representable in bfloat16.  Used
    when the oracle serves as the reference of a bfloat16 run: the GEMM
    weights are rounded once, as the bfloat16 path stores them.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    nan = np.isnan(a)
    out = r.view(np.float32).copy()
    out[nan] = np.float32("nan")
    return out


# --------------------------------------------------------------------------
# Elementary functions of the backbone
# --------------------------------------------------------------------------


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    """GELU, tanh form: 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))


def layer_norm(x: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """Per-row LayerNorm without affine parameters, biased variance."""
    x = np.asarray(x, dtype=F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def modulate(xn: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """adaLN modulation of an already normalised input: xn (1 + scale) + shift."""
    return xn * (1.0 + scale) + shift


def timestep_embedding(sigma: float, dim: int = 256, max_period: float = 10000.0) -> np.ndarray:
    """Sinusoidal embedding of t = 1000 sigma: [cos(t f_j)]_j ++ [sin(t f_j)]_j.

    f_j = exp(-ln(max_period) j / (dim/2)) for j < dim/2.
    """
    half = dim // 2
    t = 1000.0 * float(sigma)
    freqs = np.exp(-math.log(max_period) * np.arange(half, dtype=F64) / half)
    args = t * freqs
    return np.concatenate([np.cos(args), np.sin(args)])


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, chunk: int = 512) -> np.ndarray:
    """Single-head attention softmax(q k^T / sqrt(d)) v, non-causal.

    q: [Lq, d], k and v: [Lk, d].  Query rows are processed in chunks so that
    memory stays O(chunk * Lk); each chunk is the plain definition.
    """
    q = np.asarray(q, dtype=F64)
    k = np.asarray(k, dtype=F64)
    v = np.asarray(v, dtype=F64)
    d = q.shape[-1]
    out = np.empty((q.shape[0], v.shape[1]), dtype=F64)
    for s0 in range(0, q.shape[0], chunk):
        s = (q[s0:s0 + chunk] @ k.T) / math.sqrt(d)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[s0:s0 + chunk] = p @ v
    return out


def multi_head_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Token-major q [Lq, H], k/v [Lk, H]; head j uses columns j d .. (j+1) d."""
    H = q.shape[1]
    d = H // n_heads
    out = np.empty((q.shape[0], H), dtype=F64)
    for j in range(n_heads):
        c = slice(j * d, (j + 1) * d)
        out[:, c] = attention(q[:, c], k[:, c], v[:, c])
    return out


# --------------------------------------------------------------------------
# The backbone f_theta
# --------------------------------------------------------------------------

GEMM_WEIGHTS = ("qkv.w", "o.w", "ffn1.w", "ffn2.w")


class DiTModel:
    """adaLN DiT stack built from a manifest-ordered parameter dict.

    ``dtype == "bf16"`` rounds the GEMM weights (qkv, o, ffn1, ffn2, head) to
    bfloat16 once, as the bfloat16 path stores them; timestep-MLP and adaLN
    weights and all biases stay float32.  All arithmetic is float64.
    Block weights are converted lazily so very large stacks can be sampled
    block by block.
    """

    def __init__(self, cfg, params: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.p = params
        self._mod_cache: Dict[float, dict] = {}

    def w(self, name: str) -> np.ndarray:
        a = self.p[name]
        base = name.split(".", 2)[-1] if name.startswith("blocks.") else name
        if self.cfg.dtype == "bf16" and (base in GEMM_WEIGHTS or name == "head.w"):
            a = bf16_round(a)
        return np.asarray(a, dtype=F64)

    # -- timestep conditioning and adaLN modulation ------------------------
    def modulation(self, sigma: float) -> dict:
        """Per-block (shift1, scale1, gate1, shift2, scale2, gate2) and head
        (shift, scale) for noise level sigma."""
        key = float(sigma)
        if key in self._mod_cache:
            return self._mod_cache[key]
        cfg, H = self.cfg, self.cfg.hidden
        e = timestep_embedding(sigma, cfg.freq_dim)
        hid = silu(e @ self.w("temb.w1") + self.w("temb.b1"))
        c = hid @ self.w("temb.w2") + self.w("temb.b2")
        u = silu(c)
        blocks = []
        for b in range(cfg.n_blocks):
            m = u @ self.w(f"blocks.{b}.ada.w") + self.w(f"blocks.{b}.ada.b")
            blocks.append(m.reshape(6, H))
        hm = (u @ self.w("head.ada.w") + self.w("head.ada.b")).reshape(2, H)
        out = {"c": c, "blocks": blocks, "head": hm}
        self._mod_cache[key] = out
        return out

    # -- one DiT block ------------------------------------------------------
    def block(self, h: np.ndarray, b: int, mod6: np.ndarray,
              rows: Optional[np.ndarray] = None) -> np.ndarray:
        """One block on the residual stream h [L, H] (text rows first).

        Returns the block output for ``rows`` (all rows if None).  Keys and
        values always span all L tokens.
        """
        if getattr(self.cfg, "block", "sequential") == "parallel":
            return self.parallel_block(h, b, mod6, rows)
        cfg = self.cfg
        H = cfg.hidden
        shift1, scale1, gate1, shift2, scale2, gate2 = mod6
        h = np.asarray(h, dtype=F64)
        pre = f"blocks.{b}."
        a = modulate(layer_norm(h), shift1, scale1)
        wqkv, bqkv = self.w(pre + "qkv.w"), self.w(pre + "qkv.b")
        kv = a @ wqkv[:, H:] + bqkv[H:]
        k, v = kv[:, :H], kv[:, H:]
        if rows is None:
            rows = np.arange(h.shape[0])
        q = a[rows] @ wqkv[:, :H] + bqkv[:H]
        o = multi_head_attention(q, k, v, cfg.n_heads)
        hr = h[rows] + gate1 * (o @ self.w(pre + "o.w") + self.w(pre + "o.b"))
        a2 = modulate(layer_norm(hr), shift2, scale2)
        f = gelu_tanh(a2 @ self.w(pre + "ffn1.w") + self.w(pre + "ffn1.b"))
        return hr + gate2 * (f @ self.w(pre + "ffn2.w") + self.w(pre + "ffn2.b"))

    def parallel_block(self, h: np.ndarray, b: int, mod6: np.ndarray,
                       rows: Optional[np.ndarray] = None) -> np.ndarray:
        """HunyuanVideo's single-stream block (the model Section 4.1
        evaluates), in parallel form: one modulated LayerNorm a feeds both
        the attention branch and the MLP branch, whose outputs are projected
        together and added to the residual stream through one gate:

            a = LN(h) (1 + scale1) + shift1
            o = attention(a W_q + b_q, a W_k + b_k, a W_v + b_v)
            out = h + gate1 (o W_o + b_o + gelu_tanh(a W_1 + b_1) W_2 + b_2)

        i.e. linear1 = [W_qkv | W_1] (H -> 3H + F) and linear2 = [W_o ; W_2]
        (H + F -> H) of that design, from the same tensors as the sequential
        block; the second modulation triple is unused.
        """
        cfg = self.cfg
        H = cfg.hidden
        shift1, scale1, gate1 = mod6[0], mod6[1], mod6[2]
        h = np.asarray(h, dtype=F64)
        pre = f"blocks.{b}."
        a = modulate(layer_norm(h), shift1, scale1)
        wqkv, bqkv = self.w(pre + "qkv.w"), self.w(pre + "qkv.b")
        kv = a @ wqkv[:, H:] + bqkv[H:]
        k, v = kv[:, :H], kv[:, H:]
        if rows is None:
            rows = np.arange(h.shape[0])
        ar = a[rows]
        q = ar @ wqkv[:, :H] + bqkv[:H]
        o = multi_head_attention(q, k, v, cfg.n_heads)
        f = gelu_tanh(ar @ self.w(pre + "ffn1.w") + self.w(pre + "ffn1.b"))
        y = (o @ self.w(pre + "o.w") + self.w(pre + "o.b")
             + f @ self.w(pre + "ffn2.w") + self.w(pre + "ffn2.b"))
        return h[rows] + gate1 * y

    def stack(self, x: np.ndarray, sigma: float, text: Optional[np.ndarray] = None) -> np.ndarray:
        """All blocks on h_in = [text; x]; returns the video rows h_out_v."""
        mod = self.modulation(sigma)
        h = np.asarray(x, dtype=F64)
        n_text = 0 if text is None else len(text)
        if n_text:
            h = np.concatenate([np.asarray(text, dtype=F64), h], axis=0)
        for b in range(self.cfg.n_blocks):
            h = self.block(h, b, mod["blocks"][b])
        return h[n_text:]

    def head(self, h_out_v: np.ndarray, sigma: float) -> np.ndarray:
        """v = (LN(h_out_v) (1 + scale_h) + shift_h) W_out + b_out."""
        shift, scale = self.modulation(sigma)["head"]
        a = modulate(layer_norm(h_out_v), shift, scale)
        return a @ self.w("head.w") + self.w("head.b")

    def forward(self, x: np.ndarray, sigma: float, text: Optional[np.ndarray] = None):
        """f_theta(x, t, c): returns (v, h_out_v)."""
        h_out_v = self.stack(x, sigma, text)
        return self.head(h_out_v, sigma), h_out_v

    # -- TeaCache's signal input -------------------------------------------
    def temni(self, x: np.ndarray, sigma: float) -> np.ndarray:
        """Timestep-embedding-modulated noisy input: block 0's first
        modulation applied to LN(x) over the video rows."""
        shift1, scale1 = self.modulation(sigma)["blocks"][0][:2]
        return modulate(layer_norm(x), shift1, scale1)


# --------------------------------------------------------------------------
# Drift signal and the ACID gate
# --------------------------------------------------------------------------


def relative_l1_drift(m_cur: np.ndarray, m_prev: np.ndarray) -> float:
    """s = sum|m_cur - m_prev| / sum|m_prev|, sums in float64.

    A zero denominator gives 0 when the numerator is 0 and +inf otherwise.
    """
    num = float(np.abs(np.asarray(m_cur, F64) - np.asarray(m_prev, F64)).sum())
    den = float(np.abs(np.asarray(m_prev, F64)).sum())
    if den == 0.0:
        return 0.0 if num == 0.0 else math.inf
    return num / den


@dataclasses.dataclass
class GateParams:
    """Algorithm 1's parameters: tau_low, tau_high and the stability bound
    delta; n_warmup leading steps always run the model."""
    tau_low: float
    tau_high: float
    delta: float
    n_warmup: int = 1


class AcidGate:
    """Algorithm 1 of Section 3.3 as a step function over the drift sequence.

    State: accumulated drift (starts at 0) and the previous signal (starts at
    None).  Each call consumes one step's signal and returns whether the
    model is run and which threshold was used (NaN during warmup).
    """

    def __init__(self, p: GateParams):
        self.p = p
        self.sigma_sum = 0.0
        self.s_prev: Optional[float] = None
        self.step = 0

    def __call__(self, s_t: float):
        p = self.p
        i = self.step
        self.step += 1
        if i < p.n_warmup:
            # The base method's leading steps always run the model; the gate
            # state is left as it was.
            return True, math.nan
        self.sigma_sum = self.sigma_sum + s_t
        # A signal that moved by at most delta since the previous step
        # selects the larger threshold (more skipping); any larger move, or
        # no previous signal, selects the smaller one.
        moved_little = self.s_prev is not None and abs(s_t - self.s_prev) <= p.delta
        tau = p.tau_high if moved_little else p.tau_low
        # Skip while the accumulated drift has not passed the threshold; a
        # computed step starts the accumulation afresh.  (A NaN sum fails the
        # comparison and so computes.)
        compute = not (self.sigma_sum <= tau)
        if compute:
            self.sigma_sum = 0.0
        self.s_prev = s_t
        return compute, tau


def gate_schedule(s_seq: Sequence[float], p: GateParams):
    """Run the gate over a whole drift sequence (s_seq[i] used at step i;
    entries of warmup steps are ignored).  Returns (decisions, taus, sums)."""
    g = AcidGate(p)
    dec, taus, sums = [], [], []
    for s in s_seq:
        c, t = g(float(s))
        dec.append(bool(c))
        taus.append(t)
        sums.append(g.sigma_sum)
    return dec, taus, sums


# --------------------------------------------------------------------------
# The denoise loop
# --------------------------------------------------------------------------

TRACE_DTYPE = np.dtype([("compute", np.int32), ("gate_compute", np.int32),
                        ("s", np.float64), ("sigma_sum_after", np.float64),
                        ("tau_used", np.float64)])


def l1_norm(a: np.ndarray) -> float:
    """sum |a| in float64."""
    return float(np.abs(np.asarray(a, F64)).sum())


def ratio_or_inf(num: float, den: float) -> float:
    """num / den with 0/0 = 0 and num/0 = +inf (num >= 0)."""
    if den == 0.0:
        return 0.0 if num == 0.0 else math.inf
    return num / den


def easycache_loop(forward: Callable, x0: np.ndarray, sigmas: np.ndarray,
                   gate: Optional[GateParams] = None, mode: str = "easycache",
                   forced_schedule: Optional[Sequence[int]] = None):
    """EasyCache's signal under the gate of Algorithm 1 (Section 2, paragraph
    "EasyCache"; Section 3.3 for the gated variable).

    forward(x, sigma) -> v runs the whole model.  On a computed step i >= 1
    the transformation rate is k = |v_i - v_{i-1}|_1 / |x_i - x_{i-1}|_1 (output
    change over input change at that step) and the offset D = v_i - x_i is
    stored.  At step i the signal is s_i = k |x_i - x_{i-1}|_1 / |v_{i-1}|_1
    with k from the last computed step; a skipped step outputs v_i = x_i + D.
    The first n_warmup >= 2 steps run the model (k needs two).  Norms are L1.
    mode "nocache" runs the model on every step.  Returns (x_N, trace).
    """
    n = len(sigmas) - 1
    if mode == "easycache" and (gate is None or gate.n_warmup < 2):
        raise ValueError("EasyCache needs n_warmup >= 2")
    g = AcidGate(gate) if mode == "easycache" else None
    x = np.asarray(x0, dtype=F64)
    x_prev = v_prev = offset = None
    k = None
    trace = np.zeros(n, dtype=TRACE_DTYPE)
    for i in range(n):
        sig = float(sigmas[i])
        s = math.nan
        if mode == "nocache":
            gate_compute, tau = True, math.nan
        else:
            if k is not None:
                s = k * ratio_or_inf(l1_norm(x - x_prev), l1_norm(v_prev))
            gate_compute, tau = g(s)
        compute = gate_compute if forced_schedule is None else bool(forced_schedule[i])
        if compute:
            v = np.asarray(forward(x, sig), dtype=F64)
            if v_prev is not None:
                k = ratio_or_inf(l1_norm(v - v_prev), l1_norm(x - x_prev))
            offset = v - x
        else:
            if offset is None:
                raise ValueError("skip requested before any computed step")
            v = x + offset
        x_prev, v_prev = x, v
        x = x + (float(sigmas[i + 1]) - sig) * v
        trace[i] = (int(compute), int(gate_compute), s,
                    g.sigma_sum if g is not None else 0.0, tau)
    return x, trace


def dicache_loop(model, x0: np.ndarray, sigmas: np.ndarray, text=None,
                 gate: Optional[GateParams] = None, n_probe: int = 1,
                 forced_schedule: Optional[Sequence[int]] = None):
    """DiCache's probe signal under the gate of Algorithm 1 (Section 2,
    paragraph "DiCache"; Section 3.3 names the probe-feature change as the
    gated variable).

    Every step runs the first n_probe blocks (the shallow probe) on
    [text; x_i]; the signal is the relative L1 change of the probe's video
    rows p_i against p_{i-1}.  A computed step runs the remaining blocks and
    stores the deep residual R = h_out_v - p_i; a skipped step uses
    h_out_v = p_i + R.  Head and Euler update on every step.  Returns
    (x_N, trace).
    """
    cfg = model.cfg
    if not 0 <= n_probe <= cfg.n_blocks:
        raise ValueError("n_probe must be in [0, n_blocks]")
    n = len(sigmas) - 1
    g = AcidGate(gate)
    x = np.asarray(x0, dtype=F64)
    n_text = 0 if text is None else len(text)
    p_prev = r_deep = None
    trace = np.zeros(n, dtype=TRACE_DTYPE)
    for i in range(n):
        sig = float(sigmas[i])
        mod = model.modulation(sig)
        h = x if n_text == 0 else np.concatenate([np.asarray(text, F64), x], axis=0)
        for b in range(n_probe):
            h = model.block(h, b, mod["blocks"][b])
        p = h[n_text:]
        s = relative_l1_drift(p, p_prev) if p_prev is not None else math.nan
        p_prev = p
        gate_compute, tau = g(s)
        compute = gate_compute if forced_schedule is None else bool(forced_schedule[i])
        if compute:
            for b in range(n_probe, cfg.n_blocks):
                h = model.block(h, b, mod["blocks"][b])
            h_out_v = h[n_text:]
            r_deep = h_out_v - p
        else:
            if r_deep is None:
                raise ValueError("skip requested before any computed step")
            h_out_v = p + r_deep
        v = model.head(h_out_v, sig)
        x = x + (float(sigmas[i + 1]) - sig) * v
        trace[i] = (int(compute), int(gate_compute), s, g.sigma_sum, tau)
    return x, trace


def denoise_loop(model, x0: np.ndarray, sigmas: np.ndarray, text=None,
                 mode: str = "acid", gate: Optional[GateParams] = None,
                 forced_schedule: Optional[Sequence[int]] = None):
    """The sampler of Algorithm 1 around f_theta, TeaCache-style.

    model provides temni(x, sigma), stack(x, sigma, text) -> h_out_v and
    head(h_out_v, sigma) -> v.  mode is "nocache" (run f_theta every step, no
    signal) or "acid" (fixed threshold = tau_low == tau_high).  A forced
    schedule overrides the executed decision; the gate still runs on its own
    state and its decision is recorded as gate_compute.

    Returns (x_N, trace).
    """
    n = len(sigmas) - 1
    x = np.asarray(x0, dtype=F64)
    g = AcidGate(gate) if mode == "acid" else None
    trace = np.zeros(n, dtype=TRACE_DTYPE)
    m_prev = None
    r = None
    for i in range(n):
        sig = float(sigmas[i])
        s = math.nan
        if mode == "nocache":
            gate_compute, tau = True, math.nan
        else:
            # TEMNI is formed on every step, warmup and skipped ones included.
            m = model.temni(x, sig)
            if m_prev is not None:
                s = relative_l1_drift(m, m_prev)
            m_prev = m
            gate_compute, tau = g(s)
        compute = gate_compute if forced_schedule is None else bool(forced_schedule[i])
        if compute:
            h_out_v = model.stack(x, sig, text)
            if mode != "nocache":
                r = h_out_v - x              # store the residual
        else:
            if r is None:
                raise ValueError("skip requested before any computed step")
            h_out_v = x + r                  # reuse with the stored residual
        v = model.head(h_out_v, sig)
        x = x + (float(sigmas[i + 1]) - sig) * v
        trace[i] = (int(compute), int(gate_compute), s,
                    g.sigma_sum if g is not None else 0.0, tau)
    return x, trace


def psnr(x: np.ndarray, ref: np.ndarray) -> float:
    """PSNR of x against ref with peak = max(ref) - min(ref) (on latents)."""
    x = np.asarray(x, F64)
    ref = np.asarray(ref, F64)
    mse = float(((x - ref) ** 2).mean())
    rng = float(ref.max() - ref.min())
    if mse == 0.0:
        return math.inf
    return 10.0 * math.log10(rng * rng / mse)

"""Pins of the CPU oracle against things other than itself (no GPU needed).

Each test ties one oracle function to a library routine, a closed form, a
brute-force loop, an invariant or a hand-derived trace, chosen so that a
plausible slip (dropped term, wrong sign or index, transposed operand) fails.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

import acid_inputs as ai
import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ gate


def _load_dyadic():
    rows = []
    with open(os.path.join(GOLDEN, "gate_dyadic_trace.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            st, s, sig_add, tau, dec, sig_after = line.split()
            rows.append((int(st), float(s), float(sig_add), float(tau), dec, float(sig_after)))
    return rows


def test_gate_dyadic_trace():
    """Algorithm 1 on the hand-derived dyadic trace: every value exact."""
    rows = _load_dyadic()
    g = O.AcidGate(O.GateParams(0.0625, 0.25, 0.015625, n_warmup=1))
    for st, s, _sig_add, tau, dec, sig_after in rows:
        c, t = g(s)
        assert c == (dec == "C"), st
        if math.isnan(tau):
            assert math.isnan(t)
        else:
            assert t == tau, st
        assert g.sigma_sum == sig_after, st
    # ties: step 6 sits exactly on tau (skip), step 4 exactly on delta (stable)
    assert sum(1 for r in rows if r[4] == "C") == 4


def _fixed_skeleton(s_seq, tau, n_warmup=1):
    """Single-threshold caching as Section 2 describes it in prose: a running
    drift starts at zero, each step's estimate is added, a sum below tau
    skips, one that exceeds it runs the model and resets."""
    acc, out = 0.0, []
    for i, s in enumerate(s_seq):
        if i < n_warmup:
            out.append(True)
            continue
        acc += s
        if acc > tau:
            out.append(True)
            acc = 0.0
        else:
            out.append(False)
    return out


def test_gate_fixed_threshold_examples():
    s = [r[1] for r in _load_dyadic()]
    for tau, want in ((0.0625, "CSSCCCCCSC"), (0.25, "CSSSSCSSSC")):
        dec, _, _ = O.gate_schedule(s, O.GateParams(tau, tau, 0.015625))
        assert "".join("C" if d else "S" for d in dec) == want
        assert dec == _fixed_skeleton(s, tau)


def _rand_seq(seed, n=50):
    rng = np.random.default_rng(seed)
    # mixture of stable stretches and jumps, non-negative
    base = np.abs(rng.normal(0.03, 0.02, n))
    jumps = rng.random(n) < 0.2
    base[jumps] *= rng.uniform(2, 6, jumps.sum())
    return [float(np.float32(v)) for v in base]


@pytest.mark.parametrize("seed", range(20))
def test_gate_special_cases(seed):
    s = _rand_seq(seed)
    n = len(s)
    # tau = 0: every step with s > 0 computes
    dec, _, _ = O.gate_schedule(s, O.GateParams(0.0, 0.0, 0.01))
    assert all(dec[i] for i in range(n) if i == 0 or s[i] > 0)
    # tau = inf: only the warmup step computes
    dec, _, _ = O.gate_schedule(s, O.GateParams(math.inf, math.inf, 0.01))
    assert dec == [True] + [False] * (n - 1)
    # tau_low == tau_high: the fixed single-threshold skeleton
    for tau in (0.05, 0.1, 0.2):
        dec, _, _ = O.gate_schedule(s, O.GateParams(tau, tau, 0.01))
        assert dec == _fixed_skeleton(s, tau)
    # delta < 0: never stable -> fixed tau_low
    dec, taus, _ = O.gate_schedule(s, O.GateParams(0.05, 0.2, -1.0))
    assert dec == _fixed_skeleton(s, 0.05)
    assert all(t == 0.05 for t in taus[1:])
    # delta = inf: tau_low at the first non-warmup step, tau_high afterwards
    _, taus, _ = O.gate_schedule(s, O.GateParams(0.05, 0.2, math.inf))
    assert taus[1] == 0.05 and all(t == 0.2 for t in taus[2:])


@pytest.mark.parametrize("seed", range(200))
def test_gate_open_loop_sandwich(seed):
    """With tau_low <= tau_t <= tau_high per step, reset times under the larger
    threshold are never earlier, so computed-step counts are ordered."""
    s = _rand_seq(1000 + seed, n=60)
    rng = np.random.default_rng(seed)
    lo = float(rng.uniform(0.01, 0.1))
    hi = lo + float(rng.uniform(0.0, 0.3))
    delta = float(rng.uniform(0.0, 0.05))
    n_acid = sum(O.gate_schedule(s, O.GateParams(lo, hi, delta))[0])
    n_lo = sum(_fixed_skeleton(s, lo))
    n_hi = sum(_fixed_skeleton(s, hi))
    assert n_hi <= n_acid <= n_lo


def test_gate_nan_and_inf_signal():
    g = O.AcidGate(O.GateParams(0.05, 0.2, 0.01))
    assert g(123.0)[0]                 # warmup ignores the signal
    c, t = g(math.nan)                 # NaN never satisfies <=: compute, tau_low
    assert c and t == 0.05 and g.sigma_sum == 0.0
    c, t = g(0.01)                     # |0.01 - NaN| <= delta is false
    assert not c and t == 0.05
    c, _ = g(math.inf)
    assert c and g.sigma_sum == 0.0


# ------------------------------------------------------------------ drift


def test_drift_closed_form():
    m_prev = np.array([1.0, -2.0, 3.0, -4.0])
    m_cur = np.array([1.5, -2.0, 2.0, -4.0])
    assert O.relative_l1_drift(m_cur, m_prev) == pytest.approx(0.15, abs=0, rel=1e-15)


def test_drift_properties():
    rng = np.random.default_rng(0)
    a, b = rng.normal(size=(7, 5)), rng.normal(size=(7, 5))
    assert O.relative_l1_drift(a, a) == 0.0
    assert O.relative_l1_drift(3.5 * a, 3.5 * b) == pytest.approx(O.relative_l1_drift(a, b), rel=1e-14)
    assert O.relative_l1_drift(np.zeros_like(a), a) == pytest.approx(1.0, rel=1e-15)
    assert O.relative_l1_drift(np.zeros(3), np.zeros(3)) == 0.0
    assert O.relative_l1_drift(np.ones(3), np.zeros(3)) == math.inf
    # not symmetric: the denominator is the previous step's norm
    assert O.relative_l1_drift(2 * a, a) == pytest.approx(1.0, rel=1e-14)
    assert O.relative_l1_drift(a, 2 * a) == pytest.approx(0.5, rel=1e-14)


# ------------------------------------------------------------ elementary


def test_layer_norm_vs_torch():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(9, 64)) * 3 + 1
    ref = Fnn.layer_norm(torch.from_numpy(x), (64,), eps=1e-6).numpy()
    np.testing.assert_allclose(O.layer_norm(x), ref, rtol=1e-12, atol=1e-12)
    y = O.layer_norm(x)
    np.testing.assert_allclose(y.mean(1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(1), 1, rtol=1e-5)
    assert np.all(O.layer_norm(np.full((2, 8), 5.0)) == 0)


def test_gelu_silu_vs_torch():
    z = np.linspace(-8, 8, 1001)
    t = torch.from_numpy(z)
    np.testing.assert_allclose(O.gelu_tanh(z), Fnn.gelu(t, approximate="tanh").numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(O.silu(z), Fnn.silu(t).numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(O.gelu_tanh(z) - O.gelu_tanh(-z), z, atol=1e-13)
    assert O.gelu_tanh(np.array(0.0)) == 0.0


def test_timestep_embedding_pins():
    e0 = O.timestep_embedding(0.0, 256)
    assert np.all(e0[:128] == 1.0) and np.all(e0[128:] == 0.0)
    e = O.timestep_embedding(0.37, 256)
    t = 370.0
    # f_0 = 1 and f_64 = 10000^(-1/2) = 0.01 exactly
    assert e[0] == pytest.approx(math.cos(t), abs=1e-12)
    assert e[128] == pytest.approx(math.sin(t), abs=1e-12)
    assert e[64] == pytest.approx(math.cos(0.01 * t), abs=1e-12)
    assert e[192] == pytest.approx(math.sin(0.01 * t), abs=1e-12)
    np.testing.assert_allclose(e[:128] ** 2 + e[128:] ** 2, 1.0, atol=1e-12)


def test_bf16_round_vs_torch():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.normal(size=10000).astype(np.float32) * 10,
                        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -9, -(1 + 2 ** -8), 0.0, -0.0,
                                  np.inf, -np.inf, 3.4e38], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = O.bf16_round(x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    assert np.isnan(O.bf16_round(np.array([np.nan], np.float32))[0])


# -------------------------------------------------------------- attention


def _attention_brute(q, k, v):
    Lq, d = q.shape
    out = np.zeros((Lq, v.shape[1]))
    for i in range(Lq):
        sc = [sum(q[i, c] * k[j, c] for c in range(d)) / math.sqrt(d) for j in range(k.shape[0])]
        mx = max(sc)
        w = [math.exp(x - mx) for x in sc]
        z = sum(w)
        for j in range(k.shape[0]):
            for c in range(v.shape[1]):
                out[i, c] += w[j] / z * v[j, c]
    return out


@pytest.mark.parametrize("L,d", [(1, 4), (3, 2), (8, 5)])
def test_attention_brute_force(L, d):
    rng = np.random.default_rng(L * 10 + d)
    q, k, v = (rng.normal(size=(L, d)) * 2 for _ in range(3))
    np.testing.assert_allclose(O.attention(q, k, v), _attention_brute(q, k, v), rtol=1e-12, atol=1e-12)


def test_attention_invariants():
    rng = np.random.default_rng(5)
    L, d = 37, 16
    q, k, v = (rng.normal(size=(L, d)) * 3 for _ in range(3))
    ref = Fnn.scaled_dot_product_attention(*(torch.from_numpy(t)[None, None] for t in (q, k, v)))[0, 0].numpy()
    np.testing.assert_allclose(O.attention(q, k, v), ref, rtol=1e-11, atol=1e-12)
    # chunking over query rows changes nothing
    np.testing.assert_allclose(O.attention(q, k, v, chunk=1), O.attention(q, k, v), rtol=1e-14, atol=1e-14)
    # V = identity exposes P: rows are non-negative and sum to one
    P = O.attention(q, k[:d], np.eye(d))
    assert np.all(P >= 0)
    np.testing.assert_allclose(P.sum(1), 1.0, rtol=1e-14)
    # Q = 0: uniform weights -> column mean of V
    np.testing.assert_allclose(O.attention(np.zeros_like(q), k, v), np.tile(v.mean(0), (L, 1)), rtol=1e-12, atol=1e-13)
    # a single key returns its value
    np.testing.assert_allclose(O.attention(q, k[:1], v[:1]), np.tile(v[0], (L, 1)), rtol=1e-14)
    # permuting keys and values jointly leaves the output unchanged
    perm = rng.permutation(L)
    np.testing.assert_allclose(O.attention(q, k[perm], v[perm]), O.attention(q, k, v), rtol=1e-12, atol=1e-13)


def test_multi_head_split():
    rng = np.random.default_rng(6)
    L, nh, d = 10, 3, 4
    q, k, v = (rng.normal(size=(L, nh * d)) for _ in range(3))
    tq = torch.from_numpy(q).view(L, nh, d).transpose(0, 1)
    tk = torch.from_numpy(k).view(L, nh, d).transpose(0, 1)
    tv = torch.from_numpy(v).view(L, nh, d).transpose(0, 1)
    ref = Fnn.scaled_dot_product_attention(tq, tk, tv).transpose(0, 1).reshape(L, nh * d).numpy()
    np.testing.assert_allclose(O.multi_head_attention(q, k, v, nh), ref, rtol=1e-11, atol=1e-12)


# ------------------------------------------------------------- DiT pieces

TOY = ai.DiTConfig("toy", n_blocks=2, hidden=32, n_heads=4, head_dim=8, ffn=64,
                   n_video=12, n_text=3, freq_dim=16, dtype="f32", n_steps=6)


def _toy_model(cfg=TOY, std=0.2):
    return O.DiTModel(cfg, ai.weights(cfg, std=std))


def test_modulation_split_order():
    cfg = TOY
    p = ai.weights(cfg)
    H = cfg.hidden
    p["blocks.1.ada.w"] = np.zeros_like(p["blocks.1.ada.w"])
    p["blocks.1.ada.b"] = np.arange(6 * H, dtype=np.float32)
    p["temb.w1"] = np.zeros_like(p["temb.w1"])
    m = O.DiTModel(cfg, p).modulation(0.4)
    for j in range(6):
        np.testing.assert_array_equal(m["blocks"][1][j], np.arange(j * H, (j + 1) * H))
    # with w1 = 0 the hidden layer is silu(b1) whatever sigma is
    b1 = p["temb.b1"].astype(np.float64)
    c = (b1 / (1 + np.exp(-b1))) @ p["temb.w2"].astype(np.float64) + p["temb.b2"]
    np.testing.assert_allclose(m["c"], c, rtol=1e-12)


def test_block_zero_gate_is_identity():
    cfg = TOY
    p = ai.weights(cfg, std=0.2)
    H = cfg.hidden
    for b in range(cfg.n_blocks):
        p[f"blocks.{b}.ada.w"][:, 2 * H:3 * H] = 0
        p[f"blocks.{b}.ada.b"][2 * H:3 * H] = 0
        p[f"blocks.{b}.ada.w"][:, 5 * H:] = 0
        p[f"blocks.{b}.ada.b"][5 * H:] = 0
    m = O.DiTModel(cfg, p)
    x = ai.gaussian((cfg.n_video, H), 7)
    np.testing.assert_array_equal(m.stack(x, 0.5), x.astype(np.float64))


def test_block_permutation_equivariance_and_rows():
    m = _toy_model()
    cfg = TOY
    rng = np.random.default_rng(8)
    h = rng.normal(size=(cfg.n_tokens, cfg.hidden))
    mod = m.modulation(0.3)["blocks"][0]
    out = m.block(h, 0, mod)
    perm = rng.permutation(cfg.n_tokens)
    np.testing.assert_allclose(m.block(h[perm], 0, mod), out[perm], rtol=1e-11, atol=1e-12)
    rows = np.array([0, 5, 11, 14])
    np.testing.assert_allclose(m.block(h, 0, mod, rows=rows), out[rows], rtol=1e-13, atol=1e-14)


def _torch_block(p, b, h, mod6, n_heads):
    """The same block composed from torch.nn.functional routines (float64)."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    H = h.shape[1]
    d = H // n_heads
    sh1, sc1, g1, sh2, sc2, g2 = (t(r) for r in mod6)
    h = t(h)
    W = lambda n: t(p[f"blocks.{b}.{n}"])
    a = Fnn.layer_norm(h, (H,), eps=1e-6) * (1 + sc1) + sh1
    qkv = Fnn.linear(a, W("qkv.w").T, W("qkv.b"))
    q, k, v = qkv.split(H, dim=1)
    heads = lambda z: z.view(-1, n_heads, d).transpose(0, 1)
    o = Fnn.scaled_dot_product_attention(heads(q), heads(k), heads(v)).transpose(0, 1).reshape(-1, H)
    h = h + g1 * Fnn.linear(o, W("o.w").T, W("o.b"))
    a2 = Fnn.layer_norm(h, (H,), eps=1e-6) * (1 + sc2) + sh2
    f = Fnn.gelu(Fnn.linear(a2, W("ffn1.w").T, W("ffn1.b")), approximate="tanh")
    return (h + g2 * Fnn.linear(f, W("ffn2.w").T, W("ffn2.b"))).numpy()


def test_block_vs_torch_composition():
    m = _toy_model()
    cfg = TOY
    h = np.random.default_rng(9).normal(size=(cfg.n_tokens, cfg.hidden))
    mod = m.modulation(0.8)["blocks"][1]
    np.testing.assert_allclose(m.block(h, 1, mod), _torch_block(m.p, 1, h, mod, cfg.n_heads), rtol=1e-10, atol=1e-12)


def test_bf16_model_rounds_only_gemm_weights():
    cfg = TOY.replace(dtype="bf16")
    p = ai.weights(cfg)
    m = O.DiTModel(cfg, p)
    for n in ("blocks.0.qkv.w", "blocks.1.ffn2.w", "head.w"):
        np.testing.assert_array_equal(m.w(n), O.bf16_round(p[n]).astype(np.float64))
        assert not np.array_equal(m.w(n), p[n].astype(np.float64))
    for n in ("blocks.0.ada.w", "temb.w1", "blocks.0.qkv.b", "head.ada.w"):
        np.testing.assert_array_equal(m.w(n), p[n].astype(np.float64))


# ------------------------------------------------------------- the loop


class _StubModel:
    """Constant residual c and constant velocity v: the loop's result does not
    depend on which steps are skipped, and sum of the Euler steps is -1."""

    def __init__(self, H, c, v):
        self.c, self.v = c, v

    def temni(self, x, sigma):
        return np.asarray(x, np.float64) * (1 + sigma)

    def stack(self, x, sigma, text=None):
        return np.asarray(x, np.float64) + self.c

    def head(self, h, sigma):
        return self.v + 0 * h


def test_sigma_schedule():
    s = ai.sigmas(10)
    assert s[0] == 1.0 and s[-1] == 0.0 and len(s) == 11
    assert float(np.sum(np.diff(s.astype(np.float64)))) == -1.0


def test_loop_euler_and_cache_plumbing():
    rng = np.random.default_rng(10)
    x0 = rng.normal(size=(6, 4))
    c, v = rng.normal(size=(6, 4)), rng.normal(size=(6, 4))
    m = _StubModel(4, c, v)
    sig = ai.sigmas(8)
    xs = []
    for mode, gp in (("nocache", None), ("acid", O.GateParams(0.05, 0.2, 0.01)),
                     ("acid", O.GateParams(math.inf, math.inf, 0.01))):
        x, tr = O.denoise_loop(m, x0, sig, mode=mode, gate=gp)
        xs.append(x)
        np.testing.assert_allclose(x, x0 - v, rtol=1e-13, atol=1e-13)
    assert tr["compute"].sum() == 1
    # forcing a skip on step 0 has no residual to reuse
    with pytest.raises(ValueError):
        O.denoise_loop(m, x0, sig, mode="acid", gate=O.GateParams(0, 0, 0), forced_schedule=[0] * 8)


def test_loop_residual_reuse_semantics():
    """On a skipped step h_out = x + r with r from the last computed step."""
    class Rec(_StubModel):
        def __init__(self):
            self.calls = []

        def stack(self, x, sigma, text=None):
            self.calls.append(sigma)
            return 2.0 * np.asarray(x) + sigma

        def head(self, h, sigma):
            return h

    sig = ai.sigmas(4)
    x0 = np.ones((1, 1))
    m = Rec()
    x, tr = O.denoise_loop(m, x0, sig, mode="acid", gate=O.GateParams(0, 0, 0),
                           forced_schedule=[1, 0, 1, 0])
    # step 0: h = 2*1+1 = 3, r = 2, x1 = 1 - 0.25*3 = 0.25
    # step 1: skip, h = x1 + r = 2.25, x2 = 0.25 - 0.25*2.25 = -0.3125
    # step 2: h = 2*(-0.3125)+0.5 = -0.125, r = 0.1875, x3 = -0.3125 + 0.25*0.125 = -0.28125
    # step 3: skip, h = -0.28125+0.1875 = -0.09375, x4 = -0.28125 + 0.25*0.09375 = -0.2578125
    assert x[0, 0] == -0.2578125
    assert list(tr["compute"]) == [1, 0, 1, 0]
    assert m.calls == [1.0, 0.5]


def test_loop_threshold_invariants_on_dit():
    cfg = TOY
    m = _toy_model(std=0.3)
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    sig = ai.sigmas(cfg.n_steps)
    x_nc, tr_nc = O.denoise_loop(m, x0, sig, text, mode="nocache")
    assert tr_nc["compute"].all()
    x_0, tr_0 = O.denoise_loop(m, x0, sig, text, mode="acid", gate=O.GateParams(0.0, 0.0, 0.01))
    assert tr_0["compute"].all()
    assert np.array_equal(x_0, x_nc)
    x_inf, tr_inf = O.denoise_loop(m, x0, sig, text, mode="acid", gate=O.GateParams(math.inf, math.inf, 0.01))
    assert list(tr_inf["compute"]) == [1] + [0] * (cfg.n_steps - 1)
    _, tr_f = O.denoise_loop(m, x0, sig, text, mode="acid", gate=O.GateParams(0.1, 0.1, 0.01))
    assert list(tr_f["compute"].astype(bool)) == _fixed_skeleton(list(tr_f["s"]), 0.1)
    # drift trace: step 0 has no signal, later ones are positive
    assert math.isnan(tr_f["s"][0]) and np.all(tr_f["s"][1:] > 0)
    # replaying the gate on the loop's own drift trace gives the same decisions
    dec, _, _ = O.gate_schedule(list(tr_f["s"]), O.GateParams(0.1, 0.1, 0.01))
    assert dec == list(tr_f["gate_compute"].astype(bool))


def test_psnr():
    ref = np.array([0.0, 1.0, 0.5, 0.25])
    assert O.psnr(ref + 0.1, ref) == pytest.approx(20.0, rel=1e-12)
    assert O.psnr(ref, ref) == math.inf

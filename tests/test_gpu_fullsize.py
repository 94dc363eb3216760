"""GPU parity at the workloads' full sizes, in the launch configurations the
benchmark times, on outputs the oracle can compute one by one (sampled query
rows / token rows), plus properties that hold at any size.

Shapes: Wan-2.1-1.3B (12 x 32760 x 128, H 1536, F 8960), CogVideoX-5B
(48 x 17776 x 64, H 3072, F 12288; one block in both the sequential and the
parallel form) and the HunyuanVideo slice (24 x 119056 x 128).  Inputs are seeded torch / NumPy draws; bf16 operands
are compared with an oracle fed the same bf16 values.
"""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import (BF16_U, assert_close_to_scale, assert_elementwise, attention_bound,
                      make_model, need_gpu, rel_err, to_dev, to_np)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def P():
    return need_gpu()


def _seeded(shape, seed, std=1.0, dtype=torch.bfloat16):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device="cuda") * std).to(dtype)


ATTN_SHAPES = [(12, 32760, 128), (48, 17776, 64), (24, 119056, 128)]


@pytest.mark.parametrize("prescaled", [False, True], ids=["plain-q", "prescaled-q"])
@pytest.mark.parametrize("nh,L,d", ATTN_SHAPES, ids=["wan", "cogvideox", "hunyuan"])
def test_attention_fullsize_sampled(P, nh, L, d, prescaled):
    """Sampled rows at the workloads' full sizes; prescaled-q is the launch
    configuration of the model's loop (Q stored times log2(e)/sqrt(d))."""
    q = _seeded((nh, L, d), 1)
    c = np.float32(P.q_scale(d))
    if prescaled:
        q = (q.float() * float(c)).to(torch.bfloat16)
    k = _seeded((nh, L, d), 2)
    v = _seeded((nh, L, d), 3)
    vt_ld = (L + 7) // 8 * 8
    vt = torch.zeros((nh, d, vt_ld), dtype=torch.bfloat16, device="cuda")
    vt[:, :, :L] = v.transpose(1, 2)
    o = torch.empty((L, nh * d), dtype=torch.bfloat16, device="cuda")
    P.attention(q, k, vt, o, q_prescaled=prescaled)
    torch.cuda.synchronize()
    rng = np.random.default_rng(L)
    heads = sorted(rng.choice(nh, 3, replace=False))
    rows = np.unique(np.concatenate([rng.choice(L, 40, replace=False), [0, L - 1]]))
    for j in heads:
        kj, vj = to_np(k[j]), to_np(v[j])
        qj = to_np(q[j])[rows].astype(np.float64)
        if prescaled:
            qj = qj / np.float64(c)
        ref = O.attention(qj, kj, vj)
        got = to_np(o[rows, j * d:(j + 1) * d])
        assert rel_err(got, ref) < 1e-2, (j, rel_err(got, ref))
        assert_elementwise(got, ref, attention_bound(qj, kj, vj), 1.05 * BF16_U,
                           f"{nh}x{L}x{d} head {j}")


GEMM_SHAPES = [  # (name, M, N, K, epilogue)
    ("wan-qkv", 32760, 4608, 1536, "qkv"), ("wan-proj", 32760, 1536, 1536, "gate_residual"),
    ("wan-ffn1", 32760, 8960, 1536, "gelu"), ("wan-ffn2", 32760, 1536, 8960, "gate_residual"),
    ("wan-head", 32760, 1536, 1536, "euler"),
    ("cog-qkv", 17776, 9216, 3072, "qkv"), ("cog-ffn2", 17776, 3072, 12288, "gate_residual"),
    ("hunyuan-ffn1", 119056, 12288, 3072, "gelu"), ("hunyuan-head", 118800, 3072, 3072, "bias"),
]


@pytest.mark.parametrize("name,M,N,K,kind", GEMM_SHAPES, ids=[g[0] for g in GEMM_SHAPES])
def test_linear_fullsize_sampled(P, name, M, N, K, kind):
    a = _seeded((M, K), 11)
    wt = _seeded((N, K), 12, std=1.0 / math.sqrt(K))
    b = _seeded((N,), 13, std=0.1, dtype=torch.float32)
    rng = np.random.default_rng(M + N)
    rows = np.unique(np.concatenate([rng.choice(M, 48, replace=False), [0, M - 1]]))
    ref = to_np(a[rows]) @ to_np(wt).T + to_np(b)
    if kind == "qkv":
        d = 128 if name.startswith("wan") else 64
        nh = N // (3 * d)
        H = nh * d
        q = torch.empty((nh, M, d), dtype=torch.bfloat16, device="cuda")
        kk = torch.empty((nh, M, d), dtype=torch.bfloat16, device="cuda")
        vt = torch.empty((nh, d, (M + 7) // 8 * 8), dtype=torch.bfloat16, device="cuda")
        P.linear(a, wt, P.ACID_EPI_QKV, b, q=q, k=kk, vt=vt, n_heads=nh, head_dim=d)
        torch.cuda.synchronize()
        got = np.concatenate([to_np(q[:, rows, :]).transpose(1, 0, 2).reshape(len(rows), H),
                              to_np(kk[:, rows, :]).transpose(1, 0, 2).reshape(len(rows), H),
                              to_np(vt[:, :, rows]).transpose(2, 0, 1).reshape(len(rows), H)], 1)
        assert rel_err(got, ref) < 5e-3
    elif kind == "gelu":
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        P.linear(a, wt, P.ACID_EPI_BIAS_GELU, b, out=out)
        torch.cuda.synchronize()
        assert rel_err(to_np(out[rows]), O.gelu_tanh(ref)) < 5e-3
    elif kind == "bias":
        out = torch.empty((M, N), device="cuda")
        P.linear(a, wt, P.ACID_EPI_BIAS, b, out=out)
        torch.cuda.synchronize()
        assert rel_err(to_np(out[rows]), ref) < 1e-5
    else:
        h0 = _seeded((M, N), 14, dtype=torch.float32)
        h = h0.clone()
        if kind == "gate_residual":
            g = _seeded((N,), 15, dtype=torch.float32)
            P.linear(a, wt, P.ACID_EPI_GATE_RESIDUAL, b, gate=g, out=h)
            want = to_np(g) * ref
        else:
            P.linear(a, wt, P.ACID_EPI_EULER, b, out=h, dsigma=-0.02)
            want = -0.02 * ref
        torch.cuda.synchronize()
        assert rel_err(to_np(h[rows]) - to_np(h0[rows]), want) < 1e-5


@pytest.fixture(scope="module")
def wan_block(P):
    """The Wan-shape stack reduced to its first block (same weights as the
    30-block stack's block 0), with the workspace of the full token count."""
    cfg = ai.WAN13B.replace(n_blocks=1, n_steps=2)
    m, params = make_model(P, cfg, max_steps=2)
    return cfg, m, O.DiTModel(cfg, params)


def test_block_fullsize_wan_sampled(P, wan_block):
    cfg, m, om = wan_block
    H = cfg.hidden
    h0 = ai.gaussian((cfg.n_tokens, H), 21)
    mod6 = om.modulation(0.62)["blocks"][0].astype(np.float32)
    h = to_dev(h0)
    m.block_forward(0, to_dev(mod6), h)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.random.default_rng(5).choice(cfg.n_tokens, 48, replace=False),
                                     [0, cfg.n_tokens - 1]]))
    ref = om.block(h0, 0, mod6.astype(np.float64), rows=rows)
    got = to_np(h[rows])
    assert rel_err(got - h0[rows], ref - h0[rows]) < 2e-2
    assert_close_to_scale(got - h0[rows], ref - h0[rows], True, "wan block")
    assert np.all(np.isfinite(to_np(h)))


@pytest.mark.parametrize("block", ["sequential", "parallel"])
def test_block_fullsize_cogvideox_sampled(P, block):
    """One block at the CogVideoX-5B shape (226 text + 17550 video tokens,
    48 x 64 heads, H 3072, F 12288, bf16) in both block forms, on sampled
    rows (text rows, video rows, both ends) against the oracle's block with
    K/V over all tokens."""
    cfg = ai.COG5B.replace(n_blocks=1, n_steps=2, block=block)
    m, params = make_model(P, cfg, max_steps=2)
    om = O.DiTModel(cfg, params)
    H = cfg.hidden
    h0 = ai.gaussian((cfg.n_tokens, H), 23)
    mod6 = om.modulation(0.41)["blocks"][0].astype(np.float32)
    h = to_dev(h0)
    m.block_forward(0, to_dev(mod6), h)
    torch.cuda.synchronize()
    rng = np.random.default_rng(6)
    rows = np.unique(np.concatenate([rng.choice(cfg.n_text, 8, replace=False),
                                     cfg.n_text + rng.choice(cfg.n_video, 32, replace=False),
                                     [0, cfg.n_text - 1, cfg.n_text, cfg.n_tokens - 1]]))
    ref = om.block(h0, 0, mod6.astype(np.float64), rows=rows)
    assert rel_err(to_np(h[rows]) - h0[rows], ref - h0[rows]) < 2e-2
    assert_close_to_scale(to_np(h[rows]) - h0[rows], ref - h0[rows], True, f"cogvideox {block} block")
    assert np.all(np.isfinite(to_np(h)))


def test_drift_fullsize_wan(P, wan_block):
    cfg, m, om = wan_block
    x0 = ai.latents(cfg)
    x1 = (x0 + 0.02 * ai.gaussian(x0.shape, 22)).astype(np.float32)
    H = cfg.hidden
    m0 = torch.empty((cfg.n_video, H), device="cuda")
    m1 = torch.empty_like(m0)
    m.drift_signal(to_dev(x0), 1.0, None, m0)
    s = m.drift_signal(to_dev(x1), 0.98, m0, m1)
    ref = O.relative_l1_drift(om.temni(x1, 0.98), om.temni(x0, 1.0))
    assert abs(s - ref) / ref < 1e-3
    assert s == m.drift_signal(to_dev(x1), 0.98, m0, m1)  # deterministic


def test_l1_norms_and_reuse_fullsize_wan(P, wan_block):
    cfg, m, _ = wan_block
    n = cfg.n_video * cfg.hidden
    a = _seeded((n,), 41, dtype=torch.float32)
    b = _seeded((n,), 42, dtype=torch.float32)
    c = _seeded((n,), 43, dtype=torch.float32)
    got = m.l1_norms(a, b, c)
    ref0 = float((a.double() - b.double()).abs().sum())
    ref1 = float(c.double().abs().sum())
    assert got[0] == pytest.approx(ref0, rel=1e-6) and got[1] == pytest.approx(ref1, rel=1e-12)
    assert m.l1_norms(a, b, c) == got
    x0 = a.clone()
    xp = torch.empty_like(a)
    v = torch.empty_like(a)
    P.easycache_reuse(a, xp, v, b, -0.02)
    torch.cuda.synchronize()
    idx = torch.from_numpy(np.random.default_rng(6).integers(0, n, 200000)).cuda()
    assert torch.equal(v[idx], x0[idx] + b[idx]) and torch.equal(xp[idx], x0[idx])
    np.testing.assert_allclose(to_np(a[idx]), to_np(x0[idx]) + -0.02 * to_np(v[idx]),
                               rtol=1e-6, atol=1e-6)


def test_cache_fullsize_wan(P):
    n = ai.WAN13B.n_video * ai.WAN13B.hidden
    x = _seeded((n,), 31, dtype=torch.float32)
    h = _seeded((n,), 32, dtype=torch.float32)
    r = torch.empty_like(x)
    P.cache_apply(P.ACID_CACHE_STORE, x, h, r)
    h2 = torch.empty_like(x)
    P.cache_apply(P.ACID_CACHE_APPLY, x, h2, r)
    torch.cuda.synchronize()
    idx = np.random.default_rng(3).integers(0, n, 200000)
    xs, hs = to_np(x[idx]), to_np(h[idx])
    np.testing.assert_allclose(to_np(r[idx]), hs - xs, rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(to_np(h2[idx]), hs, rtol=1e-6, atol=1e-6)


def test_denoise_loop_wan_fullsize_properties(P):
    """The 30-block Wan-shape loop exactly as the benchmark runs it: the gate
    fed the loop's own drift trace reproduces its decisions bit for bit, the
    run is deterministic, and tau = inf computes only the first step."""
    cfg = ai.WAN13B
    m, _ = make_model(P, cfg, max_steps=cfg.n_steps)
    x0 = torch.from_numpy(ai.latents(cfg)).cuda()
    sig = ai.sigmas(cfg.n_steps)
    x = x0.clone()
    tr = m.denoise_loop(x, sig, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01)
    dec, _, _ = O.gate_schedule(list(tr["s"]), O.GateParams(0.05, 0.2, 0.01))
    assert list(tr["gate_compute"].astype(bool)) == dec
    assert np.all(tr["compute"] == tr["gate_compute"])
    s = tr["s"][1:]
    assert np.all(np.isfinite(s)) and np.all(s > 0)
    assert np.all(np.isfinite(to_np(x)))
    x2 = x0.clone()
    tr2 = m.denoise_loop(x2, sig, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01)
    assert torch.equal(x, x2) and np.array_equal(tr["s"][1:], tr2["s"][1:])
    # the gate on the device and the loop captured as a graph: the same bits
    for _ in range(2):
        xg = x0.clone()
        trg = m.denoise_loop(xg, sig, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01,
                             graph=True)
        assert torch.equal(xg, x)
        assert np.array_equal(trg["compute"], tr["compute"])
        assert np.array_equal(trg["s"][1:], tr["s"][1:])
        assert np.array_equal(trg["sigma_sum_after"], tr["sigma_sum_after"])
    x3 = x0.clone()
    tr3 = m.denoise_loop(x3, sig, mode="acid", tau_low=math.inf, tau_high=math.inf, delta=0.01)
    assert int(tr3["compute"].sum()) == 1 and tr3["compute"][0] == 1
    assert math.isnan(tr["s"][0])  # no drift before the first step
    # the EasyCache signal under the same gate, as the benchmark runs it
    xe = x0.clone()
    tre = m.denoise_loop(xe, sig, mode="easycache", tau_low=0.1, tau_high=0.2, delta=0.01)
    dec, _, _ = O.gate_schedule(list(tre["s"]), O.GateParams(0.1, 0.2, 0.01, 2))
    assert list(tre["gate_compute"].astype(bool)) == dec
    assert np.all(np.isfinite(tre["s"][2:])) and np.all(np.isfinite(to_np(xe)))
    xi = x0.clone()
    tri = m.denoise_loop(xi, sig, mode="easycache", tau_low=math.inf, tau_high=math.inf,
                         delta=0.01)
    assert list(tri["compute"]) == [1, 1] + [0] * (cfg.n_steps - 2)
    # DiCache's probe signal: the gate replays it, and the captured device-gate
    # loop gives the same bits as the host-gated one
    m.set_probe_blocks(1)
    xd = x0.clone()
    trd = m.denoise_loop(xd, sig, mode="dicache", tau_low=0.07, tau_high=0.225, delta=0.01)
    dec, _, _ = O.gate_schedule(list(trd["s"]), O.GateParams(0.07, 0.225, 0.01))
    assert list(trd["gate_compute"].astype(bool)) == dec
    assert 0 < trd["compute"].sum() < cfg.n_steps
    xdg = x0.clone()
    trdg = m.denoise_loop(xdg, sig, mode="dicache", tau_low=0.07, tau_high=0.225, delta=0.01,
                          graph=True)
    assert torch.equal(xdg, xd) and np.array_equal(trdg["compute"], trd["compute"])
    assert np.array_equal(trdg["s"][1:], trd["s"][1:])


def test_denoise_loop_small_bf16_vs_oracle(P):
    """The small bf16 workload (4 blocks, H 1024, 1024 tokens, 30 steps):
    the oracle loop forced to the GPU's schedule reproduces x_N and the
    drift trace; the gate fed the GPU's drift reproduces its schedule."""
    cfg = ai.SMALL
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    om = O.DiTModel(cfg, params)
    x0 = ai.latents(cfg)
    sig = ai.sigmas(cfg.n_steps)
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01)
    dec, _, _ = O.gate_schedule(list(tr["s"]), O.GateParams(0.05, 0.2, 0.01))
    assert list(tr["gate_compute"].astype(bool)) == dec
    xr, otr = O.denoise_loop(om, x0, sig, mode="acid", gate=O.GateParams(0.05, 0.2, 0.01),
                             forced_schedule=tr["compute"])
    ok = ~np.isnan(otr["s"])
    np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=2e-2)
    assert rel_err(to_np(x) - x0, xr - x0) < 2e-2
    # the captured device-gate loop gives the same bits
    xg = to_dev(x0)
    trg = m.denoise_loop(xg, sig, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01,
                         graph=True)
    assert torch.equal(xg, x) and np.array_equal(trg["compute"], tr["compute"])

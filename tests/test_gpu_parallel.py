"""The parallel (single-stream) block on the GPU.

Its pieces: the GEMM epilogue that splits Q | K | V from the GELU part into a
row-strided buffer, the gated residual with a second bias, attention writing
into a row-strided output; then the block, the step and the loop against the
oracle's parallel block, and, at the HunyuanVideo-slice shape, the property
that with zero MLP weights the parallel block is bit for bit the sequential
block (every kernel then sees identical operands, the projection's extra K
columns add exact zeros).
"""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import (assert_close_to_scale, bf16_values, make_model, need_gpu, rel_err,
                      to_dev, to_np)

pytestmark = pytest.mark.gpu

TINY_PAR = ai.TINY.replace(name="tiny-parallel", block="parallel", n_text=9, n_video=131)
SMALL_PAR = ai.DiTConfig("small-parallel-bf16", n_blocks=2, hidden=256, n_heads=2,
                         head_dim=128, ffn=640, n_video=300, n_text=7, dtype="bf16",
                         n_steps=8, block="parallel")
SMALL_PAR_D64 = SMALL_PAR.replace(name="small-parallel-d64", n_heads=4, head_dim=64,
                                  n_text=0, n_video=257)


@pytest.fixture(scope="module")
def P():
    return need_gpu()


@pytest.mark.parametrize("pre", [False, True], ids=["plain-q", "prescaled-q"])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("M,nh,d,F", [(1, 2, 64, 128), (300, 2, 64, 384), (513, 4, 128, 640)])
def test_linear_qkv_gelu(P, dtype, M, nh, d, F, pre):
    H = nh * d
    N, K = 3 * H + F, 256
    rng = np.random.default_rng(M + F)
    a = rng.normal(size=(M, K)).astype(np.float32)
    w = rng.normal(size=(K, N)).astype(np.float32) / math.sqrt(K)
    b = rng.normal(size=N).astype(np.float32) * 0.1
    if dtype == torch.bfloat16:
        a, w = bf16_values(a), bf16_values(w)
    y = a.astype(np.float64) @ w.astype(np.float64) + b
    vt_ld = ((M + 7) // 8) * 8
    q = torch.empty((nh, M, d), dtype=dtype, device="cuda")
    k = torch.empty((nh, M, d), dtype=dtype, device="cuda")
    vt = torch.zeros((nh, d, vt_ld), dtype=dtype, device="cuda")
    cat = torch.full((M, H + F), 7.0, dtype=dtype, device="cuda")  # attention half untouched
    P.linear(to_dev(a, dtype), to_dev(w.T.copy(), dtype), P.ACID_EPI_QKV_GELU, to_dev(b),
             q=q, k=k, vt=vt, n_heads=nh, head_dim=d, out=cat[:, H:], q_prescale=pre)
    tol = 1e-5 if dtype == torch.float32 else 4e-3
    qs = P.q_scale(d) if pre else 1.0
    assert rel_err(to_np(q), y[:, :H].reshape(M, nh, d).transpose(1, 0, 2) * qs) < tol
    assert rel_err(to_np(k), y[:, H:2 * H].reshape(M, nh, d).transpose(1, 0, 2)) < tol
    assert rel_err(to_np(vt)[:, :, :M], y[:, 2 * H:3 * H].reshape(M, nh, d).transpose(1, 2, 0)) < tol
    assert rel_err(to_np(cat[:, H:]), O.gelu_tanh(y[:, 3 * H:])) < tol
    assert bool((cat[:, :H] == 7.0).all())


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_linear_gate_residual_two_biases(P, dtype):
    M, N, K = 301, 384, 640
    rng = np.random.default_rng(11)
    a = rng.normal(size=(M, K)).astype(np.float32)
    w = rng.normal(size=(K, N)).astype(np.float32) / math.sqrt(K)
    b1 = rng.normal(size=N).astype(np.float32) * 0.1
    b2 = rng.normal(size=N).astype(np.float32) * 0.1
    g = rng.normal(size=N).astype(np.float32)
    if dtype == torch.bfloat16:
        a, w = bf16_values(a), bf16_values(w)
    h0 = rng.normal(size=(M, N)).astype(np.float32)
    h = to_dev(h0)
    P.linear(to_dev(a, dtype), to_dev(w.T.copy(), dtype), P.ACID_EPI_GATE_RESIDUAL, to_dev(b1),
             gate=to_dev(g), out=h, bias2=to_dev(b2))
    y = a.astype(np.float64) @ w.astype(np.float64) + b1 + b2
    assert rel_err(to_np(h) - h0, g * y) < 1e-5


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("L,d", [(65, 64), (300, 128)])
def test_parallel_without_mlp_is_sequential(P, dtype, L, d):
    """With zero MLP weights the parallel block equals the sequential block
    bit for bit: its attention, written into the first H columns of the
    [L][H + F] buffer, matches the dense write, and the projection over
    K = H + F adds exact zeros past H."""
    cfg = ai.DiTConfig("strided", n_blocks=1, hidden=2 * d, n_heads=2, head_dim=d, ffn=256,
                       n_video=L, dtype="bf16" if dtype == torch.bfloat16 else "f32",
                       n_steps=2, block="parallel")
    m, _ = make_model(P, cfg, max_steps=2)
    ref_cfg = cfg.replace(block="sequential")
    mr, _ = make_model(P, ref_cfg, max_steps=2)
    # zero MLP weights: the parallel block reduces to the sequential one exactly
    rng = np.random.default_rng(L)
    h0 = rng.normal(size=(L, cfg.hidden)).astype(np.float32)
    mod6 = to_dev(rng.normal(size=(6, cfg.hidden)).astype(np.float32) * 0.3)
    for mm, c in ((m, cfg), (mr, ref_cfg)):
        for name in ("blocks.0.ffn1.w", "blocks.0.ffn1.b", "blocks.0.ffn2.w", "blocks.0.ffn2.b"):
            tid = ai.tensor_id(c, name)
            shape = ai.manifest(c)[tid][1]
            mm.load_tensor(tid, torch.zeros(shape, device="cuda"))
    torch.cuda.synchronize()
    hp, hs = to_dev(h0), to_dev(h0)
    m.block_forward(0, mod6, hp)
    mr.block_forward(0, mod6, hs)
    torch.cuda.synchronize()
    assert torch.equal(hp, hs)


def _block_case(P, cfg, seed=3):
    m, params = make_model(P, cfg, max_steps=2, std=0.05)
    rng = np.random.default_rng(seed)
    h0 = rng.normal(size=(cfg.n_tokens, cfg.hidden)).astype(np.float32)
    mod6 = rng.normal(size=(6, cfg.hidden)).astype(np.float32) * 0.3
    h = to_dev(h0)
    m.block_forward(1 if cfg.n_blocks > 1 else 0, to_dev(mod6), h)
    torch.cuda.synchronize()
    ref = O.DiTModel(cfg, params).block(h0, 1 if cfg.n_blocks > 1 else 0, mod6.astype(np.float64))
    return to_np(h) - h0, ref - h0


@pytest.mark.parametrize("cfg,tol", [(TINY_PAR, 1e-4), (SMALL_PAR, 2e-2), (SMALL_PAR_D64, 2e-2)],
                         ids=lambda c: getattr(c, "name", str(c)))
def test_block_parallel_vs_oracle(P, cfg, tol):
    got, ref = _block_case(P, cfg)
    assert rel_err(got, ref) < tol
    assert_close_to_scale(got, ref, cfg.dtype == "bf16", f"{cfg.name} block")


@pytest.mark.parametrize("cfg,tol", [(TINY_PAR, 1e-4), (SMALL_PAR, 2e-2)], ids=lambda c: getattr(c, "name", str(c)))
def test_dit_step_parallel_vs_oracle(P, cfg, tol):
    m, params = make_model(P, cfg, max_steps=2)
    x = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    td = to_dev(text) if text is not None else None
    r = torch.empty((cfg.n_video, cfg.hidden), device="cuda")
    v = m.dit_step(to_dev(x), 0.61, td, resid=r)
    torch.cuda.synchronize()
    v_ref, h_ref = O.DiTModel(cfg, params).forward(x, 0.61, text)
    assert rel_err(to_np(v), v_ref) < tol
    assert rel_err(to_np(r), h_ref - x) < tol
    assert_close_to_scale(to_np(v), v_ref, cfg.dtype == "bf16", f"{cfg.name} v")
    assert_close_to_scale(to_np(r), h_ref - x, cfg.dtype == "bf16", f"{cfg.name} residual")


def test_denoise_loop_parallel_vs_oracle(P):
    """The fp32 parallel stack's loop: the gate replays the GPU's drift, the
    oracle loop forced to the GPU's schedule reproduces x_N, and the captured
    device-gate loop gives the same bits as the host loop."""
    cfg = TINY_PAR
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    om = O.DiTModel(cfg, params)
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    td = to_dev(text)
    sig = ai.sigmas(cfg.n_steps)
    gate = dict(tau_low=0.02, tau_high=0.06, delta=0.01)
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, td, mode="acid", **gate)
    dec, _, _ = O.gate_schedule(list(tr["s"]), O.GateParams(0.02, 0.06, 0.01))
    assert list(tr["gate_compute"].astype(bool)) == dec
    xr, otr = O.denoise_loop(om, x0, sig, text, mode="acid", gate=O.GateParams(0.02, 0.06, 0.01),
                             forced_schedule=tr["compute"])
    ok = ~np.isnan(otr["s"])
    np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=1e-3)
    assert rel_err(to_np(x), xr) < 1e-4
    xg = to_dev(x0)
    trg = m.denoise_loop(xg, sig, td, mode="acid", **gate, graph=True)
    assert torch.equal(xg, x) and np.array_equal(trg["compute"], tr["compute"])


def test_parallel_without_mlp_is_sequential_hunyuan_shape(P):
    """One block at the HunyuanVideo-slice shape (119056 tokens, H 3072,
    24 x 128 heads, F 12288, bf16) in the launch configuration the loop uses:
    with zero MLP weights the parallel block equals the sequential block bit
    for bit, and with its MLP weights it differs (both branches run)."""
    base = ai.HUNYUAN_PARALLEL.replace(n_blocks=1, n_steps=2)
    seq = base.replace(block="sequential")
    H, F = base.hidden, base.ffn
    rng = np.random.default_rng(0)
    h0 = torch.from_numpy(rng.normal(size=(base.n_tokens, H)).astype(np.float32)).cuda()
    mod6 = to_dev(rng.normal(size=(6, H)).astype(np.float32) * 0.3)
    outs = {}
    for c in (base, seq):
        m, _ = make_model(P, c, max_steps=2)
        h = h0.clone()
        m.block_forward(0, mod6, h)
        hz = h0.clone()
        for name in ("blocks.0.ffn1.w", "blocks.0.ffn1.b", "blocks.0.ffn2.w", "blocks.0.ffn2.b"):
            tid = ai.tensor_id(c, name)
            m.load_tensor(tid, torch.zeros(ai.manifest(c)[tid][1], device="cuda"))
        m.block_forward(0, mod6, hz)
        torch.cuda.synchronize()
        outs[c.block] = (h, hz)
        del m
        torch.cuda.empty_cache()
    assert torch.equal(outs["parallel"][1], outs["sequential"][1])
    assert bool(torch.isfinite(outs["parallel"][0]).all())
    assert not torch.equal(outs["parallel"][0], outs["parallel"][1])

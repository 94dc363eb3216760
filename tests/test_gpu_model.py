"""GPU parity of the five calls (dit_step, drift_signal, acid_gate inside the
loop, cache_apply inside the loop, denoise_loop) against the oracle.

Bars: fp32 step outputs within 1e-4 relative (Frobenius), bf16 within 2e-2,
drift within 1e-3 relative, gate decisions bit-exact when fed the same drift
values.  Block outputs are also compared through the residual r = h_out - x,
which removes the dominant x term.
"""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import assert_close_to_scale, make_model, need_gpu, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu

TINY_TEXT = ai.TINY.replace(name="tiny-text", n_text=9, n_video=131)
SMALL_BF16 = ai.DiTConfig("small-bf16-ragged", n_blocks=2, hidden=256, n_heads=2, head_dim=128,
                          ffn=640, n_video=300, n_text=7, dtype="bf16", n_steps=8)
SMALL_BF16_D64 = SMALL_BF16.replace(name="small-bf16-d64", n_heads=4, head_dim=64, n_text=0,
                                    n_video=257)
# FFN 4096 over 2 row tiles: the second FFN GEMM (K = 4096) splits its tiles
# into two K ranges with a fixed-order reduction of the partial sums
SMALL_BF16_SPLIT = SMALL_BF16.replace(name="small-bf16-ksplit", ffn=4096)


@pytest.fixture(scope="module")
def P():
    return need_gpu()


def _step_case(P, cfg, sigma, std=ai.WEIGHT_STD):
    m, params = make_model(P, cfg, max_steps=4, std=std)
    x = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    xd = to_dev(x)
    td = to_dev(text) if text is not None else None
    r = torch.empty_like(xd)
    v = m.dit_step(xd, sigma, td, resid=r)
    torch.cuda.synchronize()
    om = O.DiTModel(cfg, params)
    v_ref, h_ref = om.forward(x, sigma, text)
    return to_np(v), v_ref, to_np(r), h_ref - x


@pytest.mark.parametrize("cfg", [ai.TINY, TINY_TEXT], ids=lambda c: c.name)
@pytest.mark.parametrize("sigma", [1.0, 0.37])
def test_dit_step_f32(P, cfg, sigma):
    v, v_ref, r, r_ref = _step_case(P, cfg, sigma, std=0.1)
    assert rel_err(v, v_ref) < 1e-4
    assert rel_err(r, r_ref) < 1e-4
    assert_close_to_scale(v, v_ref, False, f"{cfg.name} v")
    assert_close_to_scale(r, r_ref, False, f"{cfg.name} residual")


@pytest.mark.parametrize("cfg", [SMALL_BF16, SMALL_BF16_D64, SMALL_BF16_SPLIT],
                         ids=lambda c: c.name)
def test_dit_step_bf16(P, cfg):
    v, v_ref, r, r_ref = _step_case(P, cfg, 0.6, std=0.05)
    assert rel_err(v, v_ref) < 2e-2
    assert rel_err(r, r_ref) < 2e-2
    assert_close_to_scale(v, v_ref, True, f"{cfg.name} v")
    assert_close_to_scale(r, r_ref, True, f"{cfg.name} residual")


def test_dit_step_bf16_k_split_is_deterministic(P):
    """The K-split GEMM's reduction adds the partial sums in a fixed order:
    repeated steps are bit-identical."""
    cfg = SMALL_BF16_SPLIT
    m, _ = make_model(P, cfg, max_steps=4, std=0.05)
    xd = to_dev(ai.latents(cfg))
    td = to_dev(ai.text_tokens(cfg))
    outs = []
    for _ in range(3):
        r = torch.empty_like(xd)
        v = m.dit_step(xd, 0.6, td, resid=r)
        torch.cuda.synchronize()
        outs.append((to_np(v), to_np(r)))
    for v, r in outs[1:]:
        assert np.array_equal(v, outs[0][0]) and np.array_equal(r, outs[0][1])


def test_timestep_modulation(P):
    cfg = ai.TINY.replace(n_blocks=3)
    m, params = make_model(P, cfg, max_steps=6)
    sig = ai.sigmas(5)
    tab = to_np(m.timestep_modulation(sig))
    om = O.DiTModel(cfg, params)
    for i, s in enumerate(sig):
        mod = om.modulation(float(s))
        ref = np.concatenate([np.stack(mod["blocks"]).reshape(-1, cfg.hidden), mod["head"]])
        assert rel_err(tab[i], ref) < 1e-5


# hidden 384: 96 float4 chunks per row, so 32 lanes of the second chunk
# read a clamped copy of the row's last chunk
TINY_384 = ai.TINY.replace(name="tiny-384", hidden=384, n_heads=6, ffn=768)


@pytest.mark.parametrize("cfg", [ai.TINY, SMALL_BF16, TINY_384], ids=lambda c: c.name)
def test_drift_signal(P, cfg):
    m, params = make_model(P, cfg, max_steps=4)
    om = O.DiTModel(cfg, params)
    rng = np.random.default_rng(3)
    x0 = ai.latents(cfg)
    x1 = x0 + 0.05 * rng.normal(size=x0.shape).astype(np.float32)
    H = cfg.hidden
    m0 = torch.empty((cfg.n_video, H), device="cuda")
    m1 = torch.empty_like(m0)
    s0 = m.drift_signal(to_dev(x0), 1.0, None, m0)
    assert math.isnan(s0)
    s1 = m.drift_signal(to_dev(x1), 0.9, m0, m1)
    ref_m0 = om.temni(x0, 1.0)
    ref_m1 = om.temni(x1, 0.9)
    assert rel_err(to_np(m0), ref_m0) < 1e-5
    assert rel_err(to_np(m1), ref_m1) < 1e-5
    ref_s = O.relative_l1_drift(ref_m1, ref_m0)
    assert abs(s1 - ref_s) / ref_s < 1e-3
    # deterministic reduction: bit-identical on repeat
    for _ in range(3):
        assert m.drift_signal(to_dev(x1), 0.9, m0, m1) == s1
    # identical inputs -> exactly 0
    assert m.drift_signal(to_dev(x0), 1.0, m0, torch.empty_like(m0)) == 0.0


def _replay_gate(trace, tau_low, tau_high, delta, n_warmup=1):
    dec, taus, _ = O.gate_schedule(list(trace["s"]), O.GateParams(tau_low, tau_high, delta, n_warmup))
    return np.array(dec, dtype=np.int32), taus


def _near_tie(o_trace, g_trace, i, tol=1e-3):
    """True if step i's decision could flip under drift errors of tol relative."""
    s = g_trace["s"]
    if i == 0:
        return False
    sums = abs(o_trace["sigma_sum_after"][i - 1]) + abs(s[i])
    tau = o_trace["tau_used"][i]
    near_tau = abs(o_trace["sigma_sum_after"][i - 1] + o_trace["s"][i] - tau) <= 4 * tol * sums + 1e-12
    near_delta = i > 1 and abs(abs(s[i] - s[i - 1]) - 0.01) <= 4 * tol * (abs(s[i]) + abs(s[i - 1]))
    return bool(near_tau or near_delta)


def test_denoise_loop_tiny_full(P):
    """The tiny fp32 workload end to end: schedule, drift trace and x_N."""
    cfg = ai.TINY
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    om = O.DiTModel(cfg, params)
    x0 = ai.latents(cfg)
    sig = ai.sigmas(cfg.n_steps)
    for lo, hi in ((0.05, 0.2), (0.01, 0.03), (0.02, 0.02)):
        x = to_dev(x0)
        tr = m.denoise_loop(x, sig, mode="acid", tau_low=lo, tau_high=hi, delta=0.01)
        xr, otr = O.denoise_loop(om, x0, sig, mode="acid", gate=O.GateParams(lo, hi, 0.01))
        # the gate fed the GPU's own drift trace reproduces its decisions exactly
        dec, taus = _replay_gate(tr, lo, hi, 0.01)
        assert np.array_equal(dec, tr["gate_compute"])
        # drift values agree with the oracle's
        ok = ~np.isnan(otr["s"])
        np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=1e-3)
        mism = np.nonzero(tr["compute"] != otr["compute"])[0]
        for i in mism:
            assert _near_tie(otr, tr, i), f"schedule differs at step {i} away from a tie"
        if len(mism) == 0:
            assert rel_err(to_np(x), xr) < 1e-4
        # outputs under the GPU's schedule
        xf, _ = O.denoise_loop(om, x0, sig, mode="acid", gate=O.GateParams(lo, hi, 0.01),
                               forced_schedule=tr["compute"])
        assert rel_err(to_np(x), xf) < 1e-4


def test_denoise_loop_threshold_invariants(P):
    cfg = ai.TINY
    m, _ = make_model(P, cfg, max_steps=cfg.n_steps)
    x0 = ai.latents(cfg)
    sig = ai.sigmas(cfg.n_steps)
    xn = to_dev(x0)
    trn = m.denoise_loop(xn, sig, mode="nocache")
    assert trn["compute"].all() and np.isnan(trn["s"]).all()
    x0d = to_dev(x0)
    tr0 = m.denoise_loop(x0d, sig, mode="acid", tau_low=0.0, tau_high=0.0, delta=0.01)
    assert tr0["compute"].all()
    assert torch.equal(xn, x0d)  # tau = 0 is the uncached loop, bit for bit
    xi = to_dev(x0)
    tri = m.denoise_loop(xi, sig, mode="acid", tau_low=math.inf, tau_high=math.inf, delta=0.01)
    assert list(tri["compute"]) == [1] + [0] * (cfg.n_steps - 1)
    xf = to_dev(x0)
    trf = m.denoise_loop(xf, sig, mode="acid", tau_low=0.03, tau_high=0.03, delta=0.01)
    fixed = O.gate_schedule(list(trf["s"]), O.GateParams(0.03, 0.03, 0.01))[0]
    assert list(trf["compute"].astype(bool)) == fixed
    # forced all-compute == nocache
    xa = to_dev(x0)
    m.denoise_loop(xa, sig, mode="acid", tau_low=1e9, tau_high=1e9, delta=0.01,
                   forced_schedule=np.ones(cfg.n_steps, np.uint8))
    assert torch.equal(xa, xn)


def test_denoise_loop_bf16_small(P):
    cfg = SMALL_BF16
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    om = O.DiTModel(cfg, params)
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    sig = ai.sigmas(cfg.n_steps)
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, to_dev(text), mode="acid", tau_low=0.01, tau_high=0.04, delta=0.005)
    dec, _ = _replay_gate(tr, 0.01, 0.04, 0.005)
    assert np.array_equal(dec, tr["gate_compute"])
    xr, otr = O.denoise_loop(om, x0, sig, text, mode="acid", gate=O.GateParams(0.01, 0.04, 0.005),
                             forced_schedule=tr["compute"])
    ok = ~np.isnan(otr["s"])
    np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=2e-2)
    assert rel_err(to_np(x) - x0, xr - x0) < 2e-2


def test_kernel_timer_counts_and_leaves_results_alone(P):
    """The per-kernel event timer (the bench's per-class durations): a timed
    loop gives the same bits as an untimed one, and counts one launch per
    kernel of each class (per computed block: one of each GEMM and attention,
    two LN-modulates; every step: drift, cache, head)."""
    cfg = ai.SMALL
    m, _ = make_model(P, cfg, max_steps=cfg.n_steps)
    x0 = ai.latents(cfg)
    sig = ai.sigmas(cfg.n_steps)
    gate = dict(tau_low=0.05, tau_high=0.2, delta=0.01)
    x_plain = to_dev(x0)
    tr = m.denoise_loop(x_plain, sig, mode="acid", **gate)
    m.reset_timing()
    m.set_timing(True)
    x_timed = to_dev(x0)
    tr2 = m.denoise_loop(x_timed, sig, mode="acid", **gate)
    torch.cuda.synchronize()
    tim = m.timing()
    m.set_timing(False)
    assert torch.equal(x_plain, x_timed)
    assert np.array_equal(tr["compute"], tr2["compute"])
    n_comp = int(tr["compute"].sum())
    blocks = n_comp * cfg.n_blocks
    for name in ("attention", "gemm_qkv", "gemm_proj", "gemm_ffn1", "gemm_ffn2"):
        assert tim[name][1] == blocks, (name, tim[name])
        assert tim[name][0] > 0.0
    assert tim["ln_mod"][1] == 2 * blocks + cfg.n_steps
    assert tim["gemm_head"][1] == cfg.n_steps
    assert tim["drift"][1] == cfg.n_steps


@pytest.mark.parametrize("cfg", [ai.TINY, SMALL_BF16, SMALL_BF16.replace(name="small-par", block="parallel")],
                         ids=lambda c: c.name)
def test_host_pointer_load_matches_device_load(P, cfg):
    """acid_model_load_tensor_host (fp32 [in][out] in host memory, staged
    through the workspace in row chunks) fills the arena byte for byte as
    acid_model_load_tensor does from a device copy."""
    m1 = P.Model(cfg, max_steps=2)
    m2 = P.Model(cfg, max_steps=2)
    m1.arena.zero_()
    m2.arena.zero_()
    for tid, _name, w in ai.iter_weights(cfg):
        m1.load_tensor(tid, torch.from_numpy(w).cuda())
        m2.load_tensor_host(tid, w)
    torch.cuda.synchronize()
    assert torch.equal(m1.arena, m2.arena)
    with pytest.raises(P.AcidError):
        m2.load_tensor_host(0, np.zeros(3, np.float32))  # wrong element count

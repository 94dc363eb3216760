"""GPU parity of the EasyCache path (signal of Section 2, paragraph
"EasyCache", under the gate of Algorithm 1) against the oracle: the L1-sum
and reuse kernels, and whole loops (gate decisions replayed bit-exactly from
the GPU's own signal, signal values and x_N under the GPU's schedule)."""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import make_model, need_gpu, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu

SMALL_BF16 = ai.DiTConfig("small-bf16-ragged", n_blocks=2, hidden=256, n_heads=2, head_dim=128,
                          ffn=640, n_video=300, n_text=7, dtype="bf16", n_steps=10)


@pytest.fixture(scope="module")
def P():
    return need_gpu()


@pytest.fixture(scope="module")
def tiny(P):
    cfg = ai.TINY
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    return cfg, m, O.DiTModel(cfg, params)


@pytest.mark.parametrize("n", [1, 3, 4, 1001, 4096 * 3 + 2, 128 * 256])
def test_l1_norms(P, tiny, n):
    _, m, _ = tiny
    rng = np.random.default_rng(n)
    a, b, c = (rng.normal(size=n).astype(np.float32) for _ in range(3))
    ad, bd, cd = to_dev(a), to_dev(b), to_dev(c)
    got = m.l1_norms(ad, bd, cd)
    ref0 = np.abs(a.astype(np.float64) - b).sum()
    ref1 = np.abs(c.astype(np.float64)).sum()
    assert got[0] == pytest.approx(ref0, rel=1e-6) and got[1] == pytest.approx(ref1, rel=1e-12)
    g2 = m.l1_norms(ad)
    assert g2[0] == pytest.approx(np.abs(a.astype(np.float64)).sum(), rel=1e-12) and g2[1] == 0.0
    assert m.l1_norms(ad, bd, cd) == got  # deterministic


def test_l1_norms_size_limit(P, tiny):
    cfg, m, _ = tiny
    a = torch.zeros(cfg.n_video * cfg.hidden + 4, device="cuda")
    with pytest.raises(P.AcidError):
        m.l1_norms(a)


@pytest.mark.parametrize("n", [1, 5, 4096 + 3, 300 * 256])
def test_easycache_reuse(P, n):
    rng = np.random.default_rng(n + 7)
    x = rng.normal(size=n).astype(np.float32)
    d = rng.normal(size=n).astype(np.float32)
    xd, dd = to_dev(x), to_dev(d)
    xp = torch.empty_like(xd)
    v = torch.empty_like(xd)
    P.easycache_reuse(xd, xp, v, dd, -0.125)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(v), (x + d).astype(np.float64))    # fp32 add, exact
    np.testing.assert_array_equal(to_np(xp), x.astype(np.float64))
    np.testing.assert_allclose(to_np(xd), x + (-0.125) * (x.astype(np.float64) + d),
                               rtol=1e-6, atol=1e-6)


def _replay(tr, lo, hi, delta, n_warmup=2):
    dec, _, _ = O.gate_schedule(list(tr["s"]), O.GateParams(lo, hi, delta, n_warmup))
    return np.array(dec, dtype=np.int32)


def _scale(m, cfg, x0, sig, text=None):
    """Median EasyCache signal of a run that skips every step after warmup."""
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, text, mode="easycache", tau_low=math.inf, tau_high=math.inf,
                        delta=0.0)
    assert list(tr["compute"]) == [1, 1] + [0] * (len(sig) - 3)
    s = tr["s"][2:]
    assert np.all(np.isfinite(s)) and np.all(s > 0)
    return float(np.median(s))


def test_easycache_loop_tiny(P, tiny):
    cfg, m, om = tiny
    x0 = ai.latents(cfg)
    sig = ai.sigmas(cfg.n_steps)
    sc = _scale(m, cfg, x0, sig)
    fwd = lambda x, s: om.forward(x, s)[0]
    for lo, hi, delta in ((1.5 * sc, 3.0 * sc, 0.05 * sc), (2.5 * sc, 2.5 * sc, 0.0),
                          (0.5 * sc, 4.0 * sc, 0.2 * sc)):
        x = to_dev(x0)
        tr = m.denoise_loop(x, sig, mode="easycache", tau_low=lo, tau_high=hi, delta=delta)
        # the gate fed the GPU's own signal reproduces its decisions exactly
        assert np.array_equal(_replay(tr, lo, hi, delta), tr["gate_compute"])
        assert np.array_equal(tr["compute"], tr["gate_compute"])
        # oracle loop under the GPU's schedule: signal and x_N
        xr, otr = O.easycache_loop(fwd, x0, sig, gate=O.GateParams(lo, hi, delta, 2),
                                   forced_schedule=tr["compute"])
        ok = ~np.isnan(otr["s"])
        assert np.array_equal(ok, ~np.isnan(tr["s"]))
        np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=1e-3)
        assert rel_err(to_np(x), xr) < 1e-4


def test_easycache_invariants(P, tiny):
    cfg, m, _ = tiny
    x0 = ai.latents(cfg)
    sig = ai.sigmas(cfg.n_steps)
    xn = to_dev(x0)
    m.denoise_loop(xn, sig, mode="nocache")
    x0d = to_dev(x0)
    tr0 = m.denoise_loop(x0d, sig, mode="easycache", tau_low=0.0, tau_high=0.0, delta=0.01)
    assert tr0["compute"].all()
    assert torch.equal(xn, x0d)  # tau = 0 is the uncached loop, bit for bit
    xf = to_dev(x0)
    m.denoise_loop(xf, sig, mode="easycache", tau_low=1e9, tau_high=1e9, delta=0.01,
                   forced_schedule=np.ones(cfg.n_steps, np.uint8))
    assert torch.equal(xn, xf)
    with pytest.raises(P.AcidError):
        m.denoise_loop(to_dev(x0), sig, mode="easycache", n_warmup=1)


def test_easycache_loop_bf16_text(P):
    cfg = SMALL_BF16
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    om = O.DiTModel(cfg, params)
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    sig = ai.sigmas(cfg.n_steps)
    td = to_dev(text)
    sc = _scale(m, cfg, x0, sig, td)
    lo, hi, delta = 1.5 * sc, 3.0 * sc, 0.05 * sc
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, td, mode="easycache", tau_low=lo, tau_high=hi, delta=delta)
    assert np.array_equal(_replay(tr, lo, hi, delta), tr["gate_compute"])
    xr, otr = O.easycache_loop(lambda x, s: om.forward(x, s, text)[0], x0, sig,
                               gate=O.GateParams(lo, hi, delta, 2), forced_schedule=tr["compute"])
    ok = ~np.isnan(otr["s"])
    np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=2e-2)
    assert rel_err(to_np(x) - x0, xr - x0) < 2e-2

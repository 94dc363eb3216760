"""GPU parity of the DiCache path (probe signal of Section 2, paragraph
"DiCache", under the gate of Algorithm 1) against the oracle, plus its two
limits on the GPU itself: every block in the probe reproduces the no-cache
loop bit for bit, no probe block reproduces the TeaCache-style loop under
the same schedule bit for bit."""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import make_model, need_gpu, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu

TINY3 = ai.TINY.replace(name="tiny-3blk", n_blocks=3)
SMALL_BF16 = ai.DiTConfig("small-bf16-ragged", n_blocks=3, hidden=256, n_heads=2, head_dim=128,
                          ffn=640, n_video=300, n_text=7, dtype="bf16", n_steps=10)


@pytest.fixture(scope="module")
def P():
    return need_gpu()


@pytest.fixture(scope="module")
def tiny3(P):
    m, params = make_model(P, TINY3, max_steps=TINY3.n_steps, std=0.1)
    return m, O.DiTModel(TINY3, params)


def _scale(m, x0, sig, text=None):
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, text, mode="dicache", tau_low=math.inf, tau_high=math.inf,
                        delta=0.0)
    s = tr["s"][1:]
    assert np.all(np.isfinite(s)) and np.all(s > 0)
    return float(np.median(s))


def _replay(tr, lo, hi, delta):
    dec, _, _ = O.gate_schedule(list(tr["s"]), O.GateParams(lo, hi, delta))
    return np.array(dec, dtype=np.int32)


def test_dicache_loop_tiny(P, tiny3):
    m, om = tiny3
    m.set_probe_blocks(1)
    x0 = ai.latents(TINY3)
    sig = ai.sigmas(TINY3.n_steps)
    sc = _scale(m, x0, sig)
    for lo, hi, delta in ((1.2 * sc, 2.5 * sc, 0.05 * sc), (2.0 * sc, 2.0 * sc, 0.0)):
        x = to_dev(x0)
        tr = m.denoise_loop(x, sig, mode="dicache", tau_low=lo, tau_high=hi, delta=delta)
        assert np.array_equal(_replay(tr, lo, hi, delta), tr["gate_compute"])
        assert 0 < tr["compute"].sum() < TINY3.n_steps
        xr, otr = O.dicache_loop(om, x0, sig, gate=O.GateParams(lo, hi, delta), n_probe=1,
                                 forced_schedule=tr["compute"])
        ok = ~np.isnan(otr["s"])
        np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=1e-3)
        assert rel_err(to_np(x), xr) < 1e-4


def test_dicache_limits(P, tiny3):
    m, _ = tiny3
    x0 = ai.latents(TINY3)
    sig = ai.sigmas(TINY3.n_steps)
    xn = to_dev(x0)
    m.denoise_loop(xn, sig, mode="nocache")
    # every block in the probe: the deep residual is zero, any schedule is exact
    m.set_probe_blocks(TINY3.n_blocks)
    xf = to_dev(x0)
    trf = m.denoise_loop(xf, sig, mode="dicache", tau_low=math.inf, tau_high=math.inf, delta=0.0)
    assert trf["compute"].sum() == 1
    assert torch.equal(xf, xn)
    # no probe block: residual reuse on the raw input, as the TeaCache-style loop
    m.set_probe_blocks(0)
    sc = _scale(m, x0, sig)
    x0p = to_dev(x0)
    tr0 = m.denoise_loop(x0p, sig, mode="dicache", tau_low=1.2 * sc, tau_high=2.5 * sc,
                         delta=0.05 * sc)
    assert 0 < tr0["compute"].sum() < TINY3.n_steps
    xt = to_dev(x0)
    m.denoise_loop(xt, sig, mode="acid", tau_low=1e9, tau_high=1e9, delta=0.0,
                   forced_schedule=tr0["compute"].astype(np.uint8))
    assert torch.equal(x0p, xt)
    # tau = 0: the no-cache loop
    m.set_probe_blocks(1)
    xz = to_dev(x0)
    trz = m.denoise_loop(xz, sig, mode="dicache", tau_low=0.0, tau_high=0.0, delta=0.0)
    assert trz["compute"].all() and torch.equal(xz, xn)
    with pytest.raises(P.AcidError):
        m.set_probe_blocks(TINY3.n_blocks + 1)
    with pytest.raises(P.AcidError):
        m.set_probe_blocks(-1)


def test_dicache_loop_bf16_text(P):
    cfg = SMALL_BF16
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    m.set_probe_blocks(1)
    om = O.DiTModel(cfg, params)
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    td = to_dev(text)
    sig = ai.sigmas(cfg.n_steps)
    sc = _scale(m, x0, sig, td)
    lo, hi, delta = 1.2 * sc, 2.5 * sc, 0.05 * sc
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, td, mode="dicache", tau_low=lo, tau_high=hi, delta=delta)
    assert np.array_equal(_replay(tr, lo, hi, delta), tr["gate_compute"])
    xr, otr = O.dicache_loop(om, x0, sig, text, gate=O.GateParams(lo, hi, delta), n_probe=1,
                             forced_schedule=tr["compute"])
    ok = ~np.isnan(otr["s"])
    np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=2e-2)
    assert rel_err(to_np(x) - x0, xr - x0) < 2e-2

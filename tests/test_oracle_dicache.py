"""Pins of the oracle's DiCache loop (probe signal of Section 2, paragraph
"DiCache", under the gate of Algorithm 1) through its two limits: with no
probe blocks it is residual reuse on the raw input (the pinned TeaCache loop
under the same schedule) with signal |x_i - x_{i-1}|_1 / |x_{i-1}|_1; with
every block in the probe the deep residual is zero and every schedule gives
the no-cache result."""
import math

import numpy as np
import pytest

import acid_inputs as ai
import oracle as O

CFG = ai.TINY.replace(name="tiny-3blk", n_blocks=3, n_video=24, hidden=256, n_heads=4,
                      head_dim=64, ffn=512, n_steps=8)


@pytest.fixture(scope="module")
def model():
    return O.DiTModel(CFG, ai.weights(CFG, std=0.1))


def _case():
    x0 = ai.latents(CFG).astype(np.float64)
    return x0, ai.sigmas(CFG.n_steps).astype(np.float64)


def _scale(model, x0, sig, n_probe):
    _, tr = O.dicache_loop(model, x0, sig, gate=O.GateParams(math.inf, math.inf, 0.0),
                           n_probe=n_probe)
    return float(np.median(tr["s"][1:]))


def test_dicache_no_probe_is_input_residual_reuse(model):
    x0, sig = _case()
    sc = _scale(model, x0, sig, 0)
    gp = O.GateParams(1.2 * sc, 2.5 * sc, 0.05 * sc)
    x, tr = O.dicache_loop(model, x0, sig, gate=gp, n_probe=0)
    # the signal is the relative L1 change of the raw input, recomputed here
    # from the same trajectory's schedule replayed through the TeaCache loop
    xt, _ = O.denoise_loop(model, x0, sig, mode="acid", gate=gp, forced_schedule=tr["compute"])
    np.testing.assert_allclose(x, xt, rtol=1e-12, atol=1e-12)
    assert 0 < tr["compute"].sum() < CFG.n_steps
    xs = [x0]
    for i in range(CFG.n_steps - 1):  # rebuild x_i with the loop's schedule
        xi, _ = O.denoise_loop(model, x0, sig[: i + 2], mode="acid", gate=gp,
                               forced_schedule=tr["compute"][: i + 1])
        xs.append(xi)
    for i in range(1, CFG.n_steps):
        d = np.abs(xs[i] - xs[i - 1]).sum() / np.abs(xs[i - 1]).sum()
        assert tr["s"][i] == pytest.approx(d, rel=1e-12)


def test_dicache_full_probe_is_nocache(model):
    x0, sig = _case()
    xn, _ = O.denoise_loop(model, x0, sig, mode="nocache")
    sc = _scale(model, x0, sig, CFG.n_blocks)
    for gp in (O.GateParams(1.2 * sc, 2.5 * sc, 0.05 * sc), O.GateParams(math.inf, math.inf, 0.01)):
        _, trg = O.dicache_loop(model, x0, sig, gate=gp, n_probe=CFG.n_blocks)
        assert trg["compute"].sum() < CFG.n_steps
        x, tr = O.dicache_loop(model, x0, sig, gate=gp, n_probe=CFG.n_blocks)
        np.testing.assert_allclose(x, xn, rtol=1e-13, atol=1e-13)
    assert tr["compute"].sum() == 1


def test_dicache_tau_zero_is_nocache(model):
    x0, sig = _case()
    xn, _ = O.denoise_loop(model, x0, sig, mode="nocache")
    x, tr = O.dicache_loop(model, x0, sig, gate=O.GateParams(0.0, 0.0, 0.01), n_probe=1)
    assert tr["compute"].all()
    np.testing.assert_allclose(x, xn, rtol=1e-13, atol=1e-13)


def test_dicache_rejects_bad_probe(model):
    x0, sig = _case()
    with pytest.raises(ValueError):
        O.dicache_loop(model, x0, sig, gate=O.GateParams(0.1, 0.2, 0.01), n_probe=4)

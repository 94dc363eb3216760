"""Pins of the oracle's composed model (stack of blocks, text rows, head),
beyond the single-block pins: no GPU needed.

The stack has no positional encoding, so permuting the video tokens permutes
its outputs and permuting the text tokens leaves the video outputs alone;
with block 0's gates at zero the stack is block 1 alone, under block 1's own
modulation; the head has closed forms when its weight or its scale vanish.
A text/video row mix-up, a modulation taken from the wrong block or noise
level, or a head that ignores its modulation fails one of these.
"""
import numpy as np

import acid_inputs as ai
import oracle as O

CFG = ai.DiTConfig("toy-stack", n_blocks=3, hidden=32, n_heads=4, head_dim=8, ffn=64,
                   n_video=11, n_text=4, dtype="f32", n_steps=4)


def _model(p=None):
    return O.DiTModel(CFG, ai.weights(CFG, std=0.2) if p is None else p)


def _inputs(seed=0):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=(CFG.n_video, CFG.hidden)),
            rng.normal(size=(CFG.n_text, CFG.hidden)))


def test_video_permutation_equivariance_and_text_permutation_invariance():
    m = _model()
    x, text = _inputs(1)
    v, h = m.forward(x, 0.6, text)
    rng = np.random.default_rng(2)
    pv = rng.permutation(CFG.n_video)
    v2, h2 = m.forward(x[pv], 0.6, text)
    np.testing.assert_allclose(v2, v[pv], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(h2, h[pv], rtol=1e-11, atol=1e-12)
    pt = rng.permutation(CFG.n_text)
    v3, _ = m.forward(x, 0.6, text[pt])
    np.testing.assert_allclose(v3, v, rtol=1e-11, atol=1e-12)
    # the text rows do take part (as keys and values of every block); a
    # constant shift of a row would not show it (LayerNorm removes it)
    v4, _ = m.forward(x, 0.6, rng.normal(size=text.shape))
    assert np.abs(v4 - v).max() > 1e-3


def test_each_block_uses_its_own_modulation():
    p = ai.weights(CFG, std=0.2)
    H = CFG.hidden
    for b in (0, 2):  # blocks 0 and 2 become the identity (gates 1 and 2 at zero)
        for lo, hi in ((2 * H, 3 * H), (5 * H, 6 * H)):
            p[f"blocks.{b}.ada.w"][:, lo:hi] = 0
            p[f"blocks.{b}.ada.b"][lo:hi] = 0
    m = O.DiTModel(CFG, p)
    x, text = _inputs(3)
    sigma = 0.35
    mod = m.modulation(sigma)["blocks"]
    h_in = np.concatenate([text, x])
    want = m.block(h_in, 1, mod[1])[CFG.n_text:]
    np.testing.assert_allclose(m.stack(x, sigma, text), want, rtol=1e-12, atol=1e-13)
    # the pin discriminates: block 1 under another block's or level's modulation differs
    assert np.abs(m.block(h_in, 1, mod[0])[CFG.n_text:] - want).max() > 1e-3
    other = m.modulation(0.9)["blocks"][1]
    assert np.abs(m.block(h_in, 1, other)[CFG.n_text:] - want).max() > 1e-3


def test_head_closed_forms():
    H = CFG.hidden
    x, text = _inputs(4)
    p = ai.weights(CFG, std=0.2)
    p["head.w"] = np.zeros_like(p["head.w"])
    v, _ = _model(p).forward(x, 0.5, text)
    np.testing.assert_array_equal(v, np.tile(p["head.b"].astype(np.float64), (CFG.n_video, 1)))
    # scale = -1 (1 + scale = 0): every row becomes shift W + b
    p = ai.weights(CFG, std=0.2)
    p["head.ada.w"][:, H:2 * H] = 0
    p["head.ada.b"][H:2 * H] = -1.0
    m = _model(p)
    shift = m.modulation(0.5)["head"][0]
    v, _ = m.forward(x, 0.5, text)
    want = shift @ p["head.w"].astype(np.float64) + p["head.b"]
    np.testing.assert_allclose(v, np.tile(want, (CFG.n_video, 1)), rtol=1e-12, atol=1e-13)


def test_stack_without_text_equals_empty_text():
    m = _model()
    x, _ = _inputs(5)
    cfg0 = CFG.replace(n_text=0)
    m0 = O.DiTModel(cfg0, m.p)
    np.testing.assert_array_equal(m0.stack(x, 0.2), m0.stack(x, 0.2, np.zeros((0, CFG.hidden))))

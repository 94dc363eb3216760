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


# ------------------------------------------------ TEMNI (TeaCache's signal)
#
# Section 2, paragraph "TeaCache": the signal is formed from the noisy input
# after LayerNorm and the timestep-embedding modulation of the first block,
# i.e. block 0's first (shift, scale) pair.  With every adaLN weight at zero
# the modulation vectors are the adaLN biases, known here independently of
# the oracle's modulation code, and the LayerNorm is torch's.

def _temni_pin_case():
    H = CFG.hidden
    p = ai.weights(CFG, std=0.2)
    rng = np.random.default_rng(11)
    for b in range(CFG.n_blocks):
        p[f"blocks.{b}.ada.w"][:] = 0
        p[f"blocks.{b}.ada.b"][:] = rng.normal(scale=0.5, size=6 * H).astype(np.float32)
    x = rng.normal(size=(CFG.n_video, H)) * 3.0 + 1.5
    return p, x


def _temni_expected(p, x, block=0, shift_idx=0, scale_idx=1):
    import torch
    H = CFG.hidden
    mod = p[f"blocks.{block}.ada.b"].astype(np.float64).reshape(6, H)
    ln = torch.nn.functional.layer_norm(torch.from_numpy(x), (H,), eps=1e-6).numpy()
    return ln * (1.0 + mod[scale_idx]) + mod[shift_idx]


def _temni_pin_holds(model_cls) -> bool:
    p, x = _temni_pin_case()
    m = model_cls(CFG, p)
    want = _temni_expected(p, x)
    ok = True
    for sigma in (1.0, 0.45, 0.0):
        got = m.temni(x, sigma)
        ok &= got.shape == want.shape and np.allclose(got, want, rtol=1e-12, atol=1e-12)
    return bool(ok)


def test_temni_is_block0_first_modulation_of_layer_norm():
    assert _temni_pin_holds(O.DiTModel)
    # the pin separates TEMNI from its near misses: the second triple, the
    # pair swapped, another block's pair, the gate as shift, no LayerNorm
    p, x = _temni_pin_case()
    want = _temni_expected(p, x)
    for other in (_temni_expected(p, x, 0, 3, 4), _temni_expected(p, x, 0, 1, 0),
                  _temni_expected(p, x, 1), _temni_expected(p, x, 0, 2, 1)):
        assert np.abs(other - want).max() > 0.1
    mod = p["blocks.0.ada.b"].astype(np.float64).reshape(6, CFG.hidden)
    assert np.abs(x * (1 + mod[1]) + mod[0] - want).max() > 0.1


class _TemniSecondTriple(O.DiTModel):
    def temni(self, x, sigma):
        mod = self.modulation(sigma)["blocks"][0]
        return O.modulate(O.layer_norm(x), mod[3], mod[4])


class _TemniSwapped(O.DiTModel):
    def temni(self, x, sigma):
        mod = self.modulation(sigma)["blocks"][0]
        return O.modulate(O.layer_norm(x), mod[1], mod[0])


class _TemniBlock1(O.DiTModel):
    def temni(self, x, sigma):
        mod = self.modulation(sigma)["blocks"][1]
        return O.modulate(O.layer_norm(x), mod[0], mod[1])


class _TemniNoNorm(O.DiTModel):
    def temni(self, x, sigma):
        mod = self.modulation(sigma)["blocks"][0]
        return O.modulate(np.asarray(x, np.float64), mod[0], mod[1])


def test_temni_pin_rejects_planted_mistakes():
    """Each plausible mistake in the oracle's TEMNI, planted in a subclass on
    the CPU, fails the pin above."""
    for bad in (_TemniSecondTriple, _TemniSwapped, _TemniBlock1, _TemniNoNorm):
        assert not _temni_pin_holds(bad), bad.__name__

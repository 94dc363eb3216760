"""Pins of the oracle's parallel (single-stream) block against the pinned
sequential block (no GPU needed).

The parallel block feeds one modulated LayerNorm to both branches and adds
both projections through one gate.  Three reductions pin it: without MLP
weights it is the sequential block; without attention weights and with the
second modulation triple equal to the first it is the sequential block
again; and its two branches add.  A dropped branch, a wrong gate or shift
index, or a second LayerNorm between the branches fails one of them.
"""
import numpy as np

import acid_inputs as ai
import oracle as O

TOY_SEQ = ai.DiTConfig("toy", n_blocks=2, hidden=32, n_heads=4, head_dim=8, ffn=48,
                       n_video=13, n_text=3, dtype="f32", n_steps=6)
TOY_PAR = TOY_SEQ.replace(name="toy-parallel", block="parallel")

MLP = ("ffn1.w", "ffn1.b", "ffn2.w", "ffn2.b")


def _params(seed=0):
    return ai.weights(TOY_SEQ, seed=seed, std=0.2)


def _zero(p, names, b=0):
    p = dict(p)
    for n in names:
        p[f"blocks.{b}.{n}"] = np.zeros_like(p[f"blocks.{b}.{n}"])
    return p


def _h_mod(seed=3):
    rng = np.random.default_rng(seed)
    h = rng.normal(size=(TOY_SEQ.n_tokens, TOY_SEQ.hidden))
    mod6 = rng.normal(size=(6, TOY_SEQ.hidden)) * 0.5
    return h, mod6


def test_parallel_without_mlp_is_sequential():
    p = _zero(_params(), MLP)
    h, mod6 = _h_mod()
    seq = O.DiTModel(TOY_SEQ, p).block(h, 0, mod6)
    par = O.DiTModel(TOY_PAR, p).block(h, 0, mod6)
    np.testing.assert_allclose(par, seq, rtol=1e-12, atol=1e-13)
    # and the MLP branch is not silently dropped when it is present
    full = O.DiTModel(TOY_PAR, _params()).block(h, 0, mod6)
    assert np.abs(full - par).max() > 1e-3


def test_parallel_without_attention_is_sequential_with_tied_modulation():
    p = _zero(_params(), ("qkv.w", "qkv.b", "o.b"))
    h, mod6 = _h_mod(4)
    tied = np.concatenate([mod6[:3], mod6[:3]])
    seq = O.DiTModel(TOY_SEQ, p).block(h, 0, tied)
    par = O.DiTModel(TOY_PAR, p).block(h, 0, tied)
    np.testing.assert_allclose(par, seq, rtol=1e-12, atol=1e-13)
    # the second triple is unused by the parallel block
    par2 = O.DiTModel(TOY_PAR, p).block(h, 0, mod6)
    np.testing.assert_array_equal(par, par2)


def test_parallel_branches_add():
    p = _params(1)
    h, mod6 = _h_mod(5)
    full = O.DiTModel(TOY_PAR, p).block(h, 0, mod6)
    attn_only = O.DiTModel(TOY_PAR, _zero(p, MLP)).block(h, 0, mod6)
    mlp_only = O.DiTModel(TOY_PAR, _zero(p, ("o.w", "o.b"))).block(h, 0, mod6)
    np.testing.assert_allclose(full - h, (attn_only - h) + (mlp_only - h), rtol=1e-11, atol=1e-13)


def test_parallel_gate_zero_identity_rows_and_permutation():
    p = _params(2)
    H = TOY_PAR.hidden
    m = O.DiTModel(TOY_PAR, p)
    h, mod6 = _h_mod(6)
    g0 = mod6.copy()
    g0[2] = 0.0
    np.testing.assert_array_equal(m.block(h, 0, g0), h)
    out = m.block(h, 1, mod6)
    rows = np.array([0, 4, 9, 15])
    np.testing.assert_allclose(m.block(h, 1, mod6, rows=rows), out[rows], rtol=1e-13, atol=1e-14)
    perm = np.random.default_rng(7).permutation(TOY_PAR.n_tokens)
    np.testing.assert_allclose(m.block(h[perm], 1, mod6), out[perm], rtol=1e-11, atol=1e-12)
    # a stack of parallel blocks with every gate1 at zero is the identity
    for b in range(TOY_PAR.n_blocks):
        p[f"blocks.{b}.ada.w"][:, 2 * H:3 * H] = 0
        p[f"blocks.{b}.ada.b"][2 * H:3 * H] = 0
    x = ai.gaussian((TOY_PAR.n_video, H), 8)
    np.testing.assert_array_equal(O.DiTModel(TOY_PAR, p).stack(x, 0.4), x.astype(np.float64))

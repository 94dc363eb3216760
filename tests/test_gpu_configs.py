"""Parity of the whole ACID-gated loop at the three model shapes, run exactly
as the benchmark runs it (host gate, TeaCache's drift, tau_low 0.05,
tau_high 0.2, delta 0.01, seeded latents and text), and of one block at the
HunyuanVideo-slice shape in both block forms.

Per loop (Algorithm 1 around the Wan-2.1-1.3B, CogVideoX-5B and
HunyuanVideo-slice stacks):
* the gate fed the loop's own drift trace reproduces its decisions, its
  accumulated drift and its thresholds bit for bit;
* at sampled steps k, the drift s_k in the trace equals, within 1e-3, the
  oracle's relative L1 change between the TEMNI of x_{k-1} and of x_k, where
  x_{k-1} and x_k are the loop's own latents (taken from shorter runs of the
  same loop, checked to be bit-identical prefixes of the full run).
The loop's x_N is not compared with an oracle loop at these sizes (one
computed step of the Wan stack is 2.7e14 flops); the block and the drift are
the pieces the oracle computes one by one.
"""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import assert_close_to_scale, make_model, need_gpu, rel_err, to_dev, to_np

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

GATE = dict(tau_low=0.05, tau_high=0.2, delta=0.01)


@pytest.fixture(scope="module")
def P():
    return need_gpu()


def _temni_params(name: str) -> bool:
    """Host copies needed for the oracle's TEMNI: the timestep MLP, block 0's
    and the head's adaLN tensors."""
    return (name.startswith("temb.") or name.startswith("blocks.0.ada.")
            or name.startswith("head.ada."))


def _temni_oracle(cfg, params):
    # block 0's modulation does not depend on the later blocks
    return O.DiTModel(cfg.replace(n_blocks=1), params)


def _check_gate_replay(tr, gate):
    gp = O.GateParams(gate["tau_low"], gate["tau_high"], gate["delta"])
    dec, taus, sums = O.gate_schedule(list(tr["s"]), gp)
    assert list(tr["gate_compute"].astype(bool)) == dec
    assert np.all(tr["compute"] == tr["gate_compute"])
    assert np.array_equal(tr["sigma_sum_after"], np.asarray(sums, np.float64))
    assert np.array_equal(np.isnan(tr["tau_used"]), np.isnan(taus))
    ok = ~np.isnan(tr["tau_used"])
    assert np.array_equal(tr["tau_used"][ok], np.asarray(taus)[ok])


def _latents_at(m, x0, sig, text_d, k, tr_full, gate):
    """x_k of the loop: a k-step run of the same loop over sigma_0..sigma_k,
    whose trace must be the full run's first k entries, bit for bit."""
    if k == 0:
        return to_np(x0)
    x = x0.clone()
    tr = m.denoise_loop(x, sig[:k + 1], text_d, mode="acid", **gate)
    assert np.array_equal(tr["compute"], tr_full["compute"][:k])
    assert np.array_equal(tr["s"][1:], tr_full["s"][1:k])
    return to_np(x)


def _check_drift_steps(m, om, x0, sig, text_d, tr, steps, gate):
    for k in steps:
        x_prev = _latents_at(m, x0, sig, text_d, k - 1, tr, gate)
        x_k = _latents_at(m, x0, sig, text_d, k, tr, gate)
        s_ref = O.relative_l1_drift(om.temni(x_k, float(sig[k])),
                                    om.temni(x_prev, float(sig[k - 1])))
        assert abs(tr["s"][k] - s_ref) <= 1e-3 * s_ref, (k, tr["s"][k], s_ref)


def _sampled_steps(tr, n, last=True):
    """Step 1, the first step after a skipped step, and the last step."""
    steps = [1]
    after_skip = [k for k in range(2, n) if tr["compute"][k - 1] == 0]
    if after_skip:
        steps.append(after_skip[0])
    if last and n - 1 not in steps:
        steps.append(n - 1)
    return steps


def _run_loop_case(P, cfg, steps_last=True):
    m, params = make_model(P, cfg, max_steps=cfg.n_steps, keep=_temni_params)
    om = _temni_oracle(cfg, params)
    x0 = torch.from_numpy(ai.latents(cfg)).cuda()
    text = ai.text_tokens(cfg)
    text_d = torch.from_numpy(text).cuda() if text is not None else None
    sig = ai.sigmas(cfg.n_steps)
    x = x0.clone()
    tr = m.denoise_loop(x, sig, text_d, mode="acid", **GATE)
    _check_gate_replay(tr, GATE)
    assert math.isnan(tr["s"][0]) and np.all(np.isfinite(tr["s"][1:])) and np.all(tr["s"][1:] > 0)
    assert np.all(np.isfinite(to_np(x)))
    steps = _sampled_steps(tr, cfg.n_steps, steps_last)
    _check_drift_steps(m, om, x0, sig, text_d, tr, steps, GATE)
    return m, om, x0, text_d, sig, tr


def test_loop_wan_drift_along_the_loop_and_tau_low_switching(P):
    """The 30-block Wan-shape loop: drift values along the loop against the
    oracle, and a run whose delta lies inside the signal's step-to-step
    changes, so the gate switches between tau_low and tau_high."""
    m, om, x0, text_d, sig, tr = _run_loop_case(P, ai.WAN13B)
    ds = np.abs(np.diff(tr["s"][1:]))
    delta = float(np.median(ds))
    gate = dict(tau_low=0.05, tau_high=0.2, delta=delta)
    x = x0.clone()
    tr2 = m.denoise_loop(x, sig, text_d, mode="acid", **gate)
    _check_gate_replay(tr2, gate)
    taus = tr2["tau_used"][1:]
    assert np.any(taus == 0.05) and np.any(taus == 0.2), taus
    # the drift is a function of the trajectory: equal up to the first step
    # whose decision differs from the default run
    first = int(np.argmax(tr2["compute"] != tr["compute"])) if np.any(tr2["compute"] != tr["compute"]) else len(tr)
    assert np.array_equal(tr2["s"][1:first + 1], tr["s"][1:first + 1])
    _check_drift_steps(m, om, x0, sig, text_d, tr2, [k for k in _sampled_steps(tr2, len(tr2), False)
                                                      if k > first][:1], gate)


def test_loop_cogvideox_42_blocks(P):
    """The 42-block CogVideoX-5B-shape loop with 226 text tokens."""
    _run_loop_case(P, ai.COG5B)


def test_loop_hunyuan_slice(P):
    """The 4-block HunyuanVideo-slice loop (256 text + 118800 video tokens)."""
    _run_loop_case(P, ai.HUNYUAN, steps_last=False)


@pytest.mark.parametrize("block", ["sequential", "parallel"])
def test_block_hunyuan_shape_vs_oracle(P, block):
    """One block at the HunyuanVideo-slice shape (256 text + 118800 video
    tokens, 24 x 128 heads, H 3072, F 12288, bf16) in both block forms, on
    sampled text and video rows against the oracle's block with keys and
    values over all 119056 tokens."""
    cfg = ai.HUNYUAN.replace(n_blocks=1, n_steps=2, block=block)
    m, params = make_model(P, cfg, max_steps=2)
    om = O.DiTModel(cfg, params)
    H = cfg.hidden
    h0 = ai.gaussian((cfg.n_tokens, H), 29)
    mod6 = om.modulation(0.57)["blocks"][0].astype(np.float32)
    h = to_dev(h0)
    m.block_forward(0, to_dev(mod6), h)
    torch.cuda.synchronize()
    rng = np.random.default_rng(8)
    rows = np.unique(np.concatenate([rng.choice(cfg.n_text, 8, replace=False),
                                     cfg.n_text + rng.choice(cfg.n_video, 32, replace=False),
                                     [0, cfg.n_text - 1, cfg.n_text, cfg.n_tokens - 1]]))
    ref = om.block(h0, 0, mod6.astype(np.float64), rows=rows) - h0[rows]
    got = to_np(h[rows]) - h0[rows]
    assert rel_err(got, ref) < 2e-2
    assert_close_to_scale(got, ref, True, f"hunyuan {block} block")
    assert np.all(np.isfinite(to_np(h)))

"""The device-resident gate and the captured loop (HIP graph).

Algorithm 1 (Section 3.3) run by the device gate kernel is checked against
the hand-derived dyadic trace and, bit for bit, against the oracle's gate on
random sequences with ties, NaN and infinities.  The loop with the gate on
the device (every model kernel predicated on the step's decision word,
captured once and replayed) is checked bit for bit against the host-gated
loop, over several replays with other eager work and synchronisations in
between, after recaptures, under a forced schedule and without the cache,
and once directly against the oracle's loop; the same for EasyCache's and
DiCache's signals under the device gate.
"""
import math
import os

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import make_model, need_gpu, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TINY_TEXT = ai.TINY.replace(name="tiny-text", n_text=9, n_video=131)
SMALL_BF16 = ai.DiTConfig("small-bf16-ragged", n_blocks=2, hidden=256, n_heads=2, head_dim=128,
                          ffn=640, n_video=300, n_text=7, dtype="bf16", n_steps=8)
SMALL_BF16_D64 = SMALL_BF16.replace(name="small-bf16-d64", n_heads=4, head_dim=64, n_text=0,
                                    n_video=257, n_steps=12)


@pytest.fixture(scope="module")
def P():
    return need_gpu()


def _same(a, b) -> bool:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return a.shape == b.shape and bool(np.all((a == b) | (np.isnan(a) & np.isnan(b))))


def _same_trace(t1, t2) -> bool:
    return (np.array_equal(t1["compute"], t2["compute"])
            and np.array_equal(t1["gate_compute"], t2["gate_compute"])
            and _same(t1["s"], t2["s"]) and _same(t1["sigma_sum_after"], t2["sigma_sum_after"])
            and _same(t1["tau_used"], t2["tau_used"]))


# ------------------------------------------------------------ device gate


def _load_dyadic():
    rows = []
    with open(os.path.join(GOLDEN, "gate_dyadic_trace.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            st, s, _add, tau, dec, after = line.split()
            rows.append((int(st), float(s), float(tau), dec == "C", float(after)))
    return rows


def test_device_gate_dyadic_trace(P):
    rows = _load_dyadic()
    tr = P.gate_device_sequence([r[1] for r in rows], 0.0625, 0.25, 0.015625, n_warmup=1)
    assert list(tr["compute"].astype(bool)) == [r[3] for r in rows]
    assert _same(tr["tau_used"], [r[2] for r in rows])
    assert _same(tr["sigma_sum_after"], [r[4] for r in rows])
    assert np.array_equal(tr["compute"], tr["gate_compute"])


def test_device_gate_empty_sequence(P):
    assert len(P.gate_device_sequence([], 0.05, 0.2, 0.01)) == 0


def test_device_gate_bit_exact_vs_oracle(P):
    """Random sequences (exact repeats and deltas on the boundary, NaN and
    inf signals, every warmup length, degenerate thresholds): decisions,
    thresholds and accumulators identical to the oracle's gate."""
    rng = np.random.default_rng(7)
    for k in range(300):
        n = int(rng.integers(1, 40))
        s = np.abs(rng.normal(0.04, 0.03, n))
        if k % 3 == 0:
            s = np.round(s * 64) / 64
        if k % 11 == 0:
            s[rng.integers(0, n)] = math.nan
        if k % 13 == 0:
            s[rng.integers(0, n)] = math.inf
        p = O.GateParams(float(rng.choice([0.0, 0.05, 0.1, 0.0625])),
                         float(rng.choice([0.1, 0.2, 0.25, math.inf])),
                         float(rng.choice([-1.0, 0.0, 0.01, 0.015625, math.inf])),
                         int(rng.integers(0, 3)))
        dec, taus, sums = O.gate_schedule(list(s), p)
        tr = P.gate_device_sequence(s, p.tau_low, p.tau_high, p.delta, p.n_warmup)
        assert list(tr["compute"].astype(bool)) == dec, (k, list(s), p)
        assert _same(tr["tau_used"], taus), k
        assert _same(tr["sigma_sum_after"], sums), k
        assert _same(tr["s"], s), k


# ------------------------------------------------------------ captured loop


def _loop_case(P, cfg):
    m, params = make_model(P, cfg, max_steps=cfg.n_steps)
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    td = to_dev(text) if text is not None else None
    return m, params, x0, td, ai.sigmas(cfg.n_steps)


GATES = {ai.TINY.name: (0.05, 0.2, 0.01), "tiny-text": (0.02, 0.06, 0.01),
         "small-bf16-ragged": (0.01, 0.04, 0.005), "small-bf16-d64": (0.01, 0.04, 0.005)}


@pytest.mark.parametrize("cfg", [ai.TINY, TINY_TEXT, SMALL_BF16, SMALL_BF16_D64],
                         ids=lambda c: c.name)
def test_graph_loop_bit_exact_vs_host_gate(P, cfg):
    m, _, x0, td, sig = _loop_case(P, cfg)
    lo, hi, de = GATES[cfg.name]
    xe = to_dev(x0)
    tre = m.denoise_loop(xe, sig, td, mode="acid", tau_low=lo, tau_high=hi, delta=de)
    assert 0 < tre["compute"].sum() < cfg.n_steps  # both branches exercised
    x0d = to_dev(x0)
    xg = to_dev(x0)
    scratch = to_dev(x0)
    for rep in range(4):
        if rep:
            # other eager work on the same model and stream between replays
            m.denoise_loop(scratch, sig, td, mode="acid", tau_low=hi, tau_high=hi, delta=de)
            torch.cuda.synchronize()
            xg.copy_(x0d)
        trg = m.denoise_loop(xg, sig, td, mode="acid", tau_low=lo, tau_high=hi, delta=de,
                             graph=True)
        torch.cuda.synchronize()
        assert _same_trace(trg, tre), rep
        assert torch.equal(xg, xe), rep


def test_graph_loop_recapture_forced_and_nocache(P):
    cfg = SMALL_BF16
    m, _, x0, td, sig = _loop_case(P, cfg)
    x0d = to_dev(x0)

    def both(**kw):
        xe = x0d.clone()
        tre = m.denoise_loop(xe, sig, td, **kw)
        xg = x0d.clone()
        trg = m.denoise_loop(xg, sig, td, graph=True, **kw)
        torch.cuda.synchronize()
        assert _same_trace(trg, tre), kw
        assert torch.equal(xg, xe), kw
        return tre

    a = dict(mode="acid", tau_low=0.01, tau_high=0.04, delta=0.005)
    b = dict(mode="acid", tau_low=0.03, tau_high=0.03, delta=0.005)
    ta = both(**a)
    tb = both(**b)
    assert not np.array_equal(ta["compute"], tb["compute"])
    both(**a)  # parameters changed back: captured anew, same result
    forced = np.zeros(cfg.n_steps, np.uint8)
    forced[::3] = 1
    tf = both(**a, forced_schedule=forced)
    assert np.array_equal(tf["compute"], forced)
    tn = both(mode="nocache")
    assert tn["compute"].all() and np.isnan(tn["s"]).all()
    # tau = 0 computes every step: the same x_N as the uncached loop
    x_acid0 = x0d.clone()
    m.denoise_loop(x_acid0, sig, td, mode="acid", tau_low=0.0, tau_high=0.0, delta=0.005,
                   graph=True, trace=False)
    x_nc = x0d.clone()
    m.denoise_loop(x_nc, sig, td, mode="nocache", graph=True, trace=False)
    torch.cuda.synchronize()
    assert torch.equal(x_acid0, x_nc)


def test_graph_loop_other_sigmas_and_buffers(P):
    """A new x buffer or a new noise schedule captures anew."""
    cfg = ai.TINY
    m, _, x0, td, sig = _loop_case(P, cfg)
    sig2 = np.linspace(1.0, 0.0, cfg.n_steps + 1, dtype=np.float32) ** 2
    for s_ in (sig, sig2, sig):
        for _ in range(2):
            xe = to_dev(x0)
            tre = m.denoise_loop(xe, s_, td, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01)
            xg = to_dev(x0)  # a fresh buffer each time
            trg = m.denoise_loop(xg, s_, td, mode="acid", tau_low=0.05, tau_high=0.2,
                                 delta=0.01, graph=True)
            assert _same_trace(trg, tre)
            assert torch.equal(xg, xe)


def test_graph_loop_vs_oracle(P):
    """The captured loop's x_N and schedule against the oracle's loop."""
    cfg = ai.TINY
    m, params, x0, td, sig = _loop_case(P, cfg)
    om = O.DiTModel(cfg, params)
    x = to_dev(x0)
    tr = m.denoise_loop(x, sig, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01, graph=True)
    xr, otr = O.denoise_loop(om, x0, sig, mode="acid", gate=O.GateParams(0.05, 0.2, 0.01),
                             forced_schedule=tr["compute"])
    ok = ~np.isnan(otr["s"])
    np.testing.assert_allclose(tr["s"][ok], otr["s"][ok], rtol=1e-3)
    dec, _, _ = O.gate_schedule(list(tr["s"]), O.GateParams(0.05, 0.2, 0.01))
    assert list(tr["gate_compute"].astype(bool)) == dec
    assert rel_err(to_np(x), xr) < 1e-4


TINY3 = ai.TINY.replace(name="tiny3", n_blocks=3)


def _signal_scale(m, x0, sig, td, mode):
    """Median finite signal of an all-compute run (the thresholds' scale)."""
    tr = m.denoise_loop(to_dev(x0), sig, td, mode=mode, tau_low=0.0, tau_high=0.0, delta=0.0)
    s = tr["s"][np.isfinite(tr["s"])]
    return float(np.median(s))


@pytest.mark.parametrize("cfg,mode,probe", [(ai.TINY, "easycache", 0), (SMALL_BF16, "easycache", 0),
                                            (TINY3, "dicache", 1), (TINY3, "dicache", 2),
                                            (SMALL_BF16, "dicache", 1)],
                         ids=["tiny-easycache", "bf16-easycache", "tiny3-dicache1",
                              "tiny3-dicache2", "bf16-dicache1"])
def test_graph_loop_other_signals_bit_exact(P, cfg, mode, probe):
    """EasyCache's and DiCache's signals under the device gate: the captured
    loop equals the host-gated loop bit for bit (x_N and trace), replayed
    with other eager work between replays."""
    m, _, x0, td, sig = _loop_case(P, cfg)
    if mode == "dicache":
        m.set_probe_blocks(probe)
    sc = _signal_scale(m, x0, sig, td, mode)
    if mode == "easycache":
        gate = dict(tau_low=1.5 * sc, tau_high=3.0 * sc, delta=0.05 * sc)
    else:
        gate = dict(tau_low=1.2 * sc, tau_high=2.5 * sc, delta=0.05 * sc)
    xe = to_dev(x0)
    tre = m.denoise_loop(xe, sig, td, mode=mode, **gate)
    assert 0 < tre["compute"].sum() < cfg.n_steps
    x0d = to_dev(x0)
    xg = to_dev(x0)
    for rep in range(3):
        if rep:
            m.denoise_loop(to_dev(x0), sig, td, mode="acid", tau_low=0.05, tau_high=0.2, delta=0.01)
            torch.cuda.synchronize()
            xg.copy_(x0d)
        trg = m.denoise_loop(xg, sig, td, mode=mode, **gate, graph=True)
        torch.cuda.synchronize()
        assert _same_trace(trg, tre), rep
        assert torch.equal(xg, xe), rep
    # a forced schedule through the captured loop
    forced = np.zeros(cfg.n_steps, np.uint8)
    forced[:2] = 1
    forced[4::3] = 1
    xf, xfg = to_dev(x0), to_dev(x0)
    trf = m.denoise_loop(xf, sig, td, mode=mode, **gate, forced_schedule=forced)
    trfg = m.denoise_loop(xfg, sig, td, mode=mode, **gate, forced_schedule=forced, graph=True)
    torch.cuda.synchronize()
    assert np.array_equal(trfg["compute"], forced) and _same_trace(trfg, trf)
    assert torch.equal(xfg, xf)

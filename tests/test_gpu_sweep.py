"""The gate sweep (the synthetic counterpart of the paper's threshold and
Pareto study, Section 4, Figures 6-8) through the benchmark's own sweep code
on the small bf16 workload (4 blocks, H 1024, 1024 tokens, 30 steps): the
no-cache reference, a fixed threshold, an ACID pair with delta inside the
signal's step-to-step changes, and the fixed threshold again as ACID with
tau_low == tau_high and another delta."""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import bench
import oracle as O
from gpu_util import make_model, need_gpu, to_np
from test_oracle import _fixed_skeleton

pytestmark = pytest.mark.gpu


def test_sweep_small_bf16_through_bench_code():
    P = need_gpu()
    cfg = ai.SMALL
    m, _ = make_model(P, cfg)
    x0 = torch.from_numpy(ai.latents(cfg)).cuda()
    sig = ai.sigmas(cfg.n_steps)
    grid = [("fixed", 0.1, 0.1, 0.01), ("acid", 0.05, 0.2, 0.001), ("acid", 0.1, 0.1, 0.5)]
    outs = []
    runs = bench.sweep(m, cfg, x0, None, sig, grid, outputs=outs)
    assert len(runs) == 1 + len(grid) and len(outs) == len(runs)
    assert runs[0]["trace"]["compute"].all() and runs[0]["psnr_db"] == math.inf
    ref = to_np(outs[0])
    for run, x in zip(runs[1:], outs[1:]):
        tr = run["trace"]
        gp = O.GateParams(run["tau_low"], run["tau_high"], run["delta"])
        dec, _, _ = O.gate_schedule(list(tr["s"]), gp)
        assert list(tr["gate_compute"].astype(bool)) == dec
        assert np.all(tr["compute"] == tr["gate_compute"])
        assert run["computed_steps"] == int(tr["compute"].sum()) < cfg.n_steps
        assert run["schedule"] == "".join("C" if c else "S" for c in tr["compute"])
        # the reported PSNR is the oracle's on the same two tensors
        assert run["psnr_db"] == pytest.approx(O.psnr(to_np(x), ref), rel=1e-9, abs=0)
        assert math.isfinite(run["psnr_db"])
    # a fixed threshold is ACID with tau_low == tau_high whatever delta is:
    # the same bits, and the single-threshold rule of Section 2 on its drifts
    assert torch.equal(outs[1], outs[3])
    t1, t3 = runs[1]["trace"], runs[3]["trace"]
    assert np.array_equal(t1["compute"], t3["compute"])
    assert np.array_equal(t1["sigma_sum_after"], t3["sigma_sum_after"])
    assert np.array_equal(t1["s"], t3["s"], equal_nan=True)
    assert list(runs[1]["trace"]["compute"].astype(bool)) == _fixed_skeleton(
        list(runs[1]["trace"]["s"]), 0.1)
    # the ACID point switches between its thresholds
    assert runs[2]["steps_tau_low"] > 0 and runs[2]["steps_tau_high"] > 0
    assert runs[2]["steps_tau_low"] + runs[2]["steps_tau_high"] == cfg.n_steps - 1

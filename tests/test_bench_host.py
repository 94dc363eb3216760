"""Host logic of the benchmark (no GPU): the sweep's PSNR against the
oracle's, the sweep grid, the single-GPU guard and the per-class work
figures the rates are computed from."""
import math
import subprocess
import sys

import numpy as np
import pytest
import torch

import acid_inputs as ai
import bench
import oracle as O


def test_psnr_equals_oracle_psnr():
    rng = np.random.default_rng(3)
    ref = rng.normal(size=(64, 32))
    for scale in (1e-3, 0.1, 1.0):
        x = ref + scale * rng.normal(size=ref.shape)
        got = bench.psnr(torch.from_numpy(x), torch.from_numpy(ref))
        assert got == pytest.approx(O.psnr(x, ref), rel=1e-12)
    assert bench.psnr(torch.from_numpy(ref), torch.from_numpy(ref)) == math.inf == O.psnr(ref, ref)


def test_sweep_grid():
    g = bench.sweep_grid("0.05,0.2", "0.05:0.2,0.1:0.3", "0.001,0.01", 0.01)
    assert g == [("fixed", 0.05, 0.05, 0.01), ("fixed", 0.2, 0.2, 0.01),
                 ("acid", 0.05, 0.2, 0.001), ("acid", 0.05, 0.2, 0.01),
                 ("acid", 0.1, 0.3, 0.001), ("acid", 0.1, 0.3, 0.01)]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_work_per_class_wan():
    cfg = ai.WAN13B
    w = bench.work_per_class(cfg, 10, 50)
    L, H, F = cfg.n_tokens, cfg.hidden, cfg.ffn
    assert w["attention"] == ("flop", 10 * 30 * 4.0 * L * L * H)
    gemm = sum(v for k, (_, v) in w.items() if k.startswith("gemm_") and k != "gemm_head")
    assert gemm == pytest.approx(10 * 30 * 2.0 * L * (4 * H * H + 2 * H * F))
    assert w["cache"] == ("byte", 50 * 12.0 * cfg.n_video * H)

"""Pins of the oracle's EasyCache loop (signal of Section 2, paragraph
"EasyCache", under the gate of Algorithm 1): a hand-derived dyadic trace, the
Euler identity s_i = k |sigma_i - sigma_{i-1}|, and the tau = 0 / tau = inf
limits against the no-cache loop and a direct recurrence."""
import math
import os

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "easycache_scalar_trace.txt")


def _golden_rows():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip() or line.startswith("D "):
            continue
        run, lo, hi, sched, s2, s3, sum3, t2, t3, x4 = line.split()
        rows.append((run, float(lo), float(hi), sched, float(s2), float(s3), float(sum3),
                     float(t2), float(t3), float(x4)))
    return rows


@pytest.mark.parametrize("row", _golden_rows(), ids=lambda r: r[0])
def test_easycache_scalar_trace(row):
    _, lo, hi, sched, s2, s3, sum3, t2, t3, x4 = row
    sig = np.array([1.0, 0.75, 0.5, 0.25, 0.0])
    x, tr = O.easycache_loop(lambda x, s: 2.0 * x, np.array([1.0]), sig,
                             gate=O.GateParams(lo, hi, 0.01, n_warmup=2))
    assert "".join("C" if c else "S" for c in tr["compute"]) == sched
    assert math.isnan(tr["s"][0]) and math.isnan(tr["s"][1])
    assert tr["s"][2] == s2 and tr["s"][3] == s3
    assert tr["sigma_sum_after"][3] == sum3
    assert tr["tau_used"][2] == t2 and tr["tau_used"][3] == t3
    assert x[0] == x4


def test_easycache_rate_after_skipped_step():
    """Run D: k recomputed on a computed step that follows a skipped one uses
    the reused output of the skipped step as v_{i-1}."""
    line = [l for l in open(GOLDEN) if l.startswith("D ")][0].split()
    sched, s2, s3 = line[1], float(line[2]), float(line[3])
    n4, d4 = (int(v) for v in line[4].split("/"))
    n5, d5 = (int(v) for v in line[5].split("/"))
    sig = 1.0 - np.arange(6) / 8.0
    x, tr = O.easycache_loop(lambda x, s: 2.0 * x, np.array([1.0]), sig,
                             gate=O.GateParams(0.3, 0.3, 0.01, n_warmup=2))
    assert "".join("C" if c else "S" for c in tr["compute"]) == sched
    assert tr["s"][2] == s2 and tr["s"][3] == s3
    assert tr["s"][4] == pytest.approx(n4 / d4, rel=1e-15)
    assert x[0] == n5 / d5


def _model(seed=0, n=48):
    rng = np.random.default_rng(seed)
    a = rng.normal(size=(n, n)) / math.sqrt(n)
    b = rng.normal(size=n) * 0.1
    return lambda x, s: np.tanh(x @ a) * (1.0 + s) + b


def test_easycache_euler_identity_and_tau_inf_recurrence():
    """tau = inf: after the two warmup steps k stays the rate of step 1, and
    s_i = k |sigma_i - sigma_{i-1}| (x_i - x_{i-1} = dsigma v_{i-1}); x_N equals
    the direct recurrence x <- x + dsigma (x + D)."""
    f = _model()
    x0 = np.random.default_rng(1).normal(size=48)
    sig = (1.0 - np.arange(13) / 12.0) ** 2          # non-uniform steps
    x, tr = O.easycache_loop(f, x0, sig, gate=O.GateParams(math.inf, math.inf, 0.01, n_warmup=2))
    assert list(tr["compute"]) == [1, 1] + [0] * 10
    v0 = f(x0, sig[0])
    x1 = x0 + (sig[1] - sig[0]) * v0
    v1 = f(x1, sig[1])
    k = np.abs(v1 - v0).sum() / np.abs(x1 - x0).sum()
    for i in range(2, 12):
        assert tr["s"][i] == pytest.approx(k * abs(sig[i] - sig[i - 1]), rel=1e-12)
    d = v1 - x1
    xr = x1 + (sig[2] - sig[1]) * v1
    for i in range(2, 12):
        xr = xr + (sig[i + 1] - sig[i]) * (xr + d)
    np.testing.assert_allclose(x, xr, rtol=1e-12, atol=1e-14)


def test_easycache_tau_zero_is_nocache():
    f = _model(3)
    x0 = np.random.default_rng(4).normal(size=48)
    sig = 1.0 - np.arange(11) / 10.0
    xn, trn = O.easycache_loop(f, x0, sig, mode="nocache")
    x0c, tr0 = O.easycache_loop(f, x0, sig, gate=O.GateParams(0.0, 0.0, 0.01, n_warmup=2))
    assert tr0["compute"].all() and trn["compute"].all() and np.isnan(trn["s"]).all()
    np.testing.assert_array_equal(xn, x0c)
    # a forced all-compute schedule is the no-cache loop too
    xf, _ = O.easycache_loop(f, x0, sig, gate=O.GateParams(1e9, 1e9, 0.01, n_warmup=2),
                             forced_schedule=np.ones(10, np.uint8))
    np.testing.assert_array_equal(xn, xf)


def test_easycache_rejects_short_warmup():
    with pytest.raises(ValueError):
        O.easycache_loop(lambda x, s: x, np.ones(2), np.array([1.0, 0.5, 0.0]),
                         gate=O.GateParams(0.1, 0.2, 0.01, n_warmup=1))

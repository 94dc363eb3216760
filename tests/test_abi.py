"""The C-ABI library on the host (no GPU needed): it loads, exports every
symbol include/acid.h declares, and its pure host logic (configuration
checks, manifest shapes, sizes, the gate) behaves as specified."""
import ctypes as C
import math

import numpy as np
import pytest

import acid_inputs as ai
import oracle as O
from paper_2607_12358_amd import _lib as L


@pytest.fixture(scope="module")
def lib():
    return L.lib()


def test_exports_every_declared_symbol(lib):
    names = L.header_symbols()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    for n in ("acid_dit_step", "acid_drift_signal", "acid_gate", "acid_cache_apply",
              "acid_denoise_loop"):
        assert n in names


def test_version(lib):
    assert b"gfx950" in lib.acid_version()


@pytest.mark.parametrize("cfg", list(ai.CONFIGS.values()), ids=list(ai.CONFIGS))
def test_workload_configs_accepted_and_manifest_matches(lib, cfg):
    c = L.config_c(cfg)
    assert lib.acid_config_check(C.byref(c)) == 0, L.last_error()
    man = ai.manifest(cfg)
    assert lib.acid_tensor_count(C.byref(c)) == len(man)
    for tid, (name, shape) in enumerate(man):
        rank = C.c_int32()
        dims = (C.c_int64 * 2)()
        assert lib.acid_tensor_shape(C.byref(c), tid, C.byref(rank), dims) == 0
        assert tuple(dims[:rank.value]) == shape, name
    wb = lib.acid_weights_bytes(C.byref(c))
    nparam = sum(int(np.prod(s)) for _, s in man)
    assert nparam * 2 <= wb <= nparam * 4 + 256 * len(man)
    assert lib.acid_workspace_bytes(C.byref(c), cfg.n_steps) > cfg.n_tokens * cfg.hidden * 4


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, L.ACID_ERR_SHAPE), ("hidden", 1000, L.ACID_ERR_SHAPE),
    ("ffn", 1000, L.ACID_ERR_SHAPE), ("n_blocks", 0, L.ACID_ERR_INVALID_ARG),
    ("freq_dim", 7, L.ACID_ERR_SHAPE), ("dtype", 5, L.ACID_ERR_INVALID_ARG),
    ("n_video", 1 << 26, L.ACID_ERR_SHAPE), ("ffn", 1 << 22, L.ACID_ERR_SHAPE)])
def test_config_errors(lib, field, value, status):
    c = L.config_c(ai.TINY)
    setattr(c, field, value)
    assert lib.acid_config_check(C.byref(c)) == status
    assert L.last_error()
    assert lib.acid_weights_bytes(C.byref(c)) == 0


def test_null_arguments_rejected(lib):
    assert lib.acid_config_check(None) == L.ACID_ERR_INVALID_ARG
    st = L.GateStateC()
    assert lib.acid_gate(C.byref(st), None, 0.0, None, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_cache_apply(7, None, None, None, 4, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_cache_apply(0, None, None, None, 0, None) == 0  # empty is a no-op


def test_prescaled_q_flags_checked(lib):
    """q_prescaled / q_prescale take 0 or 1; checked before any GPU work."""
    assert lib.acid_attention(L.ACID_BF16, 2, 0, 128, None, None, None, 0, None, 2,
                              None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_attention(L.ACID_BF16, 2, 0, 128, None, None, None, 0, None, 1, None) == 0
    e = L.EpilogueArgsC()
    e.kind = L.ACID_EPI_QKV
    e.q_prescale = 2
    assert lib.acid_linear(L.ACID_BF16, 0, 384, 128, None, None, C.byref(e),
                           None) == L.ACID_ERR_INVALID_ARG
    e.q_prescale = 1
    assert lib.acid_linear(L.ACID_BF16, 0, 384, 128, None, None, C.byref(e), None) == 0


def test_kernel_size_limits_checked(lib):
    """Sizes beyond the kernels' 32-bit offsets and grid limits are refused
    before any GPU work (the pointers are never looked at)."""
    def attn(dtype, nh, L_, d):
        ld = (L_ + 7) // 8 * 8
        return lib.acid_attention(dtype, nh, L_, d, None, None, None, ld, None, 0, None)
    assert attn(L.ACID_BF16, 1, 9_000_000, 128) == L.ACID_ERR_SHAPE    # 2 d vt_ld >= 2^31
    assert attn(L.ACID_BF16, 1, 9_000_000, 64) == L.ACID_ERR_INVALID_ARG  # within: NULL check
    assert attn(L.ACID_F32, 64, 2_000_000, 64) == L.ACID_ERR_SHAPE     # L n_heads >= 2^26
    assert attn(L.ACID_F32, 32, 2_000_000, 64) == L.ACID_ERR_INVALID_ARG
    e = L.EpilogueArgsC()
    e.kind = L.ACID_EPI_BIAS
    for M, N, K, st in [(1 << 20, 1 << 23, 128, L.ACID_ERR_SHAPE), (8, 128, 1 << 23, L.ACID_ERR_SHAPE),
                        ((1 << 30) + 1, 128, 128, L.ACID_ERR_SHAPE),
                        (1 << 24, 1 << 17, 128, L.ACID_ERR_SHAPE),
                        (1 << 22, 1 << 16, 128, L.ACID_ERR_INVALID_ARG)]:
        assert lib.acid_linear(L.ACID_BF16, M, N, K, None, None, C.byref(e), None) == st, (M, N, K)


def test_device_gate_and_graph_loop_argument_errors(lib):
    """Argument checks that return before any GPU work."""
    pc = L.GateParamsC(0.05, 0.2, 0.01, 1)
    assert lib.acid_gate_device_sequence(None, None, 0, None, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_gate_device_sequence(C.byref(pc), None, 3, None, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_gate_device_sequence(C.byref(pc), None, -1, None, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_gate_device_sequence(C.byref(pc), None, 0, None, None) == 0  # empty: no-op
    sig = (C.c_float * 3)(1.0, 0.5, 0.0)
    assert lib.acid_denoise_loop_graph(None, None, sig, 2, None, 1, C.byref(pc), None, None,
                                       None) == L.ACID_ERR_INVALID_ARG


def _c_gate_run(lib, s_seq, p):
    st = L.GateStateC()
    pc = L.GateParamsC(p.tau_low, p.tau_high, p.delta, p.n_warmup)
    dec, taus, sums = [], [], []
    comp, tau = C.c_int32(), C.c_double()
    for s in s_seq:
        assert lib.acid_gate(C.byref(st), C.byref(pc), float(s), C.byref(comp), C.byref(tau)) == 0
        dec.append(bool(comp.value))
        taus.append(tau.value)
        sums.append(st.sigma_sum)
    return dec, taus, sums


def _same(a, b):
    return all((x == y) or (math.isnan(x) and math.isnan(y)) for x, y in zip(a, b))


def test_c_gate_dyadic_trace(lib):
    s = [0.0, 0.03125, 0.03125, 0.0625, 0.078125, 0.078125, 0.09375, 0.09375, 0.0625, 0.125]
    dec, _, sums = _c_gate_run(lib, s, O.GateParams(0.0625, 0.25, 0.015625, 1))
    assert "".join("C" if d else "S" for d in dec) == "CSSCSSSCSC"
    assert sums[6] == 0.25


def test_c_gate_bit_exact_vs_oracle(lib):
    """10^4 random sequences (with near-ties and NaN/inf) give identical
    decisions, thresholds and accumulators in the C gate and the oracle."""
    rng = np.random.default_rng(42)
    for k in range(10000):
        n = int(rng.integers(1, 40))
        s = np.abs(rng.normal(0.04, 0.03, n))
        if k % 7 == 0:  # exact repeats and deltas on the boundary
            s = np.round(s * 64) / 64
        if k % 97 == 0:
            s[rng.integers(0, n)] = math.nan
        if k % 89 == 0:
            s[rng.integers(0, n)] = math.inf
        p = O.GateParams(float(rng.choice([0.0, 0.05, 0.1, 0.0625])),
                         float(rng.choice([0.1, 0.2, 0.25, math.inf])),
                         float(rng.choice([-1.0, 0.0, 0.01, 0.015625, math.inf])),
                         int(rng.integers(0, 3)))
        d1, t1, s1 = O.gate_schedule(list(s), p)
        d2, t2, s2 = _c_gate_run(lib, list(s), p)
        assert d1 == d2, (k, list(s), p)
        assert _same(t1, t2) and _same(s1, s2), k


def test_q_scale_is_the_documented_float(lib):
    """acid_q_scale(d) is the fp32 value 1.4426950408889634f / sqrtf(d) the
    header documents (log2(e)/sqrt(d) rounded to float)."""
    import numpy as np
    for d in (64, 128, 96, 1):
        want = np.float32(np.float32(1.4426950408889634) / np.sqrt(np.float32(d)))
        assert lib.acid_q_scale(d) == float(want)
        assert abs(float(want) - math.log2(math.e) / math.sqrt(d)) <= 2 ** -23 * float(want)
    assert lib.acid_q_scale(0) == 0.0


def test_noalloc_l1_argument_errors(lib):
    out = (C.c_double * 2)()
    assert lib.acid_l1_norms_noalloc(None, None, None, -1, out, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_l1_norms_noalloc(None, None, None, 4, out, None) == L.ACID_ERR_INVALID_ARG
    assert lib.acid_l1_norms_noalloc(None, None, None, 4, None, None) == L.ACID_ERR_INVALID_ARG
    # n == 0: empty sums without touching any buffer or the device
    out[0] = out[1] = 7.0
    assert lib.acid_l1_norms_noalloc(None, None, None, 0, out, None) == L.ACID_OK
    assert out[0] == 0.0 and out[1] == 0.0


def test_host_load_argument_errors(lib):
    assert lib.acid_model_load_tensor_host(None, 0, None, 0, None) == L.ACID_ERR_INVALID_ARG

"""GPU parity of the individual kernels, through the C ABI, against the oracle.

Sizes span several tiles plus ragged tails; bf16 inputs are compared with an
oracle fed the same bf16-rounded values.  Tolerances: fp32 kernels 1e-5
relative (Frobenius), bf16 attention/GEMM outputs 2e-2 (the bf16 bar) with
typical errors far below it.
"""
import math

import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O
from gpu_util import (BF16_U, assert_elementwise, attention_bound, bf16_values, make_model,
                      need_gpu, rel_err, to_dev, to_np)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    return need_gpu()


# ------------------------------------------------------------------ cache


@pytest.mark.parametrize("n", [0, 1, 3, 4, 1001, 4096 * 3 + 2, 32760 * 1536])
def test_cache_store_apply(P, n):
    x = torch.randn(n, device="cuda")
    h = torch.randn(n, device="cuda")
    r = torch.empty(n, device="cuda")
    P.cache_apply(P.ACID_CACHE_STORE, x, h, r)
    xs, hs = to_np(x), to_np(h)
    if n:
        idx = np.random.default_rng(n).integers(0, n, min(n, 100000))
        np.testing.assert_allclose(to_np(r)[idx], (hs - xs)[idx], rtol=1e-6, atol=1e-7)
    h2 = torch.empty(n, device="cuda")
    P.cache_apply(P.ACID_CACHE_APPLY, x, h2, r)
    if n:
        np.testing.assert_allclose(to_np(h2)[idx], hs[idx], rtol=1e-6, atol=1e-6)


# ------------------------------------------------------- LN + modulation


@pytest.mark.parametrize("rows,H", [(1, 256), (37, 1024), (300, 1536), (5, 3072), (0, 256),
                                    (64, 100), (33, 1000), (7, 2052), (3, 4)])
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_ln_modulate(P, rows, H, out):
    rng = np.random.default_rng(rows * 7 + H)
    x = rng.normal(size=(rows, H)).astype(np.float32) * 2 + 0.5
    shift = rng.normal(size=H).astype(np.float32) * 0.1
    scale = rng.normal(size=H).astype(np.float32) * 0.1
    dt = torch.bfloat16 if out == "bf16" else torch.float32
    o = torch.empty((rows, H), dtype=dt, device="cuda")
    P.ln_modulate(to_dev(x), to_dev(shift), to_dev(scale), o)
    torch.cuda.synchronize()
    if rows == 0:
        return
    ref = O.modulate(O.layer_norm(x), shift.astype(np.float64), scale.astype(np.float64))
    tol = 1e-5 if out == "f32" else 4e-3
    assert rel_err(to_np(o), ref) < tol
    if out == "bf16":  # each element is the bf16 rounding of a value within fp32 error
        assert np.max(np.abs(to_np(o) - ref) / (np.abs(ref) + 1e-3)) < 2 ** -7


# -------------------------------------------------------------- attention


def prescale_q(P, q, d, dtype):
    """Q as the model's QKV epilogue stores it for attention with
    q_prescaled: the float32 product with log2(e)/sqrt(d), rounded once to
    the storage type.  Returns the stored values and the Q they stand for
    (stored / factor, in float64), the input of the attention definition."""
    c = np.float32(P.q_scale(d))
    stored = (q.astype(np.float32) * c).astype(np.float32)
    if dtype == torch.bfloat16:
        stored = bf16_values(stored)
    return stored, stored.astype(np.float64) / np.float64(c)


def _attn_case(P, n_heads, L, d, dtype, std, seed, prescaled=False):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(n_heads, L, d)).astype(np.float32) * std
    k = rng.normal(size=(n_heads, L, d)).astype(np.float32) * std
    v = rng.normal(size=(n_heads, L, d)).astype(np.float32)
    if dtype == torch.bfloat16:
        q, k, v = bf16_values(q), bf16_values(k), bf16_values(v)
    q_dev = q
    if prescaled:
        q_dev, q = prescale_q(P, q, d, dtype)
    vt_ld = ((L + 7) // 8) * 8
    vt = np.zeros((n_heads, d, vt_ld), np.float32)
    vt[:, :, :L] = v.transpose(0, 2, 1)
    vt[:, :, L:] = np.nan  # padding must never reach the output
    o = torch.empty((L, n_heads * d), dtype=dtype, device="cuda")
    P.attention(to_dev(q_dev, dtype), to_dev(k, dtype), to_dev(vt, dtype), o, q_prescaled=prescaled)
    torch.cuda.synchronize()
    return q, k, v, to_np(o)


@pytest.mark.parametrize("prescaled", [False, True], ids=["plain-q", "prescaled-q"])
@pytest.mark.parametrize("L", [1, 63, 64, 65, 128, 130, 256, 300, 320, 1000])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("std", [1.0, 4.0])
def test_attention_bf16(P, L, d, std, prescaled):
    nh = 2
    q, k, v, o = _attn_case(P, nh, L, d, torch.bfloat16, std, seed=L * 131 + d + int(std),
                            prescaled=prescaled)
    assert np.all(np.isfinite(o))
    for j in range(nh):
        ref = O.attention(q[j], k[j], v[j])
        got = o[:, j * d:(j + 1) * d]
        e = rel_err(got, ref)
        assert e < 2e-2, (j, e)
        assert e < 1e-2  # typical bf16 P rounding error is ~3e-3
        # and element by element, within the bound the bf16 rounding of the
        # probabilities and of the output allows (a single wrong element,
        # row or lane column fails here even when the head's norm hides it)
        assert_elementwise(got, ref, attention_bound(q[j], k[j], v[j]), 1.05 * BF16_U,
                           f"L={L} d={d} head {j}")


@pytest.mark.parametrize("prescaled", [False, True], ids=["plain-q", "prescaled-q"])
@pytest.mark.parametrize("L", [1, 37, 128, 300])
@pytest.mark.parametrize("d", [64, 128])
def test_attention_f32(P, L, d, prescaled):
    nh = 3
    q, k, v, o = _attn_case(P, nh, L, d, torch.float32, 1.0, seed=L + d, prescaled=prescaled)
    for j in range(nh):
        ref = O.attention(q[j], k[j], v[j])
        assert rel_err(o[:, j * d:(j + 1) * d], ref) < 1e-5
        assert_elementwise(o[:, j * d:(j + 1) * d], ref, attention_bound(q[j], k[j], v[j], False),
                           3e-5, f"fp32 L={L} d={d} head {j}")


@pytest.mark.parametrize("prescaled", [False, True], ids=["plain-q", "prescaled-q"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("L", [300, 1000])
def test_attention_growing_and_spiking_scores(P, d, L, prescaled):
    """Scores that grow along the key axis (the reference max must move on
    later tiles, by far more than the lazy bound) and one key whose score
    dwarfs all others (a probability that would overflow without a rescale)."""
    rng = np.random.default_rng(L + d)
    nh = 2
    q = bf16_values(rng.normal(size=(nh, L, d)).astype(np.float32))
    k = rng.normal(size=(nh, L, d)).astype(np.float32)
    k *= (1.0 + 6.0 * np.arange(L) / L)[None, :, None]
    k[1, L // 2] = 40.0 * q[1].mean(0)
    k = bf16_values(k)
    v = bf16_values(rng.normal(size=(nh, L, d)).astype(np.float32))
    vt_ld = ((L + 7) // 8) * 8
    vt = np.zeros((nh, d, vt_ld), np.float32)
    vt[:, :, :L] = v.transpose(0, 2, 1)
    o = torch.empty((L, nh * d), dtype=torch.bfloat16, device="cuda")
    q_dev = q
    if prescaled:
        q_dev, q = prescale_q(P, q, d, torch.bfloat16)
    P.attention(to_dev(q_dev, torch.bfloat16), to_dev(k, torch.bfloat16), to_dev(vt, torch.bfloat16),
                o, q_prescaled=prescaled)
    got = to_np(o)
    assert np.all(np.isfinite(got))
    for j in range(nh):
        ref = O.attention(q[j], k[j], v[j])
        assert rel_err(got[:, j * d:(j + 1) * d], ref) < 1e-2
        assert_elementwise(got[:, j * d:(j + 1) * d], ref, attention_bound(q[j], k[j], v[j]),
                           1.05 * BF16_U, f"growing scores L={L} d={d} head {j}")


def test_attention_uniform_and_single_key(P):
    """Q = 0 gives the mean of V; L = 1 returns V (properties at any size)."""
    for L in (1, 777):
        nh, d = 1, 128
        v = np.random.default_rng(L).normal(size=(nh, L, d)).astype(np.float32)
        v = bf16_values(v)
        vt_ld = ((L + 7) // 8) * 8
        vt = np.zeros((nh, d, vt_ld), np.float32)
        vt[:, :, :L] = v.transpose(0, 2, 1)
        q = torch.zeros((nh, L, d), dtype=torch.bfloat16, device="cuda")
        k = to_dev(np.random.default_rng(1).normal(size=(nh, L, d)), torch.bfloat16)
        o = torch.empty((L, d), dtype=torch.bfloat16, device="cuda")
        P.attention(q, k, to_dev(vt, torch.bfloat16), o)
        np.testing.assert_allclose(to_np(o), np.tile(v[0].mean(0), (L, 1)), atol=2e-2)


# -------------------------------------------------------------------- GEMM

KINDS = ["bias", "gelu", "gate_residual", "qkv", "qkv_prescaled", "euler"]


def _linear_case(P, kind, M, N, K, dtype, seed):
    rng = np.random.default_rng(seed)
    a = rng.normal(size=(M, K)).astype(np.float32)
    w = rng.normal(size=(K, N)).astype(np.float32) / math.sqrt(K)
    b = rng.normal(size=N).astype(np.float32) * 0.1
    if dtype == torch.bfloat16:
        a, w = bf16_values(a), bf16_values(w)
    y = a.astype(np.float64) @ w.astype(np.float64) + b
    # bound of the fp32 accumulation (exact products, K fp32 additions) per
    # output, plus |b|: the element-wise check's absolute part
    acc_err = K * 2.0 ** -24 * (np.abs(a).astype(np.float64) @ np.abs(w).astype(np.float64)
                                + np.abs(b))
    ad, wtd, bd = to_dev(a, dtype), to_dev(w.T.copy(), dtype), to_dev(b)
    if kind == "bias":
        out = torch.empty((M, N), device="cuda")
        P.linear(ad, wtd, P.ACID_EPI_BIAS, bd, out=out)
        return [(to_np(out), y, 1e-5, acc_err)]
    if kind == "gelu":
        out = torch.empty((M, N), dtype=dtype, device="cuda")
        P.linear(ad, wtd, P.ACID_EPI_BIAS_GELU, bd, out=out)
        # GELU's slope is at most 1.13; its fp32 evaluation adds a few ulp
        return [(to_np(out), O.gelu_tanh(y), 1e-5 if dtype == torch.float32 else 4e-3,
                 1.13 * acc_err + 1e-6)]
    if kind == "gate_residual":
        h0 = rng.normal(size=(M, N)).astype(np.float32)
        g = rng.normal(size=N).astype(np.float32)
        h = to_dev(h0)
        P.linear(ad, wtd, P.ACID_EPI_GATE_RESIDUAL, bd, gate=to_dev(g), out=h)
        # plus the rounding of the fp32 update h + g y
        return [(to_np(h) - h0, g * y, 1e-5,
                 np.abs(g) * acc_err + 2.0 ** -23 * (np.abs(h0) + np.abs(g * y)))]
    if kind == "euler":
        x0 = rng.normal(size=(M, N)).astype(np.float32)
        x = to_dev(x0)
        v = torch.empty((M, N), device="cuda")
        P.linear(ad, wtd, P.ACID_EPI_EULER, bd, out=x, v_out=v, dsigma=-0.125)
        return [(to_np(v), y, 1e-5, acc_err),
                (to_np(x) - x0, -0.125 * y, 1e-5,
                 0.125 * acc_err + 2.0 ** -23 * (np.abs(x0) + np.abs(0.125 * y)))]
    # qkv: N = 3 * heads * d; qkv_prescaled stores Q times log2(e)/sqrt(d)
    d = 64
    nh = N // (3 * d)
    H = nh * d
    vt_ld = ((M + 7) // 8) * 8
    q = torch.empty((nh, M, d), dtype=dtype, device="cuda")
    k = torch.empty((nh, M, d), dtype=dtype, device="cuda")
    vt = torch.zeros((nh, d, vt_ld), dtype=dtype, device="cuda")
    pre = kind == "qkv_prescaled"
    P.linear(ad, wtd, P.ACID_EPI_QKV, bd, q=q, k=k, vt=vt, n_heads=nh, head_dim=d, q_prescale=pre)
    tol = 1e-5 if dtype == torch.float32 else 4e-3
    c = P.q_scale(d) if pre else 1.0
    yq = y[:, :H].reshape(M, nh, d).transpose(1, 0, 2) * c
    yk = y[:, H:2 * H].reshape(M, nh, d).transpose(1, 0, 2)
    yv = y[:, 2 * H:].reshape(M, nh, d).transpose(1, 2, 0)
    eq = acc_err[:, :H].reshape(M, nh, d).transpose(1, 0, 2) * c + 2.0 ** -23 * np.abs(yq)
    ek = acc_err[:, H:2 * H].reshape(M, nh, d).transpose(1, 0, 2)
    ev = acc_err[:, 2 * H:].reshape(M, nh, d).transpose(1, 2, 0)
    return [(to_np(q), yq, tol, eq), (to_np(k), yk, tol, ek), (to_np(vt)[:, :, :M], yv, tol, ev)]


def _check_linear_elementwise(got, ref, atol, bf16_out, what):
    """fp32 outputs: within the accumulation bound (and 2 ulp of the value);
    bf16 outputs (GELU, Q, K, V): plus one bf16 rounding of the value."""
    rtol = 1.01 * 2.0 ** -8 if bf16_out else 2.0 ** -22
    assert_elementwise(got, ref, atol, rtol, what)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("M,N,K", [(1, 384, 128), (255, 384, 256), (300, 768, 384), (600, 384, 640), (513, 1152, 1536)])
def test_linear(P, kind, dtype, M, N, K):
    bf16_out = dtype == torch.bfloat16 and kind in ("gelu", "qkv", "qkv_prescaled")
    for got, ref, tol, atol in _linear_case(P, kind, M, N, K, dtype, seed=M + N + K):
        e = rel_err(got, ref)
        assert e < tol, (kind, e)
        _check_linear_elementwise(got, ref, atol, bf16_out, f"{kind} M={M} N={N} K={K}")


@pytest.mark.parametrize("kind", KINDS)
def test_linear_large_tiles_ragged(P, kind):
    """Large ragged shapes: ragged M over many 256-row tiles and, for
    N = 2176, a half-width last feature tile."""
    M, K = 8200, 256
    N = 2304 if kind.startswith("qkv") else 2176
    # the qkv case in _linear_case uses d = 64: 2304 = 3 x 12 x 64
    for got, ref, tol, atol in _linear_case(P, kind, M, N, K, torch.bfloat16, seed=17):
        assert rel_err(got, ref) < tol, kind
        _check_linear_elementwise(got, ref, atol, kind in ("gelu", "qkv", "qkv_prescaled"),
                                  f"{kind} M={M} N={N} K={K}")


@pytest.mark.parametrize("d", [64, 128])
def test_linear_qkv_prescale_fp32_bits(P, d):
    """fp32 QKV with q_prescale: Q is the float32 product of the unscaled
    Q with log2(e)/sqrt(d) bit for bit; K and V are unchanged."""
    M, nh, K = 300, 2, 256
    N = 3 * nh * d
    rng = np.random.default_rng(d)
    a = to_dev(rng.normal(size=(M, K)).astype(np.float32))
    wt = to_dev((rng.normal(size=(N, K)) / math.sqrt(K)).astype(np.float32))
    b = to_dev(rng.normal(size=N).astype(np.float32) * 0.1)
    outs = []
    for pre in (False, True):
        q = torch.empty((nh, M, d), device="cuda")
        k = torch.empty((nh, M, d), device="cuda")
        vt = torch.zeros((nh, d, (M + 7) // 8 * 8), device="cuda")
        P.linear(a, wt, P.ACID_EPI_QKV, b, q=q, k=k, vt=vt, n_heads=nh, head_dim=d, q_prescale=pre)
        outs.append((to_np(q), to_np(k), to_np(vt)))
    (q0, k0, v0), (q1, k1, v1) = outs
    np.testing.assert_array_equal(q1, (q0 * np.float32(P.q_scale(d))).astype(np.float32))
    np.testing.assert_array_equal(k1, k0)
    np.testing.assert_array_equal(v1, v0)


def test_linear_shape_errors(P):
    a = torch.zeros((4, 128), dtype=torch.bfloat16, device="cuda")
    wt = torch.zeros((100, 128), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(100, device="cuda")
    out = torch.zeros((4, 100), device="cuda")
    with pytest.raises(P.AcidError) as ei:
        P.linear(a, wt, P.ACID_EPI_BIAS, b, out=out)
    assert ei.value.status == 2
    wt = torch.zeros((128, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(P.AcidError) as ei:
        P.linear(a[:, :64].contiguous(), wt, P.ACID_EPI_BIAS, b[:128], out=out[:, :128].contiguous())
    assert ei.value.status == 2


def test_linear_deterministic(P):
    got = []
    for _ in range(3):
        (o, _, _, _), = _linear_case(P, "bias", 700, 1536, 1536, torch.bfloat16, seed=5)
        got.append(o)
    assert np.array_equal(got[0], got[1]) and np.array_equal(got[0], got[2])


def test_empty_inputs_are_no_ops(P):
    """Zero-length work through every component call returns cleanly and
    writes nothing: attention over 0 tokens, a GEMM with 0 rows, the cache,
    EasyCache's reuse and L1 sums over 0 elements."""
    dev = "cuda"
    for d in (64, 128):
        q = torch.empty((2, 0, d), dtype=torch.bfloat16, device=dev)
        vt = torch.empty((2, d, 0), dtype=torch.bfloat16, device=dev)
        P.attention(q, q, vt, torch.empty((0, 2 * d), dtype=torch.bfloat16, device=dev))
    wt = torch.zeros((256, 128), dtype=torch.bfloat16, device=dev)
    b = torch.zeros(256, device=dev)
    P.linear(torch.empty((0, 128), dtype=torch.bfloat16, device=dev), wt, P.ACID_EPI_BIAS, b,
             out=torch.empty((0, 256), device=dev))
    z = torch.empty(0, device=dev)
    P.cache_apply(P.ACID_CACHE_STORE, z, z, z)
    P.easycache_reuse(z, z, z, z, -0.1)
    torch.cuda.synchronize()
    m, _ = make_model(P, ai.TINY, max_steps=2)
    x = torch.ones(4, device=dev)
    assert m.l1_norms(x[:0], x[:0], x[:0]) == (0.0, 0.0)

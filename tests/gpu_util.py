"""Helpers shared by the GPU parity tests (marshalling and error metrics only)."""
import numpy as np
import pytest
import torch

import acid_inputs as ai
import oracle as O


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_12358_amd as P
    P.lib()  # raises if the HIP library is not built
    return P


def rel_err(got, ref) -> float:
    """Frobenius relative error ||got - ref|| / ||ref||."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def to_dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(dtype)


def to_np(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def bf16_values(a) -> np.ndarray:
    """The float32 values a bf16 device tensor made from `a` holds (oracle rounding)."""
    return O.bf16_round(np.asarray(a, np.float32))


def make_model(P, cfg, max_steps=None, seed=ai.SEED_WEIGHTS, std=ai.WEIGHT_STD, keep=None):
    """The library model with the seeded weights; returns it with the host
    copies of the tensors whose names pass `keep` (all if None)."""
    m = P.Model(cfg, max_steps=max_steps or cfg.n_steps)
    params = {}

    def gen():
        for tid, name, w in ai.iter_weights(cfg, seed, std):
            if keep is None or keep(name):
                params[name] = w
            yield tid, name, w

    m.load_weights(gen())
    torch.cuda.synchronize()
    return m, params


def assert_elementwise(got, ref, atol, rtol, what="") -> float:
    """|got - ref| <= atol + rtol |ref| for every element (atol may be an
    array of per-element bounds).  Returns the largest ratio of error to
    bound (<= 1), and names the worst element when the bound fails."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    bound = np.broadcast_to(np.asarray(atol, np.float64), ref.shape) + rtol * np.abs(ref)
    ratio = np.where(err == 0, 0.0, err / np.maximum(bound, 1e-300))
    ratio = np.where(np.isnan(ratio), np.inf, ratio)
    i = np.unravel_index(int(np.argmax(ratio)), ratio.shape) if ratio.size else ()
    worst = float(ratio[i]) if ratio.size else 0.0
    print(f"[elementwise] {what}: worst error / bound {worst:.3f}", flush=True)
    assert worst <= 1.0, (f"{what}: |got - ref| = {err[i]:.3e} exceeds {bound[i]:.3e} at {i} "
                          f"(got {got[i]:.6g}, ref {ref[i]:.6g}; worst ratio {worst:.2f})")
    return worst


def assert_close_to_scale(got, ref, bf16: bool, what="") -> float:
    """Element bound for a composed output (a block's or a step's), whose
    error collects the roundings of several GEMM operands and cannot be
    bounded term by term: |got - ref| <= a rms(ref) + r |ref| with
    (a, r) = (2^-5, 2^-6) for bf16 operands and (4e-4, 1e-4) for fp32.  A
    wrong row, column or tile is off by the output's own scale and fails."""
    ref = np.asarray(ref, np.float64)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    a, r = (2.0 ** -5, 2.0 ** -6) if bf16 else (4e-4, 1e-4)
    return assert_elementwise(got, ref, a * rms, r, what)


BF16_U = 2.0 ** -8  # unit roundoff of bfloat16 (8-bit significand)


def attention_bound(q, k, v, dtype_bf16=True):
    """Per-element error bound of the attention kernel against the definition
    on the same operands.  bf16: each probability is rounded once to bf16
    (relative error <= u) and the row sum is taken over those rounded values,
    so the normalised weights differ from the exact ones by at most 2u of
    their own size: |o_kernel - o| <= 2u sum_j p_j |v_j|, before the output's
    own rounding (u |o|, the rtol part).  sum_j p_j |v_j| is attention with
    |V|.  Returns the atol array (5% slack for the fp32 arithmetic); fp32
    runs use 3e-5 of it instead."""
    import oracle as O
    a = O.attention(q, k, np.abs(np.asarray(v, np.float64)))
    return (1.05 * 2 * BF16_U if dtype_bf16 else 3e-5) * a

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


def make_model(P, cfg, max_steps=None, seed=ai.SEED_WEIGHTS, std=ai.WEIGHT_STD):
    m = P.Model(cfg, max_steps=max_steps or cfg.n_steps)
    params = {}

    def gen():
        for tid, name, w in ai.iter_weights(cfg, seed, std):
            params[name] = w
            yield tid, name, w

    m.load_weights(gen())
    torch.cuda.synchronize()
    return m, params

"""acid_l1_norms_noalloc (no model, partial sums in the library's own device
array) against acid_l1_norms (partial sums in a model's workspace), through
the C ABI: two calls in a row, the second on a smaller input, so the array's
contents from the first call must not leak into the second."""
import ctypes as C

import numpy as np
import pytest
import torch

import acid_inputs as ai
from gpu_util import need_gpu

pytestmark = pytest.mark.gpu


def _seeded(n, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return torch.randn(n, generator=g, device="cuda")


def _noalloc(P, a, b, c, n):
    out = (C.c_double * 2)()
    ptr = lambda t: None if t is None else C.c_void_p(t.data_ptr())
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    P._L.check(P.lib().acid_l1_norms_noalloc(ptr(a), ptr(b), ptr(c), n, out, stream))
    return out[0], out[1]


def test_l1_norms_noalloc_matches_model_call():
    P = need_gpu()
    # n_video >= 1024: the model call runs the full 1024-workgroup grid too,
    # so both calls sum in the same order and must agree bit for bit
    cfg = ai.SMALL.replace(n_blocks=1, n_steps=2)
    m = P.Model(cfg, max_steps=2)
    n_big = cfg.n_video * cfg.hidden           # 1M elements, 1024 workgroups
    n_small = 3 * 1024 * 37 + 3                # ragged, fewer workgroups
    a, b, c = _seeded(n_big, 1), _seeded(n_big, 2), _seeded(n_big, 3)
    for n in (n_big, n_small):
        for bb, cc in ((b, c), (b, None), (None, c), (None, None)):
            want = m.l1_norms(a[:n], None if bb is None else bb[:n],
                              None if cc is None else cc[:n])
            got = _noalloc(P, a[:n], None if bb is None else bb[:n],
                           None if cc is None else cc[:n], n)
            assert got == want, (n, bb is None, cc is None, got, want)
    # against the same sum on the host (fp32 differences, as the kernel
    # forms them, added in fp64), and the empty and tiny cases
    ref0 = float((a[:n_small] - b[:n_small]).abs().double().sum())
    got = _noalloc(P, a[:n_small], b[:n_small], None, n_small)
    assert got[0] == pytest.approx(ref0, rel=1e-12) and got[1] == 0.0
    assert _noalloc(P, None, None, None, 0) == (0.0, 0.0)
    x = torch.tensor([1.5, -2.0, 0.25, 4.0, -8.0], device="cuda")
    assert _noalloc(P, x, None, x, 5) == (15.75, 15.75)
    # errors are reported, not launched
    with pytest.raises(P.AcidError):
        _noalloc(P, a, b, c, -1)
    with pytest.raises(P.AcidError):
        _noalloc(P, a[1:], None, None, 16)  # not 16-byte aligned

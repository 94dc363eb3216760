"""ACID-gated video-DiT denoise loop on AMD Instinct MI355X (gfx950).

Python face of libacid: each function marshals torch tensors (device memory)
and the current HIP stream into one C-ABI call.  All arithmetic runs in the
library's HIP kernels; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import math
from typing import Iterable, Optional, Sequence

import numpy as np

from . import _lib as _L
from ._lib import (ACID_BF16, ACID_CACHE_APPLY, ACID_CACHE_STORE, ACID_EPI_BIAS,  # noqa: F401
                   ACID_EPI_BIAS_GELU, ACID_EPI_EULER, ACID_EPI_GATE_RESIDUAL, ACID_EPI_QKV,
                   ACID_EPI_QKV_GELU, ACID_BLOCK_PARALLEL, ACID_BLOCK_SEQUENTIAL,
                   ACID_F32, ACID_MODE_ACID, ACID_MODE_DICACHE, ACID_MODE_EASYCACHE,
                   ACID_MODE_NOCACHE,
                   KERNEL_CLASSES, AcidError,
                   TRACE_DTYPE, check, lib)

__all__ = ["Model", "gate", "GateState", "gate_device_sequence", "cache_apply", "easycache_reuse", "attention", "linear",
           "ln_modulate", "q_scale", "version", "AcidError", "KERNEL_CLASSES"]


def _torch():
    import torch
    return torch


def _stream(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return C.c_void_p(t.data_ptr())


def version() -> str:
    return lib().acid_version().decode()


def _torch_dtype(code):
    torch = _torch()
    return torch.bfloat16 if code == ACID_BF16 else torch.float32


# ------------------------------------------------------------------ gate


class GateState:
    """Algorithm 1's state (plain data, zero = initial)."""

    def __init__(self):
        self.c = _L.GateStateC()


def gate(state: GateState, tau_low: float, tau_high: float, delta: float, s_t: float,
         n_warmup: int = 1):
    """One step of the host gate. Returns (compute: bool, tau_used: float)."""
    p = _L.GateParamsC(tau_low, tau_high, delta, n_warmup)
    comp = C.c_int32()
    tau = C.c_double()
    check(lib().acid_gate(C.byref(state.c), C.byref(p), float(s_t), C.byref(comp), C.byref(tau)))
    return bool(comp.value), tau.value


def gate_device_sequence(signals, tau_low: float, tau_high: float, delta: float,
                         n_warmup: int = 1, device="cuda", stream=None) -> np.ndarray:
    """Algorithm 1 run by the device gate over a whole signal sequence (NaN
    where a step has no signal); returns the trace (waits for the GPU)."""
    torch = _torch()
    sig = np.ascontiguousarray(signals, dtype=np.float64)
    n = len(sig)
    p = _L.GateParamsC(tau_low, tau_high, delta, n_warmup)
    s_d = torch.from_numpy(sig).to(device)
    tsz = C.sizeof(_L.StepTraceC)
    tr_d = torch.zeros(max(n, 1) * tsz, dtype=torch.uint8, device=device)
    check(lib().acid_gate_device_sequence(C.byref(p), _ptr(s_d), n, _ptr(tr_d),
                                          _stream(stream)))
    raw = tr_d.cpu().numpy()  # waits for the stream
    tr = (_L.StepTraceC * max(n, 1))()
    C.memmove(tr, raw.ctypes.data, max(n, 1) * tsz)
    out = np.zeros(n, dtype=TRACE_DTYPE)
    for i in range(n):
        out[i] = (tr[i].compute, tr[i].gate_compute, tr[i].s, tr[i].sigma_sum_after,
                  tr[i].tau_used)
    return out


# ------------------------------------------------------------ components


def cache_apply(op: int, x, h_out, r, stream=None) -> None:
    n = x.numel()
    if h_out.numel() != n or r.numel() != n:
        raise ValueError("x, h_out and r must have the same number of elements")
    check(lib().acid_cache_apply(op, _ptr(x), _ptr(h_out), _ptr(r), n, _stream(stream)))


def easycache_reuse(x, x_prev, v, offset, dsigma: float, stream=None) -> None:
    """EasyCache's skipped step: v = x + offset; x_prev = x; x += dsigma v."""
    n = x.numel()
    if x_prev.numel() != n or v.numel() != n or offset.numel() != n:
        raise ValueError("x, x_prev, v and offset must have the same number of elements")
    check(lib().acid_easycache_reuse(_ptr(x), _ptr(x_prev), _ptr(v), _ptr(offset), n,
                                     float(dsigma), _stream(stream)))


def ln_modulate(x, shift, scale, out, stream=None) -> None:
    rows, hidden = x.shape
    code = ACID_BF16 if out.dtype == _torch().bfloat16 else ACID_F32
    check(lib().acid_ln_modulate(code, _ptr(x), rows, hidden, _ptr(shift), _ptr(scale),
                                 _ptr(out), _stream(stream)))


def attention(q, k, vt, o, stream=None, q_prescaled: bool = False) -> None:
    """q, k [heads, L, d]; vt [heads, d, vt_ld]; o [L, heads*d]; all bf16 or all fp32.
    q_prescaled: q holds Q * q_scale(d), as the QKV epilogue stores it with
    q_prescale=True (the model's own path)."""
    n_heads, L, d = q.shape
    code = ACID_BF16 if q.dtype == _torch().bfloat16 else ACID_F32
    check(lib().acid_attention(code, n_heads, L, d, _ptr(q), _ptr(k), _ptr(vt), vt.shape[2],
                               _ptr(o), int(bool(q_prescaled)), _stream(stream)))


def q_scale(d: int) -> float:
    """The float32 factor log2(e)/sqrt(d) a pre-scaled Q carries (the
    library's own constant, acid_q_scale)."""
    return float(lib().acid_q_scale(int(d)))


def linear(a, wt, kind: int, bias, gate=None, out=None, v_out=None, q=None, k=None, vt=None,
           n_heads=0, head_dim=0, dsigma=0.0, bias2=None, q_prescale=False,
           stream=None) -> None:
    """Fused GEMM y = a @ wt.T + bias with an epilogue (see include/acid.h).
    For ACID_EPI_QKV_GELU, out may be a row-strided view (unit column
    stride); its row stride is passed as out_ld."""
    M, K = a.shape
    N = wt.shape[0]
    code = ACID_BF16 if a.dtype == _torch().bfloat16 else ACID_F32
    e = _L.EpilogueArgsC()
    e.kind = kind
    e.bias = _ptr(bias)
    e.gate = _ptr(gate)
    e.bias2 = _ptr(bias2)
    if kind == _L.ACID_EPI_QKV_GELU and out is not None:
        if not out.is_cuda or out.stride(-1) != 1:
            raise ValueError("out must be a device tensor with unit column stride")
        e.out = C.c_void_p(out.data_ptr())
        e.out_ld = out.stride(0)
    else:
        e.out = _ptr(out)
    e.v_out = _ptr(v_out)
    e.q, e.k, e.vt = _ptr(q), _ptr(k), _ptr(vt)
    e.vt_ld = vt.shape[-1] if vt is not None else 0
    e.n_heads, e.head_dim, e.dsigma = n_heads, head_dim, dsigma
    e.q_prescale = int(bool(q_prescale))
    check(lib().acid_linear(code, M, N, K, _ptr(a), _ptr(wt), C.byref(e), _stream(stream)))


# ------------------------------------------------------------------ model


class Model:
    """A DiT stack bound to a caller-side (torch) weight arena and workspace."""

    def __init__(self, cfg, max_steps: int = 1, device="cuda"):
        torch = _torch()
        self.cfg = cfg
        self.c = _L.config_c(cfg)
        check(lib().acid_config_check(C.byref(self.c)))
        self.max_steps = max_steps
        wb = lib().acid_weights_bytes(C.byref(self.c))
        kb = lib().acid_workspace_bytes(C.byref(self.c), max_steps)
        self.arena = torch.empty(wb, dtype=torch.uint8, device=device)
        self.workspace = torch.empty(kb, dtype=torch.uint8, device=device)
        h = C.c_void_p()
        check(lib().acid_model_create(C.byref(self.c), _ptr(self.arena), _ptr(self.workspace),
                                      max_steps, C.byref(h)))
        self.h = h
        self.device = device
        self.dtype_code = self.c.dtype

    def __del__(self):
        try:
            if getattr(self, "h", None) and _L._lib is not None:
                _L._lib.acid_model_destroy(self.h)
                self.h = None
        except Exception:
            pass

    # -- weights ----------------------------------------------------------
    def tensor_count(self) -> int:
        return lib().acid_tensor_count(C.byref(self.c))

    def tensor_shape(self, tid: int):
        rank = C.c_int32()
        dims = (C.c_int64 * 2)()
        check(lib().acid_tensor_shape(C.byref(self.c), tid, C.byref(rank), dims))
        return tuple(dims[:rank.value])

    def load_tensor(self, tid: int, src, stream=None) -> None:
        """src: fp32 device tensor of the manifest shape [in, out]."""
        check(lib().acid_model_load_tensor(self.h, tid, _ptr(src), src.numel(), _stream(stream)))

    def load_tensor_host(self, tid: int, src: np.ndarray, stream=None) -> None:
        """src: fp32 host array of the manifest shape [in, out] (staged through
        the workspace; the call waits for the stream)."""
        a = np.ascontiguousarray(src, dtype=np.float32)
        check(lib().acid_model_load_tensor_host(self.h, tid, a.ctypes.data_as(C.c_void_p),
                                                a.size, _stream(stream)))

    def load_weights(self, tensors: Iterable) -> None:
        """tensors: iterable of (id, name, fp32 numpy array) in any order."""
        torch = _torch()
        for tid, _name, arr in tensors:
            src = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(self.device)
            self.load_tensor(tid, src)
            torch.cuda.current_stream().synchronize()
            del src

    # -- the five calls ---------------------------------------------------
    def dit_step(self, x, sigma: float, text=None, v=None, resid=None, stream=None):
        torch = _torch()
        if v is None:
            v = torch.empty_like(x)
        check(lib().acid_dit_step(self.h, _ptr(x), float(sigma), _ptr(text), _ptr(v),
                                  _ptr(resid), _stream(stream)))
        return v

    def drift_signal(self, x, sigma: float, m_prev, m_cur, stream=None) -> float:
        s = C.c_double()
        check(lib().acid_drift_signal(self.h, _ptr(x), float(sigma), _ptr(m_prev), _ptr(m_cur),
                                      C.byref(s), _stream(stream)))
        return s.value

    def set_probe_blocks(self, n_probe: int) -> None:
        """DiCache probe depth (first n_probe blocks run on every step)."""
        check(lib().acid_model_set_probe_blocks(self.h, int(n_probe)))

    def l1_norms(self, a, b=None, c=None, stream=None):
        """(sum |a - b| or sum |a|, sum |c| or 0) in fp64, deterministic."""
        out = (C.c_double * 2)()
        check(lib().acid_l1_norms(self.h, _ptr(a), _ptr(b), _ptr(c), a.numel(), out,
                                  _stream(stream)))
        return out[0], out[1]

    def denoise_loop(self, x, sigmas: Sequence[float], text=None, mode: str = "acid",
                     tau_low: float = 0.05, tau_high: float = 0.2, delta: float = 0.01,
                     n_warmup: Optional[int] = None, forced_schedule=None,
                     stream=None, graph: bool = False,
                     trace: bool = True) -> Optional[np.ndarray]:
        """Runs the loop in place on x; returns the per-step trace.  mode is
        "nocache", "acid" (TeaCache's signal), "easycache" or "dicache"
        (probe depth: set_probe_blocks); n_warmup defaults to 1 (2 for
        "easycache").  graph=True runs the device-gate loop captured as a
        HIP graph (any mode); with trace=False it returns None without
        waiting for the GPU."""
        sig = np.ascontiguousarray(sigmas, dtype=np.float32)
        n = len(sig) - 1
        modes = {"acid": ACID_MODE_ACID, "nocache": ACID_MODE_NOCACHE,
                 "easycache": ACID_MODE_EASYCACHE, "dicache": ACID_MODE_DICACHE}
        if mode not in modes:
            raise ValueError(f"unknown mode {mode!r}")
        modec = modes[mode]
        if n_warmup is None:
            n_warmup = 2 if mode == "easycache" else 1
        p = _L.GateParamsC(tau_low, tau_high, delta, n_warmup)
        tr = (_L.StepTraceC * n)()
        forced = None
        if forced_schedule is not None:
            fs = np.ascontiguousarray(forced_schedule, dtype=np.uint8)
            forced = fs.ctypes.data_as(C.POINTER(C.c_uint8))
        fn = lib().acid_denoise_loop_graph if graph else lib().acid_denoise_loop
        check(fn(self.h, _ptr(x), sig.ctypes.data_as(C.POINTER(C.c_float)), n, _ptr(text),
                 modec, C.byref(p), forced, tr if trace else None, _stream(stream)))
        if not trace:
            return None
        out = np.zeros(n, dtype=TRACE_DTYPE)
        for i in range(n):
            out[i] = (tr[i].compute, tr[i].gate_compute, tr[i].s, tr[i].sigma_sum_after,
                      tr[i].tau_used)
        return out

    # -- components --------------------------------------------------------
    def timestep_modulation(self, sigmas, stream=None):
        torch = _torch()
        sig = np.ascontiguousarray(sigmas, dtype=np.float32)
        H, nb = self.cfg.hidden, self.cfg.n_blocks
        table = torch.empty((len(sig), 6 * nb + 2, H), dtype=torch.float32, device=self.device)
        check(lib().acid_timestep_modulation(self.h, sig.ctypes.data_as(C.POINTER(C.c_float)),
                                             len(sig), _ptr(table), _stream(stream)))
        return table

    def block_forward(self, block: int, mod6, h, stream=None) -> None:
        check(lib().acid_block_forward(self.h, block, _ptr(mod6), _ptr(h), _stream(stream)))

    # -- timing ------------------------------------------------------------
    def set_timing(self, enable: bool) -> None:
        check(lib().acid_model_set_timing(self.h, int(enable)))

    def reset_timing(self) -> None:
        check(lib().acid_model_reset_timing(self.h))

    def timing(self) -> dict:
        out = {}
        for i, name in enumerate(KERNEL_CLASSES):
            ms = C.c_double()
            n = C.c_int64()
            check(lib().acid_model_timing(self.h, i, C.byref(ms), C.byref(n)))
            out[name] = (ms.value, n.value)
        return out

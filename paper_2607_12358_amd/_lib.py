"""ctypes binding of libacid.so (argument marshalling only).

Every computation runs in the library's HIP kernels; PyTorch is used only to
allocate device memory and to supply the current HIP stream.  Loading fails
loudly if the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
import re
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libacid.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "acid.h")

ACID_OK, ACID_ERR_INVALID_ARG, ACID_ERR_SHAPE, ACID_ERR_HIP, ACID_ERR_UNSUPPORTED = range(5)
ACID_F32, ACID_BF16 = 0, 1
ACID_MODE_NOCACHE, ACID_MODE_ACID, ACID_MODE_EASYCACHE, ACID_MODE_DICACHE = 0, 1, 2, 3
ACID_CACHE_STORE, ACID_CACHE_APPLY = 0, 1
(ACID_EPI_BIAS, ACID_EPI_BIAS_GELU, ACID_EPI_GATE_RESIDUAL, ACID_EPI_QKV,
 ACID_EPI_EULER, ACID_EPI_QKV_GELU) = range(6)
ACID_BLOCK_SEQUENTIAL, ACID_BLOCK_PARALLEL = 0, 1
KERNEL_CLASSES = ("temb", "ln_mod", "gemm_qkv", "attention", "gemm_proj", "gemm_ffn1",
                  "gemm_ffn2", "gemm_head", "drift", "cache", "misc")


class AcidError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libacid status {status}: {msg}")
        self.status = status


class DitConfigC(C.Structure):
    _fields_ = [("n_blocks", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("ffn", C.c_int32), ("freq_dim", C.c_int32),
                ("n_video", C.c_int32), ("n_text", C.c_int32), ("dtype", C.c_int32),
                ("block_kind", C.c_int32)]


class GateParamsC(C.Structure):
    _fields_ = [("tau_low", C.c_double), ("tau_high", C.c_double), ("delta", C.c_double),
                ("n_warmup", C.c_int32)]


class GateStateC(C.Structure):
    _fields_ = [("sigma_sum", C.c_double), ("s_prev", C.c_double), ("has_prev", C.c_int32),
                ("step", C.c_int32)]


class StepTraceC(C.Structure):
    _fields_ = [("compute", C.c_int32), ("gate_compute", C.c_int32), ("s", C.c_double),
                ("sigma_sum_after", C.c_double), ("tau_used", C.c_double)]


class EpilogueArgsC(C.Structure):
    _fields_ = [("kind", C.c_int32), ("bias", C.c_void_p), ("gate", C.c_void_p),
                ("bias2", C.c_void_p), ("out", C.c_void_p), ("out_ld", C.c_int64),
                ("v_out", C.c_void_p), ("q", C.c_void_p),
                ("k", C.c_void_p), ("vt", C.c_void_p), ("vt_ld", C.c_int64),
                ("n_heads", C.c_int32), ("head_dim", C.c_int32), ("dsigma", C.c_float),
                ("q_prescale", C.c_int32)]


_P = C.c_void_p
_SIGS = {
    "acid_version": (C.c_char_p, []),
    "acid_last_error": (C.c_char_p, []),
    "acid_config_check": (C.c_int, [C.POINTER(DitConfigC)]),
    "acid_weights_bytes": (C.c_size_t, [C.POINTER(DitConfigC)]),
    "acid_workspace_bytes": (C.c_size_t, [C.POINTER(DitConfigC), C.c_int32]),
    "acid_tensor_count": (C.c_int32, [C.POINTER(DitConfigC)]),
    "acid_tensor_shape": (C.c_int, [C.POINTER(DitConfigC), C.c_int32, C.POINTER(C.c_int32),
                                    C.POINTER(C.c_int64)]),
    "acid_model_create": (C.c_int, [C.POINTER(DitConfigC), _P, _P, C.c_int32, C.POINTER(_P)]),
    "acid_model_load_tensor": (C.c_int, [_P, C.c_int32, _P, C.c_int64, _P]),
    "acid_model_load_tensor_host": (C.c_int, [_P, C.c_int32, _P, C.c_int64, _P]),
    "acid_q_scale": (C.c_float, [C.c_int32]),
    "acid_model_destroy": (None, [_P]),
    "acid_model_set_timing": (C.c_int, [_P, C.c_int32]),
    "acid_model_reset_timing": (C.c_int, [_P]),
    "acid_model_timing": (C.c_int, [_P, C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    "acid_dit_step": (C.c_int, [_P, _P, C.c_float, _P, _P, _P, _P]),
    "acid_drift_signal": (C.c_int, [_P, _P, C.c_float, _P, _P, C.POINTER(C.c_double), _P]),
    "acid_gate": (C.c_int, [C.POINTER(GateStateC), C.POINTER(GateParamsC), C.c_double,
                            C.POINTER(C.c_int32), C.POINTER(C.c_double)]),
    "acid_cache_apply": (C.c_int, [C.c_int, _P, _P, _P, C.c_int64, _P]),
    "acid_l1_norms": (C.c_int, [_P, _P, _P, _P, C.c_int64, C.POINTER(C.c_double), _P]),
    "acid_l1_norms_noalloc": (C.c_int, [_P, _P, _P, C.c_int64, C.POINTER(C.c_double), _P]),
    "acid_model_set_probe_blocks": (C.c_int, [_P, C.c_int32]),
    "acid_easycache_reuse": (C.c_int, [_P, _P, _P, _P, C.c_int64, C.c_float, _P]),
    "acid_denoise_loop": (C.c_int, [_P, _P, C.POINTER(C.c_float), C.c_int32, _P, C.c_int32,
                                    C.POINTER(GateParamsC), C.POINTER(C.c_uint8),
                                    C.POINTER(StepTraceC), _P]),
    "acid_denoise_loop_graph": (C.c_int, [_P, _P, C.POINTER(C.c_float), C.c_int32, _P,
                                          C.c_int32, C.POINTER(GateParamsC),
                                          C.POINTER(C.c_uint8), C.POINTER(StepTraceC), _P]),
    "acid_gate_device_sequence": (C.c_int, [C.POINTER(GateParamsC), _P, C.c_int32, _P, _P]),
    "acid_timestep_modulation": (C.c_int, [_P, C.POINTER(C.c_float), C.c_int32, _P, _P]),
    "acid_ln_modulate": (C.c_int, [C.c_int32, _P, C.c_int64, C.c_int32, _P, _P, _P, _P]),
    "acid_attention": (C.c_int, [C.c_int32, C.c_int32, C.c_int64, C.c_int32, _P, _P, _P,
                                 C.c_int64, _P, C.c_int32, _P]),
    "acid_linear": (C.c_int, [C.c_int32, C.c_int64, C.c_int32, C.c_int32, _P, _P,
                              C.POINTER(EpilogueArgsC), _P]),
    "acid_block_forward": (C.c_int, [_P, C.c_int32, _P, _P, _P]),
}

_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    """The loaded library; raises if it was not built (no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_12358_amd.build` (there is no CPU fallback)")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def header_symbols() -> list:
    """Function names declared in include/acid.h."""
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(acid_[a-z0-9_]+)\s*\(", src)))


def check(status: int) -> None:
    if status != ACID_OK:
        raise AcidError(status, lib().acid_last_error().decode())


def last_error() -> str:
    return lib().acid_last_error().decode()


def dtype_code(dtype) -> int:
    if dtype in ("bf16", ACID_BF16):
        return ACID_BF16
    if dtype in ("f32", "fp32", ACID_F32):
        return ACID_F32
    raise ValueError(f"unknown dtype {dtype!r}")


def config_c(cfg) -> DitConfigC:
    """acid_dit_config from any object with the DiT shape attributes."""
    kind = {"sequential": ACID_BLOCK_SEQUENTIAL, "parallel": ACID_BLOCK_PARALLEL}[
        getattr(cfg, "block", "sequential")]
    return DitConfigC(cfg.n_blocks, cfg.hidden, cfg.n_heads, cfg.head_dim, cfg.ffn,
                      cfg.freq_dim, cfg.n_video, cfg.n_text, dtype_code(cfg.dtype), kind)


TRACE_DTYPE = np.dtype([("compute", np.int32), ("gate_compute", np.int32), ("s", np.float64),
                        ("sigma_sum_after", np.float64), ("tau_used", np.float64)])

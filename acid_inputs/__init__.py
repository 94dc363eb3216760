"""Seeded synthetic inputs for the ACID-gated video-DiT denoise loop.

This module is shared by the CPU oracle, the tests and the benchmark.  It
holds shapes, the parameter manifest and seeded random draws only: none of the
method's arithmetic lives here.

The paper evaluates trained HunyuanVideo, Wan 2.1 and CogVideoX models on
VBench prompts (Section 4.1).  Neither the weights nor the prompts are used
here: random-init stacks with the same shapes stand in for the models, and
N(0, 1) tokens stand in for latents and text embeddings.

Manifest (tensor id order, shapes in [in, out] convention, y = x @ W + b):

    0 temb.w1 [F_t, H]   1 temb.b1 [H]   2 temb.w2 [H, H]   3 temb.b2 [H]
    per block b (ids 4 + 10 b + j):
      j=0 ada.w [H, 6H]  1 ada.b [6H]  2 qkv.w [H, 3H]  3 qkv.b [3H]
      4 o.w [H, H]       5 o.b [H]     6 ffn1.w [H, F]  7 ffn1.b [F]
      8 ffn2.w [F, H]    9 ffn2.b [H]
    head (ids 4 + 10 n_b + j):
      j=0 head.ada.w [H, 2H]  1 head.ada.b [2H]  2 head.w [H, H]  3 head.b [H]

Tensor k is drawn as ``default_rng([seed_w, k]).standard_normal(shape,
float32) * 0.02`` so tensors can be produced one at a time.
"""
from __future__ import annotations

import dataclasses
from typing import Iterator, List, Optional, Tuple

import numpy as np

SEED_WEIGHTS = 0
SEED_LATENTS = 1
SEED_TEXT = 2
WEIGHT_STD = 0.02

BLOCK_TENSORS = ("ada.w", "ada.b", "qkv.w", "qkv.b", "o.w", "o.b",
                 "ffn1.w", "ffn1.b", "ffn2.w", "ffn2.b")
TEMB_TENSORS = ("temb.w1", "temb.b1", "temb.w2", "temb.b2")
HEAD_TENSORS = ("head.ada.w", "head.ada.b", "head.w", "head.b")


@dataclasses.dataclass(frozen=True)
class DiTConfig:
    """Shape of a synthetic video-DiT stack (no arithmetic)."""
    name: str
    n_blocks: int
    hidden: int
    n_heads: int
    head_dim: int
    ffn: int
    n_video: int
    n_text: int = 0
    freq_dim: int = 256
    dtype: str = "bf16"          # "f32" or "bf16"
    n_steps: int = 50
    # "sequential": attention then MLP, each with its own LN-modulate and
    # gated residual; "parallel": HunyuanVideo's single-stream form, both
    # branches from one LN-modulate and one gated residual, reusing the same
    # tensors as [qkv.w | ffn1.w] and [o.w ; ffn2.w].
    block: str = "sequential"

    @property
    def n_tokens(self) -> int:
        return self.n_text + self.n_video

    def replace(self, **kw) -> "DiTConfig":
        return dataclasses.replace(self, **kw)


# The five workloads: a tiny fp32 stack, a small bf16 stack, and stacks shaped
# like Wan 2.1 1.3B, CogVideoX 1.5 5B and a HunyuanVideo single-stream slice.
TINY = DiTConfig("tiny-dit-f32", n_blocks=1, hidden=256, n_heads=4, head_dim=64,
                 ffn=1024, n_video=2 * 8 * 8, dtype="f32", n_steps=10)
SMALL = DiTConfig("small-dit-bf16", n_blocks=4, hidden=1024, n_heads=16,
                  head_dim=64, ffn=4096, n_video=4 * 16 * 16, n_steps=30)
WAN13B = DiTConfig("wan2.1-1.3b-shape", n_blocks=30, hidden=1536, n_heads=12,
                   head_dim=128, ffn=8960, n_video=21 * 30 * 52, n_steps=50)
COG5B = DiTConfig("cogvideox-5b-shape", n_blocks=42, hidden=3072, n_heads=48,
                  head_dim=64, ffn=12288, n_video=13 * 30 * 45, n_text=226,
                  n_steps=50)
HUNYUAN = DiTConfig("hunyuanvideo-slice", n_blocks=4, hidden=3072, n_heads=24,
                    head_dim=128, ffn=12288, n_video=33 * 45 * 80, n_text=256,
                    n_steps=50)
HUNYUAN_PARALLEL = HUNYUAN.replace(name="hunyuanvideo-slice-parallel", block="parallel")
CONFIGS = {c.name: c for c in (TINY, SMALL, WAN13B, COG5B, HUNYUAN, HUNYUAN_PARALLEL)}


def manifest(cfg: DiTConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """(name, shape) for every parameter tensor, in tensor-id order."""
    H, F, Ft = cfg.hidden, cfg.ffn, cfg.freq_dim
    out: List[Tuple[str, Tuple[int, ...]]] = [
        ("temb.w1", (Ft, H)), ("temb.b1", (H,)), ("temb.w2", (H, H)),
        ("temb.b2", (H,))]
    for b in range(cfg.n_blocks):
        shapes = [(H, 6 * H), (6 * H,), (H, 3 * H), (3 * H,), (H, H), (H,),
                  (H, F), (F,), (F, H), (H,)]
        out += [(f"blocks.{b}.{n}", s) for n, s in zip(BLOCK_TENSORS, shapes)]
    out += [("head.ada.w", (H, 2 * H)), ("head.ada.b", (2 * H,)),
            ("head.w", (H, H)), ("head.b", (H,))]
    return out


def tensor_id(cfg: DiTConfig, name: str) -> int:
    for i, (n, _) in enumerate(manifest(cfg)):
        if n == name:
            return i
    raise KeyError(name)


def weight_tensor(cfg: DiTConfig, k: int, seed: int = SEED_WEIGHTS,
                  std: float = WEIGHT_STD) -> np.ndarray:
    """Tensor k of the manifest: N(0, std^2), fp32, seeded by (seed, k)."""
    _, shape = manifest(cfg)[k]
    rng = np.random.default_rng([seed, k])
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)


def iter_weights(cfg: DiTConfig, seed: int = SEED_WEIGHTS,
                 std: float = WEIGHT_STD) -> Iterator[Tuple[int, str, np.ndarray]]:
    for k, (name, _) in enumerate(manifest(cfg)):
        yield k, name, weight_tensor(cfg, k, seed, std)


def weights(cfg: DiTConfig, seed: int = SEED_WEIGHTS,
            std: float = WEIGHT_STD) -> dict:
    """All parameters as a name -> fp32 array dict."""
    return {name: w for _, name, w in iter_weights(cfg, seed, std)}


def latents(cfg: DiTConfig, seed: int = SEED_LATENTS) -> np.ndarray:
    """x_0 ~ N(0, 1), fp32 [n_video, hidden] (frames x rows x cols flattened)."""
    rng = np.random.default_rng([seed])
    return rng.standard_normal((cfg.n_video, cfg.hidden), dtype=np.float32)


def text_tokens(cfg: DiTConfig, seed: int = SEED_TEXT) -> Optional[np.ndarray]:
    """Random text-token embeddings N(0, 1), fp32 [n_text, hidden], or None."""
    if cfg.n_text == 0:
        return None
    rng = np.random.default_rng([seed])
    return rng.standard_normal((cfg.n_text, cfg.hidden), dtype=np.float32)


def sigmas(n_steps: int) -> np.ndarray:
    """Flow-matching noise levels 1 -> 0, linear, N+1 values.

    Computed in float64 and rounded once to float32; the array is an input to
    both implementations.
    """
    return (1.0 - np.arange(n_steps + 1, dtype=np.float64) / n_steps).astype(np.float32)


def gaussian(shape, seed, std: float = 1.0) -> np.ndarray:
    """Generic seeded N(0, std^2) fp32 array (kernel-level test inputs)."""
    rng = np.random.default_rng(list(np.atleast_1d(seed)))
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)

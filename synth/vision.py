"""Seeded synthetic inputs of the vision tower: images and weights.

The paper feeds its text encoder a 256x256 source patch through the
Qwen3-VL vision tower (Sec. I; Sec. III-A "Notation and Setup"); neither the
DAVIS-2017 frames nor trained weights are available, so these draws stand in
for them with the same shapes: images of normalised pixels N(0, 1), linear
weights and biases N(0, 0.02), LayerNorm gains 1 + U(-0.5, 0.5) and biases
N(0, 0.1).

Seeds: block ``l``'s weights from ``default_rng([1, l])``, the patch
embedding and the merger from ``default_rng([1, 10_000])``, image ``f`` from
``default_rng(2000 + f)``. Values are drawn in float32 and rounded to bf16
(ties to even) for bf16 configurations, as in ``synth.workloads``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict

import numpy as np

from .workloads import _gain, _normal, _store


@dataclasses.dataclass(frozen=True)
class VisionDims:
    depth: int
    hidden: int
    n_heads: int
    head_dim: int
    ffn: int
    patch: int = 16
    merge: int = 2
    in_channels: int = 3
    out_hidden: int = 2048
    ln_eps: float = 1e-6
    rope_theta: float = 10000.0
    dtype: str = "bf16"

    def with_(self, **kw) -> "VisionDims":
        return dataclasses.replace(self, **kw)

    def tokens_per_image(self, h: int, w: int) -> int:
        s = self.patch * self.merge
        return (h // s) * (w // s)

    def patches_per_image(self, h: int, w: int) -> int:
        return (h // self.patch) * (w // self.patch)


# A ViT of the width that feeds a 2048-wide decoder (24 blocks of 1024, 16
# heads of 64, MLP 4096, 16-pixel patches merged 2x2), and a tiny fp32 one.
VDIMS_FULL = VisionDims(depth=24, hidden=1024, n_heads=16, head_dim=64, ffn=4096)
VDIMS_TINY = VisionDims(depth=2, hidden=128, n_heads=2, head_dim=64, ffn=256, out_hidden=256, dtype="f32")


def _bias(rng, n, std=0.02):
    return _normal(rng, (n,), std)


def block_weights(v: VisionDims, layer: int) -> Dict[str, np.ndarray]:
    rng = np.random.default_rng([1, layer])
    D, F = v.hidden, v.ffn
    w = {
        "ln1_g": _gain(rng, D), "ln1_b": _bias(rng, D, 0.1),
        "w_qkv": _normal(rng, (3 * D, D)), "b_qkv": _bias(rng, 3 * D),
        "w_o": _normal(rng, (D, D)), "b_o": _bias(rng, D),
        "ln2_g": _gain(rng, D), "ln2_b": _bias(rng, D, 0.1),
        "w_fc1": _normal(rng, (F, D)), "b_fc1": _bias(rng, F),
        "w_fc2": _normal(rng, (D, F)), "b_fc2": _bias(rng, D),
    }
    return {k: _store(x, v.dtype) for k, x in w.items()}


def outer_weights(v: VisionDims) -> Dict[str, np.ndarray]:
    rng = np.random.default_rng([1, 10_000])
    D, mm = v.hidden, v.merge * v.merge
    kp = v.in_channels * v.patch * v.patch
    w = {
        "patch_w": _normal(rng, (D, kp)), "patch_b": _bias(rng, D),
        "merge_ln_g": _gain(rng, D), "merge_ln_b": _bias(rng, D, 0.1),
        "merge_w1": _normal(rng, (mm * D, mm * D)), "merge_b1": _bias(rng, mm * D),
        "merge_w2": _normal(rng, (v.out_hidden, mm * D)), "merge_b2": _bias(rng, v.out_hidden),
    }
    return {k: _store(x, v.dtype) for k, x in w.items()}


def images(v: VisionDims, n: int, h: int, w: int) -> np.ndarray:
    """[n, C, h, w] normalised pixels, image f from seed 2000 + f."""
    out = np.stack([np.random.default_rng(2000 + f).standard_normal((v.in_channels, h, w), dtype=np.float32)
                    for f in range(n)]) if n else np.zeros((0, v.in_channels, h, w), np.float32)
    return _store(out, v.dtype)

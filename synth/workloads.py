"""Workload definitions and seeded generators for the text-encoder prefill.

The paper measures its text encoder (a Qwen3-VL-2B-class decoder stack,
Sec. III-A) on DAVIS-2017 frames with style instructions (Sec. IV-A); neither
the frames nor the trained weights are available, so these generators stand
in for them with synthetic draws of the same token-level shape:

* one frame = a 2-D grid of merged image-patch tokens (8x8 for a 256x256
  source at patch 16 with a 2x2 merge, 16x16 for 512x512) followed by the
  instruction tokens;
* frames are batched and packed back to back, as in the batched text-encoder
  dispatch of Sec. III-B;
* linear weights and embeddings are N(0, 0.02); norm gains are
  1 + U(-0.5, 0.5), so that a dropped gain is visible in any comparison.

Seeds: layer ``l``'s weights come from ``default_rng([0, l])``, the final norm
gain from ``default_rng([0, 10_000])``, frame ``f``'s image tokens from
``default_rng(1000 + f)``, the instruction tokens from ``default_rng(7)`` and
the mixed-length draw from ``default_rng(11)``.

Values are drawn in float32 and, for bf16 workloads, rounded to the nearest
bf16 (ties to even) so that both the oracle and the HIP path see exactly the
same numbers.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Sequence, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class Dims:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rms_eps: float = 1e-6
    rope_theta: float = 5e6
    mrope_section: Tuple[int, int, int] = (24, 20, 20)
    mrope_layout: int = 0  # 0: contiguous sections, 1: interleaved
    qk_norm: int = 1
    dtype: str = "bf16"  # storage type of weights / embeddings: "f32" | "bf16"

    def with_(self, **kw) -> "Dims":
        return dataclasses.replace(self, **kw)

    @property
    def params_per_layer(self) -> int:
        d, hq, hkv, hd, f = (self.hidden, self.n_q_heads, self.n_kv_heads,
                             self.head_dim, self.ffn)
        return d * (hq + 2 * hkv) * hd + hq * hd * d + 3 * d * f


@dataclasses.dataclass(frozen=True)
class SeqLayout:
    """Token layout of one packed sequence: text, then an image grid, then text."""
    n_text_before: int
    grid_t: int
    grid_h: int
    grid_w: int
    n_text_after: int

    @property
    def n_image(self) -> int:
        return self.grid_t * self.grid_h * self.grid_w

    @property
    def length(self) -> int:
        return self.n_text_before + self.n_image + self.n_text_after


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dims: Dims
    layouts: Tuple[SeqLayout, ...]

    @property
    def batch(self) -> int:
        return len(self.layouts)

    @property
    def tokens(self) -> int:
        return sum(s.length for s in self.layouts)


# Tiny fp32 decoder: 2 layers, hidden 256, 4 q / 2 kv heads, head_dim 64,
# FFN 768, rotary pairs 12/10/10.
DIMS_TINY = Dims(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                 ffn=768, mrope_section=(12, 10, 10), dtype="f32")
# Full-width Qwen3-VL-2B-class decoder layer: hidden 2048, 16 q / 8 kv heads,
# head_dim 128, FFN 6144, rotary pairs 24/20/20; 28 layers in the stack.
DIMS_FULL = Dims(n_layers=28, hidden=2048, n_q_heads=16, n_kv_heads=8,
                 head_dim=128, ffn=6144, mrope_section=(24, 20, 20), dtype="bf16")

FRAME_96 = SeqLayout(0, 1, 8, 8, 32)     # 256x256 source: 8x8 grid + 32 text
FRAME_320 = SeqLayout(0, 1, 16, 16, 64)  # 512x512 source: 16x16 grid + 64 text


def grid_for_length(length: int, n_text_min: int = 32) -> Tuple[int, int]:
    """Largest grid gh x gw with 8 <= gh, gw <= 16 and gh*gw <= length - n_text_min.

    Ties in area go to the squarer grid, then to the taller one.
    """
    best = None
    for gh in range(8, 17):
        for gw in range(8, 17):
            area = gh * gw
            if area > length - n_text_min:
                continue
            key = (area, -abs(gh - gw), gh)
            if best is None or key > best[0]:
                best = (key, (gh, gw))
    if best is None:
        raise ValueError(f"length {length} too short for an 8x8 grid")
    return best[1]


def mixed_layouts(batch: int = 32, lo: int = 96, hi: int = 320, seed: int = 11) -> Tuple[SeqLayout, ...]:
    rng = np.random.default_rng(seed)
    lens = rng.integers(lo, hi + 1, size=batch)
    out = []
    for L in lens.tolist():
        gh, gw = grid_for_length(L)
        out.append(SeqLayout(0, 1, gh, gw, L - gh * gw))
    return tuple(out)


def _wl(name: str, dims: Dims, layouts: Sequence[SeqLayout]) -> Workload:
    return Workload(name, dims, tuple(layouts))


WORKLOADS: Dict[str, Workload] = {
    # fp32 parity case: 16 image tokens (4x4 grid at t=0) + 16 text tokens
    "tiny_fp32": _wl("tiny_fp32", DIMS_TINY, [SeqLayout(0, 1, 4, 4, 16)]),
    # one full-width layer, one 96-token frame
    "layer1_b1": _wl("layer1_b1", DIMS_FULL.with_(n_layers=1), [FRAME_96]),
    # 28-layer stack, single frame: weight-streaming regime
    "stack_b1": _wl("stack_b1", DIMS_FULL, [FRAME_96]),
    # 28-layer stack, batched frames of 96 tokens
    "stack_b8": _wl("stack_b8", DIMS_FULL, [FRAME_96] * 8),
    "stack_b16": _wl("stack_b16", DIMS_FULL, [FRAME_96] * 16),
    # 28-layer stack, 32 frames of 320 tokens (512x512 source)
    "stack_b32_l320": _wl("stack_b32_l320", DIMS_FULL, [FRAME_320] * 32),
    # 28-layer stack, 32 frames of lengths U{96..320}
    "stack_mixed32": _wl("stack_mixed32", DIMS_FULL, mixed_layouts()),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), kept as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return round_to_bf16(x) if dtype == "bf16" else np.ascontiguousarray(x, np.float32)


def _normal(rng, shape, std=0.02) -> np.ndarray:
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)


def _gain(rng, n) -> np.ndarray:
    return (1.0 + rng.uniform(-0.5, 0.5, size=n)).astype(np.float32)


def layer_weights(dims: Dims, layer: int) -> Dict[str, np.ndarray]:
    """Weights of one decoder layer, nn.Linear layout [out_features, in_features]."""
    rng = np.random.default_rng([0, layer])
    d, hq, hkv, hd, f = dims.hidden, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.ffn
    w = {
        "attn_norm": _gain(rng, d),
        "w_q": _normal(rng, (hq * hd, d)),
        "w_k": _normal(rng, (hkv * hd, d)),
        "w_v": _normal(rng, (hkv * hd, d)),
        "q_norm": _gain(rng, hd),
        "k_norm": _gain(rng, hd),
        "w_o": _normal(rng, (d, hq * hd)),
        "mlp_norm": _gain(rng, d),
        "w_gate": _normal(rng, (f, d)),
        "w_up": _normal(rng, (f, d)),
        "w_down": _normal(rng, (d, f)),
    }
    return {k: _store(v, dims.dtype) for k, v in w.items()}


def final_norm_gain(dims: Dims) -> np.ndarray:
    return _store(_gain(np.random.default_rng([0, 10_000]), dims.hidden), dims.dtype)


def seq_lens(layouts: Sequence[SeqLayout]) -> List[int]:
    return [s.length for s in layouts]


def embeddings(dims: Dims, layouts: Sequence[SeqLayout], std: float = 0.02,
               outliers: int = 0) -> np.ndarray:
    """Packed [T, hidden] input embeddings.

    Frame ``f``'s image tokens are fresh draws from seed ``1000 + f``; the
    instruction tokens (before and after the image) are the leading rows of
    one draw from seed 7, so every frame carries the same instruction.
    ``outliers`` > 0 plants that many entries of magnitude 1160 per frame
    (the wide activation range the paper reports for the trained encoder),
    at positions drawn from seed ``5000 + f``.
    """
    D = dims.hidden
    max_text = max([s.n_text_before + s.n_text_after for s in layouts] + [1])
    text = _normal(np.random.default_rng(7), (max_text, D), std)
    rows = []
    for f, s in enumerate(layouts):
        img = _normal(np.random.default_rng(1000 + f), (s.n_image, D), std)
        seq = np.concatenate([text[:s.n_text_before], img,
                              text[s.n_text_before:s.n_text_before + s.n_text_after]], axis=0)
        if outliers:
            r = np.random.default_rng(5000 + f)
            idx = r.integers(0, seq.size, size=outliers)
            sign = np.where(r.integers(0, 2, size=outliers) == 0, -1.0, 1.0)
            seq = seq.copy()
            seq.reshape(-1)[idx] = (1160.0 * sign).astype(np.float32)
        rows.append(seq)
    x = np.concatenate(rows, axis=0) if rows else np.zeros((0, D), np.float32)
    return _store(x, dims.dtype)

"""Plain fp64 CPU oracle of the text-encoder prefill forward.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import or call this
module: only the tests, the smoke check and the benchmark's CPU-baseline leg
use it. It shares no code with the HIP path; the only shared module is the
seeded input generator (``synth``), which holds none of the arithmetic.

What it computes. The paper's text encoder is a Qwen3-VL decoder that jointly
attends to the image-patch tokens of the source frame and the instruction
tokens (Sec. I; Sec. III-A), run once per batch of buffered frames with each
frame an independent sequence (Sec. III-B, "Asymmetric batched dispatch";
Table "tab:batch"). The paper gives no layer-level formula, so the oracle
writes out the standard pre-norm decoder stack such a model is defined by:

    for each layer:
        a = RMSNorm(x) * g_attn
        q, k, v = a Wq^T, a Wk^T, a Wv^T                 (no biases)
        q, k = RMSNorm_d(q) * g_q, RMSNorm_d(k) * g_k    (per head, optional)
        q, k = M-RoPE(q, pos), M-RoPE(k, pos)
        o = softmax(q k^T / sqrt(d) + causal mask) v     (per sequence, GQA)
        x = x + o Wo^T
        m = RMSNorm(x) * g_mlp
        x = x + (silu(m Wg^T) * (m Wu^T)) Wd^T
    out = RMSNorm(x) * g_final

Readings where the paper is silent (each a choice the paper leaves open):
rotate-half pairing (element j with j + d/2); inverse frequencies
theta^(-2j/d); rotary pairs split into contiguous t/h/w sections, or the
interleaved assignment; positions of image tokens (t, h, w) on the merged
grid offset by the preceding text, text after an image starting at one past
the largest earlier position; contiguous GQA grouping; RMSNorm with eps inside
the square root and a plain gain; scale 1/sqrt(d); no cross-sequence
attention.

Everything is computed in float64 from the (float32 / bf16-exact) inputs; the
oracle never rounds to a narrower type.
"""
from __future__ import annotations

from typing import Callable, Dict, Iterable, List, Sequence

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------- positions
def positions(layouts: Sequence) -> np.ndarray:
    """3-D (t, h, w) rotary positions of a packed batch -> int64 [3, T].

    Per sequence (Sec. III-A: the instruction and the source image are one
    sequence): text tokens before the image count up t = h = w = i; image
    token k of a (gt, gh, gw) grid starting after ``o`` text tokens sits at
    (o + k // (gh*gw), o + (k // gw) % gh, o + k % gw); text after the image
    starts at one past the largest position used so far and counts up.
    """
    cols: List[np.ndarray] = []
    for s in layouts:
        p = []
        for i in range(s.n_text_before):
            p.append((i, i, i))
        o = s.n_text_before
        plane = s.grid_h * s.grid_w
        for k in range(s.grid_t * plane):
            p.append((o + k // plane, o + (k // s.grid_w) % s.grid_h, o + k % s.grid_w))
        nxt = (max(max(t) for t in p) + 1) if p else 0
        for j in range(s.n_text_after):
            p.append((nxt + j,) * 3)
        cols.append(np.array(p, dtype=np.int64).reshape(-1, 3).T)
    if not cols:
        return np.zeros((3, 0), np.int64)
    return np.concatenate(cols, axis=1)


# ------------------------------------------------------------------ M-RoPE
def inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """theta^(-2j/d) for rotary pair j = 0 .. d/2-1."""
    j = np.arange(head_dim // 2, dtype=F64)
    return np.power(F64(theta), -2.0 * j / head_dim)


def pair_axis(head_dim: int, section: Sequence[int], layout: int) -> np.ndarray:
    """Which position axis (0 = t, 1 = h, 2 = w) drives each rotary pair.

    layout 0: contiguous sections [t]*s_t + [h]*s_h + [w]*s_w.
    layout 1: interleaved: pair j is h if j % 3 == 1 and j < 3*s_h, w if
    j % 3 == 2 and j < 3*s_w, t otherwise.
    """
    half = head_dim // 2
    if sum(section) != half:
        raise ValueError("rotary sections must sum to head_dim / 2")
    if layout == 0:
        return np.array([0] * section[0] + [1] * section[1] + [2] * section[2], np.int64)
    ax = np.zeros(half, np.int64)
    for j in range(half):
        if j % 3 == 1 and j < 3 * section[1]:
            ax[j] = 1
        elif j % 3 == 2 and j < 3 * section[2]:
            ax[j] = 2
    return ax


def mrope(z: np.ndarray, pos: np.ndarray, head_dim: int, theta: float,
          section: Sequence[int], layout: int) -> np.ndarray:
    """Rotate z [L, H, d] by the multimodal rotary embedding.

    Pair j = (z_j, z_{j+d/2}) of token i turns by phi = p * theta^(-2j/d),
    p the token's position on the pair's axis:
    (u, w) -> (u cos phi - w sin phi, w cos phi + u sin phi).
    """
    half = head_dim // 2
    ax = pair_axis(head_dim, section, layout)
    f = inv_freq(head_dim, theta)
    p = pos[ax, :].T.astype(F64)              # [L, half]
    phi = p * f[None, :]
    c, s = np.cos(phi)[:, None, :], np.sin(phi)[:, None, :]
    u, w = z[..., :half], z[..., half:]
    return np.concatenate([u * c - w * s, w * c + u * s], axis=-1)


# ------------------------------------------------------------ small pieces
def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = x.astype(F64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g.astype(F64)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """One sequence: q [L, Hq, d], k/v [L, Hkv, d] -> o [L, Hq, d].

    Query head h reads key/value head h // (Hq / Hkv). Scores are scaled by
    1/sqrt(d); token i attends to tokens j <= i of its own sequence.
    """
    L, hq, d = q.shape
    hkv = k.shape[1]
    rep = hq // hkv
    o = np.empty((L, hq, d), F64)
    mask = np.triu(np.ones((L, L), bool), k=1)
    for h in range(hq):
        kh, vh = k[:, h // rep, :], v[:, h // rep, :]
        s = (q[:, h, :] @ kh.T) / np.sqrt(F64(d))
        s = np.where(mask, -np.inf, s)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        o[:, h, :] = p @ vh
    return o


# ------------------------------------------------------------------ layers
def layer_forward(x: np.ndarray, pos: np.ndarray, seq_lens: Sequence[int],
                  w: Dict[str, np.ndarray], dims) -> np.ndarray:
    """One decoder layer on the packed residual stream x [T, D] (float64)."""
    hq, hkv, hd = dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    W = {k: v.astype(F64) for k, v in w.items()}
    x = x.astype(F64)
    T = x.shape[0]
    a = rmsnorm(x, W["attn_norm"], dims.rms_eps)
    q = (a @ W["w_q"].T).reshape(T, hq, hd)
    k = (a @ W["w_k"].T).reshape(T, hkv, hd)
    v = (a @ W["w_v"].T).reshape(T, hkv, hd)
    if dims.qk_norm:
        q = rmsnorm(q, W["q_norm"], dims.rms_eps)
        k = rmsnorm(k, W["k_norm"], dims.rms_eps)
    q = mrope(q, pos, hd, dims.rope_theta, dims.mrope_section, dims.mrope_layout)
    k = mrope(k, pos, hd, dims.rope_theta, dims.mrope_section, dims.mrope_layout)
    o = np.empty((T, hq, hd), F64)
    start = 0
    for L in seq_lens:
        sl = slice(start, start + L)
        o[sl] = causal_attention(q[sl], k[sl], v[sl])
        start += L
    x = x + o.reshape(T, hq * hd) @ W["w_o"].T
    m = rmsnorm(x, W["mlp_norm"], dims.rms_eps)
    x = x + (silu(m @ W["w_gate"].T) * (m @ W["w_up"].T)) @ W["w_down"].T
    return x


def encode(embeds: np.ndarray, pos: np.ndarray, seq_lens: Sequence[int], dims,
           layer_weights: Callable[[int], Dict[str, np.ndarray]],
           final_norm: np.ndarray, n_layers: int | None = None,
           keep: Iterable[int] = ()) -> np.ndarray:
    """Whole stack: embeddings [T, D] -> final-norm hidden states [T, D].

    ``layer_weights(l)`` supplies layer l's weights (so a long stack can be
    streamed); ``keep`` lists layer indices whose *input* residual stream is
    stored in ``encode.kept`` for per-layer comparisons.
    """
    if sum(seq_lens) != embeds.shape[0] or pos.shape[1] != embeds.shape[0]:
        raise ValueError("sequence lengths, positions and embeddings disagree")
    x = embeds.astype(F64)
    keep = set(keep)
    encode.kept = {}
    for l in range(dims.n_layers if n_layers is None else n_layers):
        if l in keep:
            encode.kept[l] = x.copy()
        x = layer_forward(x, pos, seq_lens, layer_weights(l), dims)
    return rmsnorm(x, final_norm, dims.rms_eps)


encode.kept = {}

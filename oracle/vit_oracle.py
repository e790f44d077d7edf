"""Plain fp64 CPU oracle of the vision tower (images -> image tokens).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle``: only the tests, the
smoke check and the benchmark's CPU-baseline leg may use it. It shares no
code with the HIP path.

What it computes. The paper's text encoder receives the 256x256 source patch
through Qwen3-VL's vision tower, whose output fills the prompt's image
placeholder with the image tokens the decoder attends to (Sec. I; Sec. III-A
"Notation and Setup"). The paper gives no architecture, so this writes out
the plain pre-norm ViT with a patch merger that such a tower is defined by,
with these readings (each a choice the paper leaves open):

    patch vectors: C x patch x patch pixels in (channel, row, column) order,
        patches enumerated in merge-group order (groups of merge x merge
        patches row-major over the image, row-major inside a group)
    x = patches W_patch^T + b_patch
    per block:  a = LN(x) g1 + b1;  q, k, v = split(a W_qkv^T + b_qkv)
                q, k = RoPE2d(q, k)  (pair j of a head: patch row for j < d/4,
                                      patch column otherwise, theta^(-2j/d))
                o = softmax(q k^T / sqrt(d)) v   over all patches of the image
                x = x + o W_o^T + b_o
                m = LN(x) g2 + b2;  x = x + gelu(m W_fc1^T + b_fc1) W_fc2^T + b_fc2
    merger:     u = the merge x merge normalised patches of a group, concatenated
                tokens = gelu(u W_m1^T + b_m1) W_m2^T + b_m2

LN(x) = (x - mean) / sqrt(var + eps) (biased variance); gelu is the tanh form.
"""
from __future__ import annotations

from typing import Callable, Dict, Iterable, Sequence

import numpy as np

from .te_oracle import mrope

F64 = np.float64


def patch_grid(h: int, w: int, patch: int, merge: int):
    """(row, column) of every patch of an h x w image, in merge-group order."""
    gh, gw = h // (patch * merge), w // (patch * merge)
    rows, cols = [], []
    for gr in range(gh):
        for gc in range(gw):
            for dr in range(merge):
                for dc in range(merge):
                    rows.append(gr * merge + dr)
                    cols.append(gc * merge + dc)
    return np.array(rows, np.int64), np.array(cols, np.int64)


def patchify(images: np.ndarray, patch: int, merge: int) -> np.ndarray:
    """[n, C, h, w] -> [n * patches, C * patch * patch] in merge-group order."""
    n, C, h, w = images.shape
    rows, cols = patch_grid(h, w, patch, merge)
    out = []
    for i in range(n):
        for r, c in zip(rows, cols):
            out.append(images[i, :, r * patch:(r + 1) * patch, c * patch:(c + 1) * patch].reshape(-1))
    return np.asarray(out, F64).reshape(n * len(rows), C * patch * patch)


def layernorm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    x = x.astype(F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g.astype(F64) + b.astype(F64)


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def rope2d(z: np.ndarray, rows: np.ndarray, cols: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """z [L, H, d] rotated by the 2-D rotary embedding: the multimodal rotary
    embedding with no t pairs, d/4 row pairs and d/4 column pairs."""
    pos = np.stack([np.zeros_like(rows), rows, cols])
    q = head_dim // 4
    return mrope(z, pos, head_dim, theta, (0, q, q), 0)


def full_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """One image: q, k, v [L, H, d] -> o [L, H, d], every patch attends to all."""
    L, H, d = q.shape
    o = np.empty((L, H, d), F64)
    for h in range(H):
        s = (q[:, h, :] @ k[:, h, :].T) / np.sqrt(F64(d))
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        o[:, h, :] = (p / p.sum(axis=1, keepdims=True)) @ v[:, h, :]
    return o


def block_forward(x: np.ndarray, rows, cols, per_image: int, w: Dict[str, np.ndarray], v) -> np.ndarray:
    """One ViT block on the packed residual stream x [n * per_image, D]."""
    W = {k: a.astype(F64) for k, a in w.items()}
    x = x.astype(F64)
    T, D = x.shape
    H, hd = v.n_heads, v.head_dim
    a = layernorm(x, W["ln1_g"], W["ln1_b"], v.ln_eps)
    qkv = a @ W["w_qkv"].T + W["b_qkv"]
    q, k, vv = (qkv[:, i * D:(i + 1) * D].reshape(T, H, hd) for i in range(3))
    rr, cc = np.tile(rows, T // per_image), np.tile(cols, T // per_image)
    q = rope2d(q, rr, cc, hd, v.rope_theta)
    k = rope2d(k, rr, cc, hd, v.rope_theta)
    o = np.empty((T, H, hd), F64)
    for s in range(0, T, per_image):
        sl = slice(s, s + per_image)
        o[sl] = full_attention(q[sl], k[sl], vv[sl])
    x = x + o.reshape(T, D) @ W["w_o"].T + W["b_o"]
    m = layernorm(x, W["ln2_g"], W["ln2_b"], v.ln_eps)
    return x + gelu_tanh(m @ W["w_fc1"].T + W["b_fc1"]) @ W["w_fc2"].T + W["b_fc2"]


def merge_tokens(x: np.ndarray, outer: Dict[str, np.ndarray], v) -> np.ndarray:
    """Final residual stream [T, D] -> image tokens [T / merge^2, out_hidden]."""
    W = {k: a.astype(F64) for k, a in outer.items()}
    T, D = x.shape
    mm = v.merge * v.merge
    y = layernorm(x, W["merge_ln_g"], W["merge_ln_b"], v.ln_eps)
    u = np.stack([np.concatenate([y[t * mm + j] for j in range(mm)]) for t in range(T // mm)])
    return gelu_tanh(u @ W["merge_w1"].T + W["merge_b1"]) @ W["merge_w2"].T + W["merge_b2"]


def encode(images: np.ndarray, v, block_weights: Callable[[int], Dict[str, np.ndarray]],
           outer: Dict[str, np.ndarray], depth: int | None = None, keep: Iterable[int] = ()) -> np.ndarray:
    """[n, C, h, w] images -> [n * tokens per image, out_hidden] image tokens.
    ``keep`` lists blocks whose input residual stream goes to ``encode.kept``."""
    n, _, h, w = images.shape
    rows, cols = patch_grid(h, w, v.patch, v.merge)
    per = len(rows)
    x = patchify(images, v.patch, v.merge) @ outer["patch_w"].astype(F64).T + outer["patch_b"].astype(F64)
    keep = set(keep)
    encode.kept = {}
    for l in range(v.depth if depth is None else depth):
        if l in keep:
            encode.kept[l] = x.copy()
        x = block_forward(x, rows, cols, per, block_weights(l), v)
    encode.kept["final"] = x.copy()
    return merge_tokens(x, outer, v)

"""Shared helpers of the GPU tests: seeded workloads -> device encoder, and the
error metric max|gpu - oracle| / rms(oracle) used for every float comparison."""
from __future__ import annotations

import functools

import numpy as np

from oracle import te_oracle as O
from synth import workloads as W


def rel_err(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.abs(got - ref).max() / np.sqrt(np.mean(ref * ref)))


@functools.lru_cache(maxsize=None)
def layer_w(dims: W.Dims, layer: int):
    return W.layer_weights(dims, layer)


@functools.lru_cache(maxsize=None)
def final_g(dims: W.Dims):
    return W.final_norm_gain(dims)


def layer_w_e4m3(dims: W.Dims, layer: int):
    """The layer's weights with every linear weight replaced by its e4m3
    dequantised value (oracle quantiser), float64. Weights depend on the
    layer index and the shapes, not on the number of layers."""
    return _layer_w_e4m3(dims.with_(n_layers=1), layer)


@functools.lru_cache(maxsize=4)
def _layer_w_e4m3(dims: W.Dims, layer: int):
    from oracle import e4m3 as Q
    w = dict(layer_w(dims, layer))
    for k in ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down"):
        codes, scales = Q.quantize_rows(w[k])
        w[k] = Q.dequantize_rows(codes, scales)
    return w


def config_for(B, dims: W.Dims, max_tokens=4096, max_batch=64, max_seq=4096, out_dtype=None,
               weight_format=0):
    dt = B.MTE_BF16 if dims.dtype == "bf16" else B.MTE_F32
    return B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads, dims.head_dim,
                         dims.ffn, rms_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                         mrope_section=dims.mrope_section, mrope_layout=dims.mrope_layout,
                         qk_norm=dims.qk_norm, dtype=dt, out_dtype=dt if out_dtype is None else out_dtype,
                         max_tokens=max_tokens, max_batch=max_batch, max_seq=max_seq,
                         weight_format=weight_format)


def make_encoder(dims: W.Dims, **kw):
    """Device encoder for `dims`; its output is fp32 unless out_dtype says otherwise, so that
    comparisons measure the computation rather than the rounding of the result."""
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder
    kw.setdefault("out_dtype", B.MTE_F32)
    cfg = config_for(B, dims, **kw)
    return TextEncoder.from_host(cfg, (layer_w(dims, l) for l in range(dims.n_layers)), final_g(dims))


def layout_tuples(layouts):
    return [(s.n_text_before, s.grid_t, s.grid_h, s.grid_w, s.n_text_after) for s in layouts]


def oracle_encode(dims: W.Dims, emb: np.ndarray, layouts, keep=()):
    pos = O.positions(layouts)
    return O.encode(emb, pos, W.seq_lens(layouts), dims, lambda l: layer_w(dims, l), final_g(dims),
                    keep=keep)


def seq_slices(layouts):
    out, s = [], 0
    for L in W.seq_lens(layouts):
        out.append(slice(s, s + L))
        s += L
    return out

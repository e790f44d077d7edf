"""e4m3 weights (MTE_WEIGHTS_E4M3) on the GPU, through the C ABI.

The quantiser is integer work: codes and row scales are compared bit for bit
with the oracle's (oracle/e4m3.py, a nearest-value search). The forward with
e4m3 weights computes the same function as the bf16 path with every linear
weight replaced by its dequantised value, so it is held to the same bars
against the fp64 oracle run on the oracle's own dequantised weights: <= 1e-2
(max|gpu - oracle| / rms(oracle)) for one layer, <= 3e-2 for a stack.
How far e4m3 weights move the output from the bf16 model is a property of
the format, not of the kernels; it is printed, and only checked for sanity.
"""
import sys

import numpy as np
import pytest

from oracle import e4m3 as Q
from oracle import te_oracle as O
from synth import workloads as W
from tests.gpu_common import (final_g, layer_w, layer_w_e4m3, layout_tuples, make_encoder, rel_err,
                              seq_slices)

pytestmark = pytest.mark.gpu

TOL_LAYER = 1e-2
TOL_STACK = 3e-2
E4M3 = 1


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "no GPU"
    return t


def _bf16(x):
    return W.round_to_bf16(np.asarray(x, np.float32))


@pytest.mark.parametrize("shape,src", [((1, 1), "bf16"), ((7, 300), "bf16"), ((64, 2048), "f32"),
                                       ((6144, 2048), "bf16")])
def test_quantizer_bit_exact(torch, shape, src):
    from paper_2606_05981_amd.encoder import quantize_e4m3_rows
    rng = np.random.default_rng(shape[0] * 7 + shape[1])
    rows, cols = shape
    w = rng.normal(0, 0.02, shape)
    if rows >= 7:
        w[1] = 0.0                                   # all-zero row
        w[2] *= 1e-25                                # tiny row (bf16 keeps fp32's exponent range)
        w[3, cols // 2] = 1e4                        # outlier
        w[4] = 448.0 * rng.integers(-8, 9, cols) / 8  # exact codes, and 448 itself
        w[5] = rng.choice([-1, 1], cols) * (Q.decode_table()[1:0x7E] + Q.decode_table()[2:0x7F])[
            rng.integers(0, 125, cols)] / 2 * 2.0 ** -3   # midpoints of the row's grid
        w[5, 0] = 448.0 * 2.0 ** -3
    w = _bf16(w) if src == "bf16" else w.astype(np.float32)
    _say("quantize", shape, src)
    dt = torch.bfloat16 if src == "bf16" else torch.float32
    codes, scales = quantize_e4m3_rows(torch.from_numpy(w).to("cuda", dt))
    torch.cuda.synchronize()
    ref_c, ref_s = Q.quantize_rows(w)
    assert np.array_equal(scales.cpu().numpy().astype(np.float64), ref_s)
    got = codes.cpu().numpy()
    bad = np.argwhere(got != ref_c)
    assert bad.size == 0, (bad[:5], got[tuple(bad[0])], ref_c[tuple(bad[0])])


def _encode_layers(torch, enc, x, layouts, l0, l1):
    from paper_2606_05981_amd.encoder import build_positions
    h = enc.encode_layers(torch.from_numpy(x.astype(np.float32)).cuda(), build_positions(layout_tuples(layouts)),
                          W.seq_lens(layouts), l0, l1)
    torch.cuda.synchronize()
    return h.cpu().numpy()


@pytest.mark.parametrize("frames", [1, 2, 16])
def test_e4m3_one_layer(torch, frames):
    """Residual stream after one full-size layer (96, 192 and 1536 rows: the GEMM plans of a
    batch of one, two and sixteen frames) against the oracle on dequantised weights."""
    dims = W.DIMS_FULL.with_(n_layers=1)
    layouts = [W.workload("stack_b1").layouts[0]] * frames
    emb = W.embeddings(dims, layouts)
    pos = O.positions(layouts)
    _say("e4m3 one layer, frames", frames)
    enc = make_encoder(dims, weight_format=E4M3)
    got = _encode_layers(torch, enc, emb, layouts, 0, 1)
    enc.close()
    ref = O.layer_forward(emb, pos, W.seq_lens(layouts), layer_w_e4m3(dims, 0), dims)
    err = rel_err(got, ref)
    _say("  err vs dequantised oracle", err)
    assert err <= TOL_LAYER
    if frames == 1:
        ref_bf16 = O.layer_forward(emb, pos, W.seq_lens(layouts), layer_w(dims, 0), dims)
        d = got - emb
        d0 = ref_bf16 - emb
        q = float(np.sqrt(np.mean((d - d0) ** 2) / np.mean(d0 ** 2)))
        _say("  rms change of the layer's update vs bf16 weights", q)
        assert q < 0.2


def test_e4m3_two_layer_stack(torch):
    """Two full-size layers and the final norm, one and two frames (the encoder's whole
    e4m3 path: quantisation at creation, the layer loop, the output)."""
    dims = W.DIMS_FULL.with_(n_layers=2)
    enc = make_encoder(dims, weight_format=E4M3)
    from paper_2606_05981_amd.encoder import build_positions
    for frames in (1, 2):
        layouts = [W.workload("stack_b1").layouts[0]] * frames
        emb = W.embeddings(dims, layouts)
        _say("e4m3 two layers, frames", frames)
        x = torch.from_numpy(emb).to("cuda", torch.bfloat16)
        out = enc.encode(x, build_positions(layout_tuples(layouts)), W.seq_lens(layouts))
        torch.cuda.synchronize()
        got = out.float().cpu().numpy()
        ref = O.encode(emb, O.positions(layouts), W.seq_lens(layouts), dims, lambda l: layer_w_e4m3(dims, l),
                       final_g(dims))
        err = rel_err(got, ref)
        _say("  err", err)
        assert err <= TOL_STACK
        for sl in seq_slices(layouts):
            assert rel_err(got[sl], ref[sl]) <= TOL_STACK
    enc.close()


def test_e4m3_graph_replays_match_eager(torch):
    """The e4m3 encoder (quantised at creation) captures into a graph like the bf16 one."""
    from paper_2606_05981_amd.encoder import build_positions
    dims = W.DIMS_FULL.with_(n_layers=2)
    layouts = [W.workload("stack_b1").layouts[0]] * 2
    x = torch.from_numpy(W.embeddings(dims, layouts)).to("cuda", torch.bfloat16)
    pos = build_positions(layout_tuples(layouts))
    lens = W.seq_lens(layouts)
    enc = make_encoder(dims, weight_format=E4M3)
    eager = enc.encode(x, pos, lens).clone()
    out = torch.empty_like(eager)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            enc.encode(x, pos, lens, out=out)
    torch.cuda.current_stream().wait_stream(s)
    for r in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), r
        enc.encode(x, pos, lens)
        torch.cuda.synchronize()
    enc.close()

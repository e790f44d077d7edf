"""Parity of the HIP path (through the C ABI) with the fp64 CPU oracle.

Tolerances (error = max|gpu - oracle| / rms(oracle) over all tokens and
channels): fp32 storage <= 1e-4; bf16 storage with fp32 accumulation
<= 1e-2 for one layer (residual stream after the layer, from the oracle's
exact layer input) and <= 3e-2 for the 28-layer stack output.
"""
import sys

import numpy as np
import pytest

from oracle import te_oracle as O
from synth import workloads as W
from tests.gpu_common import (final_g, layer_w, layout_tuples, make_encoder, oracle_encode,
                              rel_err, seq_slices)

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_LAYER = 1e-2
TOL_STACK = 3e-2


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "no GPU"
    return t


def _gpu_encode(torch, enc, dims, emb, layouts, raw=False):
    from paper_2606_05981_amd.encoder import build_positions
    dt = torch.bfloat16 if dims.dtype == "bf16" else torch.float32
    x = torch.from_numpy(emb).to("cuda", dt)
    pos = build_positions(layout_tuples(layouts))
    out = enc.encode(x, pos, W.seq_lens(layouts))
    torch.cuda.synchronize()
    return out.cpu() if raw else out.float().cpu().numpy()


# ------------------------------------------------------------ positions
@pytest.mark.parametrize("case", ["tiny", "frames96", "mixed32", "text_before", "temporal", "many"])
def test_positions_bit_exact(torch, case):
    from paper_2606_05981_amd.encoder import build_positions
    layouts = {
        "tiny": W.workload("tiny_fp32").layouts,
        "frames96": W.workload("stack_b16").layouts,
        "mixed32": W.workload("stack_mixed32").layouts,
        "text_before": (W.SeqLayout(3, 1, 2, 2, 2), W.SeqLayout(5, 0, 0, 0, 0), W.SeqLayout(0, 1, 3, 5, 0)),
        "temporal": (W.SeqLayout(2, 3, 4, 2, 7), W.SeqLayout(0, 2, 2, 2, 1)),
        "many": tuple(W.SeqLayout(i % 3, 1, 1 + i % 4, 2, i % 5) for i in range(300)),
    }[case]
    _say("positions", case)
    got = build_positions(layout_tuples(layouts)).cpu().numpy()
    np.testing.assert_array_equal(got, O.positions(layouts))


# ------------------------------------------------------- tiny fp32 stack
@pytest.mark.parametrize("mrope_layout,qk_norm", [(0, 1), (1, 1), (0, 0)])
def test_tiny_fp32_stack(torch, mrope_layout, qk_norm):
    wl = W.workload("tiny_fp32")
    dims = wl.dims.with_(mrope_layout=mrope_layout, qk_norm=qk_norm)
    _say("tiny fp32", mrope_layout, qk_norm)
    emb = W.embeddings(dims, wl.layouts)
    enc = make_encoder(dims)
    got = _gpu_encode(torch, enc, dims, emb, wl.layouts)
    enc.close()
    err = rel_err(got, oracle_encode(dims, emb, wl.layouts))
    _say("  err", err)
    assert err <= TOL_F32


def test_tiny_fp32_ragged_edges(torch):
    """Lengths 1, 2, tile edges +-1 and text-only sequences in one packed batch."""
    dims = W.DIMS_TINY
    layouts = (W.SeqLayout(1, 0, 0, 0, 0), W.SeqLayout(0, 1, 1, 1, 1), W.SeqLayout(0, 1, 4, 4, 15),
               W.SeqLayout(0, 1, 4, 4, 16), W.SeqLayout(0, 1, 4, 4, 17), W.SeqLayout(3, 1, 6, 5, 30),
               W.SeqLayout(64, 0, 0, 0, 1), W.SeqLayout(0, 1, 8, 8, 33), W.SeqLayout(2, 2, 4, 4, 100))
    emb = W.embeddings(dims, layouts)
    _say("tiny ragged", W.seq_lens(layouts))
    enc = make_encoder(dims)
    got = _gpu_encode(torch, enc, dims, emb, layouts)
    enc.close()
    ref = oracle_encode(dims, emb, layouts)
    for sl in seq_slices(layouts):
        assert rel_err(got[sl], ref[sl]) <= TOL_F32, sl
    assert rel_err(got, ref) <= TOL_F32


def test_tiny_fp32_many_short_sequences(torch):
    """300 sequences of 1..8 tokens in one packed batch: the attention launches in chunks of
    256 sequences and the position kernel in chunks of 128, so this crosses both chunk
    boundaries; every sequence must still see only itself."""
    dims = W.DIMS_TINY
    layouts = tuple(W.SeqLayout(1 + i % 3, 1 if i % 4 else 0, 1 if i % 4 else 0, 1 + i % 2 if i % 4 else 0,
                                i % 4) for i in range(300))
    lens = W.seq_lens(layouts)
    assert len(lens) > 256 and min(lens) >= 1
    emb = W.embeddings(dims, layouts)
    _say("tiny many", len(lens), sum(lens))
    enc = make_encoder(dims, max_tokens=4096, max_batch=512, max_seq=64)
    got = _gpu_encode(torch, enc, dims, emb, layouts)
    enc.close()
    ref = oracle_encode(dims, emb, layouts)
    assert rel_err(got, ref) <= TOL_F32
    sl = seq_slices(layouts)
    for i in (0, 127, 128, 255, 256, 299):
        assert rel_err(got[sl[i]], ref[sl[i]]) <= TOL_F32, i


def test_tiny_zero_layers_is_final_norm(torch):
    dims = W.DIMS_TINY.with_(n_layers=0)
    wl = W.workload("tiny_fp32")
    emb = W.embeddings(dims, wl.layouts)
    enc = make_encoder(dims)
    got = _gpu_encode(torch, enc, dims, emb, wl.layouts)
    enc.close()
    assert rel_err(got, O.rmsnorm(emb, final_g(dims), dims.rms_eps)) <= TOL_F32


# ----------------------------------------------------- one bf16 layer
def test_layer1_bf16_residual_after_layer(torch):
    wl = W.workload("layer1_b1")
    dims = wl.dims
    emb = W.embeddings(dims, wl.layouts)
    pos = O.positions(wl.layouts)
    _say("layer1 bf16 per-layer")
    enc = make_encoder(dims)
    from paper_2606_05981_amd.encoder import build_positions
    h_in = torch.from_numpy(emb.astype(np.float32)).cuda()
    h = enc.encode_layers(h_in, build_positions(layout_tuples(wl.layouts)), W.seq_lens(wl.layouts), 0, 1)
    torch.cuda.synchronize()
    ref = O.layer_forward(emb, pos, W.seq_lens(wl.layouts), layer_w(dims, 0), dims)
    err = rel_err(h.cpu().numpy(), ref)
    _say("  err", err)
    assert err <= TOL_LAYER
    got = _gpu_encode(torch, enc, dims, emb, wl.layouts)
    enc.close()
    err2 = rel_err(got, O.rmsnorm(ref, final_g(dims), dims.rms_eps))
    _say("  err(final norm)", err2)
    assert err2 <= TOL_LAYER


def test_bf16_output_is_rounded_fp32_result(torch):
    """With a bf16 output, each value is the fp32 result rounded to nearest even bf16: both
    encoders run the same kernels in the same order (K-split partial sums are added in
    split order), so the comparison is bit-exact."""
    from paper_2606_05981_amd import binding as B
    wl = W.workload("layer1_b1")
    dims = wl.dims
    emb = W.embeddings(dims, wl.layouts, std=37.0, outliers=6)
    e32 = make_encoder(dims)
    e16 = make_encoder(dims, out_dtype=B.MTE_BF16)
    y32 = _gpu_encode(torch, e32, dims, emb, wl.layouts, raw=True)
    y16 = _gpu_encode(torch, e16, dims, emb, wl.layouts, raw=True)
    e32.close(); e16.close()
    assert y16.dtype == torch.bfloat16
    assert torch.equal(y16, y32.to(torch.bfloat16))


def test_fp16_range_prescales(torch):
    """Norm gains x4096 push RMSNorm outputs, v and the SwiGLU product far past fp16's
    range (65504) and a down-projection x2^18 has weights beyond it: the power-of-two
    pre-scales chosen at creation from the static bounds keep every fp16 operand finite,
    and the layer still meets the per-layer tolerance."""
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder, build_positions
    wl = W.workload("layer1_b1")
    dims = wl.dims
    w = dict(layer_w(dims, 0))
    w["attn_norm"] = w["attn_norm"] * np.float32(4096.0)
    w["mlp_norm"] = w["mlp_norm"] * np.float32(4096.0)
    w["w_down"] = w["w_down"] * np.float32(2.0 ** 18)
    cfg = B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads, dims.head_dim,
                        dims.ffn, rms_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                        mrope_section=dims.mrope_section, dtype=B.MTE_BF16, out_dtype=B.MTE_F32,
                        max_tokens=256, max_batch=4, max_seq=256)
    enc = TextEncoder.from_host(cfg, [w], final_g(dims))
    emb = W.embeddings(dims, wl.layouts)
    pos = O.positions(wl.layouts)
    h = enc.encode_layers(torch.from_numpy(emb.astype(np.float32)).cuda(),
                          build_positions(layout_tuples(wl.layouts)), W.seq_lens(wl.layouts), 0, 1)
    torch.cuda.synchronize()
    enc.close()
    got = h.cpu().numpy()
    assert np.isfinite(got).all()
    ref = O.layer_forward(emb, pos, W.seq_lens(wl.layouts), w, dims)
    err = rel_err(got, ref)
    _say("  prescaled layer err", err)
    assert err <= TOL_LAYER


# --------------------------------------------------- 28-layer stacks
@pytest.fixture(scope="module")
def full_enc(torch):
    _say("building the 28-layer encoder")
    enc = make_encoder(W.DIMS_FULL, max_tokens=32 * 320, max_batch=64, max_seq=4096)
    yield enc
    enc.close()


def test_stack_b1_and_per_layer(torch, full_enc):
    wl = W.workload("stack_b1")
    dims = wl.dims
    emb = W.embeddings(dims, wl.layouts)
    _say("stack b1")
    got = _gpu_encode(torch, full_enc, dims, emb, wl.layouts)
    keep = (0, 13, 27)
    ref = oracle_encode(dims, emb, wl.layouts, keep=keep)
    kept = dict(O.encode.kept)
    err = rel_err(got, ref)
    _say("  err 28 layers", err)
    assert err <= TOL_STACK
    from paper_2606_05981_amd.encoder import build_positions
    pos_g = build_positions(layout_tuples(wl.layouts))
    pos = O.positions(wl.layouts)
    for l in keep:
        x = kept[l].astype(np.float32)
        h = full_enc.encode_layers(torch.from_numpy(x).cuda(), pos_g, W.seq_lens(wl.layouts), l, l + 1)
        torch.cuda.synchronize()
        r = O.layer_forward(x, pos, W.seq_lens(wl.layouts), layer_w(dims, l), dims)
        e = rel_err(h.cpu().numpy(), r)
        _say(f"  err layer {l}", e)
        assert e <= TOL_LAYER


def _oracle_batch_with_layer_inputs(dims, emb, layouts, keep):
    ref = oracle_encode(dims, emb, layouts, keep=keep)
    return ref, dict(O.encode.kept)


def _per_layer(torch, enc, dims, layouts, kept, layers, tag):
    """Each layer l of `layers` run alone on the GPU from the oracle's exact input of that
    layer (the whole packed batch), against the oracle's output of the same layer."""
    from paper_2606_05981_amd.encoder import build_positions
    lens = W.seq_lens(layouts)
    pos_g = build_positions(layout_tuples(layouts))
    pos = O.positions(layouts)
    for l in layers:
        x = kept[l].astype(np.float32)
        h = enc.encode_layers(torch.from_numpy(x).cuda(), pos_g, lens, l, l + 1)
        torch.cuda.synchronize()
        r = O.layer_forward(x, pos, lens, layer_w(dims, l), dims)
        e = rel_err(h.cpu().numpy(), r)
        _say(f"  {tag}: layer {l} (T={sum(lens)}) err {e:.3e}")
        assert e <= TOL_LAYER, (tag, l, e)


@pytest.mark.parametrize("name", ["stack_b16", "stack_b8"])
def test_stack_batched_every_frame_and_per_layer(torch, full_enc, name):
    """The benchmark's batched configurations, checked in full: every frame of the packed
    batch against the oracle run on the same packed batch (stack bar), and layers 0, 13 and
    27 each run alone from the oracle's exact input at the batch's token count (per-layer
    bar), so the tile plans and K splits used at that row count meet both bars."""
    wl = W.workload(name)
    dims = wl.dims
    emb = W.embeddings(dims, wl.layouts)
    _say(name, "T =", wl.tokens)
    got = _gpu_encode(torch, full_enc, dims, emb, wl.layouts)
    keep = (0, 13, 27)
    ref, kept = _oracle_batch_with_layer_inputs(dims, emb, wl.layouts, keep)
    worst = 0.0
    for i, sl in enumerate(seq_slices(wl.layouts)):
        e = rel_err(got[sl], ref[sl])
        worst = max(worst, e)
        assert e <= TOL_STACK, (i, e)
    _say(f"  every frame <= {worst:.3e}; whole batch {rel_err(got, ref):.3e}")
    assert rel_err(got, ref) <= TOL_STACK
    _per_layer(torch, full_enc, dims, wl.layouts, kept, keep, name)


@pytest.mark.parametrize("name", ["stack_b32_l320", "stack_mixed32"])
def test_layer0_per_layer_at_large_token_counts(torch, full_enc, name):
    """Layer 0 from the embeddings at 10240 (32 x 320) and 6759 (32 mixed lengths) rows:
    the large-M tile plans meet the per-layer bar on the whole packed batch."""
    wl = W.workload(name)
    emb = W.embeddings(wl.dims, wl.layouts)
    _per_layer(torch, full_enc, wl.dims, wl.layouts, {0: emb}, (0,), name)


@pytest.mark.parametrize("name,sample", [
    ("stack_mixed32", "minmax"),
    ("stack_b32_l320", (0, 15, 31)),
])
def test_stack_batched_sampled_sequences(torch, full_enc, name, sample):
    """The whole batch runs on the GPU; sampled sequences are re-run alone in the oracle
    (sequences are independent: the oracle pins packed == alone). The 28-layer oracle of all
    6759 or 10240 tokens would take minutes; layer 0 of the whole batch is checked above."""
    wl = W.workload(name)
    dims = wl.dims
    emb = W.embeddings(dims, wl.layouts)
    _say(name, "T =", wl.tokens)
    got = _gpu_encode(torch, full_enc, dims, emb, wl.layouts)
    lens = W.seq_lens(wl.layouts)
    if sample == "minmax":
        sample = (0, int(np.argmin(lens)), int(np.argmax(lens)), len(lens) - 1)
    sl = seq_slices(wl.layouts)
    for i in sample:
        ref = oracle_encode(dims, emb[sl[i]], [wl.layouts[i]])
        e = rel_err(got[sl[i]], ref)
        _say(f"  seq {i} (L={lens[i]}) err", e)
        assert e <= TOL_STACK


# Ragged lengths through the measured bf16 path (fp16 operands, K-split small-M tiles,
# fp16 attention operands): 1, 2, the 32-row tile edges, 64/65 and 129. Packed, the
# 129-token sequence's later query chunks see more than four key tiles, so the staged
# attention takes two LDS rounds there; one at a time, every length but 129 fits one.
RAGGED = (W.SeqLayout(1, 0, 0, 0, 0), W.SeqLayout(0, 1, 1, 1, 1), W.SeqLayout(0, 1, 4, 4, 15),
          W.SeqLayout(0, 1, 4, 4, 16), W.SeqLayout(0, 1, 4, 4, 17), W.SeqLayout(0, 1, 6, 5, 34),
          W.SeqLayout(0, 1, 8, 8, 1), W.SeqLayout(0, 1, 8, 8, 65), W.SeqLayout(5, 1, 8, 8, 27))
DIMS_2L = W.DIMS_FULL.with_(n_layers=2)


@pytest.fixture(scope="module")
def enc_2l(torch):
    enc = make_encoder(DIMS_2L, max_tokens=4096, max_batch=512, max_seq=4096)
    yield enc
    enc.close()


def test_bf16_ragged_edges_packed(torch, enc_2l):
    """One packed batch of lengths 1, 2, 31, 32, 33, 64, 65, 129 and 96 at full width:
    both layers from the oracle's inputs (per-layer bar) and the two-layer output of every
    sequence (stack bar)."""
    dims, layouts = DIMS_2L, RAGGED
    lens = W.seq_lens(layouts)
    assert lens == [1, 2, 31, 32, 33, 64, 65, 129, 96]
    emb = W.embeddings(dims, layouts)
    got = _gpu_encode(torch, enc_2l, dims, emb, layouts)
    ref, kept = _oracle_batch_with_layer_inputs(dims, emb, layouts, (0, 1))
    for i, sl in enumerate(seq_slices(layouts)):
        e = rel_err(got[sl], ref[sl])
        _say(f"  L={lens[i]}: {e:.3e}")
        assert e <= TOL_STACK, (lens[i], e)
    _per_layer(torch, enc_2l, dims, layouts, kept, (0, 1), "ragged")


@pytest.mark.parametrize("idx", [0, 1, 4, 6, 7, 8])
def test_bf16_single_sequence_lengths(torch, enc_2l, idx):
    """One sequence per call at lengths 1, 2, 33, 65, 129 and 96: the batch-of-one row
    counts, whose plans take the 4- and 8-way K splits, at both bars."""
    dims, layouts = DIMS_2L, (RAGGED[idx],)
    emb = W.embeddings(dims, layouts)
    got = _gpu_encode(torch, enc_2l, dims, emb, layouts)
    ref, kept = _oracle_batch_with_layer_inputs(dims, emb, layouts, (0, 1))
    e = rel_err(got, ref)
    _say(f"  alone L={W.seq_lens(layouts)[0]}: {e:.3e}")
    assert e <= TOL_STACK
    _per_layer(torch, enc_2l, dims, layouts, kept, (0, 1), f"alone L={W.seq_lens(layouts)[0]}")


def test_bf16_many_short_sequences(torch, enc_2l):
    """300 sequences of 1..8 tokens at full width: past the 256-sequence attention launch
    chunk and the 128-sequence position chunk; every sequence against the oracle."""
    dims = DIMS_2L
    layouts = tuple(W.SeqLayout(1 + i % 3, 1 if i % 4 else 0, 1 if i % 4 else 0, 1 + i % 2 if i % 4 else 0,
                                i % 4) for i in range(300))
    lens = W.seq_lens(layouts)
    assert len(lens) > 256
    emb = W.embeddings(dims, layouts)
    got = _gpu_encode(torch, enc_2l, dims, emb, layouts)
    ref, kept = _oracle_batch_with_layer_inputs(dims, emb, layouts, (0,))
    sl = seq_slices(layouts)
    worst = max(rel_err(got[s], ref[s]) for s in sl)
    _say(f"  300 short sequences, worst {worst:.3e}")
    assert worst <= TOL_STACK
    _per_layer(torch, enc_2l, dims, layouts, kept, (0,), "300 short")


def test_no_leak_between_sequences_bit_exact(torch, enc_2l):
    """Replacing one sequence's embeddings by other values of the same length leaves every
    other sequence's output bit-identical: the launch plan depends on the token count only,
    and no step mixes rows of different sequences."""
    dims = DIMS_2L
    layouts = (W.FRAME_96, W.SeqLayout(0, 1, 10, 9, 41), W.SeqLayout(0, 1, 8, 8, 1), W.FRAME_96)
    emb = W.embeddings(dims, layouts)
    base = _gpu_encode(torch, enc_2l, dims, emb, layouts)
    sl = seq_slices(layouts)
    for i in range(len(layouts)):
        alt = emb.copy()
        alt[sl[i]] = W.round_to_bf16(np.random.default_rng(90 + i).standard_normal(
            alt[sl[i]].shape).astype(np.float32) * np.float32(0.02))
        out = _gpu_encode(torch, enc_2l, dims, alt, layouts)
        assert not np.array_equal(out[sl[i]], base[sl[i]])
        for j in range(len(layouts)):
            if j != i:
                np.testing.assert_array_equal(out[sl[j]], base[sl[j]], err_msg=f"{i} -> {j}")


# Ragged lengths that all stay within four 32-token key tiles at their packed offsets
# (0, 96, 129, 194, 284, 285, 381): every key range is one LDS round of the staged attention,
# with sequences starting inside a tile (the packed-edge batch above needs two rounds).
RAGGED_STAGED = (W.FRAME_96, W.SeqLayout(0, 1, 4, 4, 17), W.SeqLayout(0, 1, 8, 8, 1),
                 W.SeqLayout(2, 1, 8, 8, 24), W.SeqLayout(1, 0, 0, 0, 0), W.FRAME_96,
                 W.SeqLayout(0, 1, 4, 4, 15))


def test_bf16_ragged_staged_attention(torch, enc_2l):
    """Packed lengths 96, 33, 65, 90, 1, 96, 31: every sequence against the oracle at both bars,
    and replacing a sequence that starts inside a key tile leaves every other one
    bit-identical."""
    dims, layouts = DIMS_2L, RAGGED_STAGED
    lens = W.seq_lens(layouts)
    assert lens == [96, 33, 65, 90, 1, 96, 31]
    starts = np.cumsum([0] + lens[:-1])
    assert all(((s0 + L - 1) >> 5) - (s0 >> 5) + 1 <= 4 for s0, L in zip(starts, lens))
    emb = W.embeddings(dims, layouts)
    got = _gpu_encode(torch, enc_2l, dims, emb, layouts)
    ref, kept = _oracle_batch_with_layer_inputs(dims, emb, layouts, (0, 1))
    sl = seq_slices(layouts)
    for i in range(len(layouts)):
        e = rel_err(got[sl[i]], ref[sl[i]])
        _say(f"  L={lens[i]} at {starts[i]}: {e:.3e}")
        assert e <= TOL_STACK, (lens[i], e)
    _per_layer(torch, enc_2l, dims, layouts, kept, (0, 1), "ragged staged")
    for i in (2, 3):
        alt = emb.copy()
        alt[sl[i]] = W.round_to_bf16(np.random.default_rng(70 + i).standard_normal(
            alt[sl[i]].shape).astype(np.float32) * np.float32(0.02))
        out = _gpu_encode(torch, enc_2l, dims, alt, layouts)
        assert not np.array_equal(out[sl[i]], got[sl[i]])
        for j in range(len(layouts)):
            if j != i:
                np.testing.assert_array_equal(out[sl[j]], got[sl[j]], err_msg=f"{i} -> {j}")


def test_stack_wide_range_inputs(torch, full_enc):
    """Embeddings with std 37 and +-1160 outliers (the trained encoder's activation range)."""
    wl = W.workload("stack_b1")
    dims = wl.dims
    emb = W.embeddings(dims, wl.layouts, std=37.0, outliers=6)
    got = _gpu_encode(torch, full_enc, dims, emb, wl.layouts)
    assert np.isfinite(got).all()
    err = rel_err(got, oracle_encode(dims, emb, wl.layouts))
    _say("wide range err", err)
    assert err <= TOL_STACK


# ------------------------------------------------- GPU-side invariants
def test_packed_equals_alone_and_permutation(torch):
    """No sequence sees another, and a sequence's result does not depend on where it sits in
    the packed batch beyond rounding order. Attention walks keys in the batch's 32-token
    tiles, so permuting sequences whose lengths are multiples of 32 keeps every sequence's
    offset modulo 32, the launch plan (it depends on the token count only) and every row's
    arithmetic: the permuted result is bit-identical. Ragged lengths shift those offsets,
    which only reorders the attention's sums (the bit-exact leak test above rules out any
    mixing of rows across sequences): such a permutation, and each sequence run alone
    (another token count: possibly other tiles and K splits), agree within the per-layer
    tolerance."""
    dims = W.DIMS_FULL.with_(n_layers=2)
    enc = make_encoder(dims)
    aligned = (W.FRAME_96, W.SeqLayout(0, 1, 8, 4, 32), W.SeqLayout(0, 1, 8, 12, 32))   # 96, 64, 128 tokens
    ragged = (W.FRAME_96, W.SeqLayout(0, 1, 10, 9, 41), W.SeqLayout(0, 1, 8, 8, 1))     # 96, 131, 65 tokens
    for layouts, exact in ((aligned, True), (ragged, False)):
        emb = W.embeddings(dims, layouts)
        full = _gpu_encode(torch, enc, dims, emb, layouts)
        sl = seq_slices(layouts)
        if not exact:
            for i, s in enumerate(layouts):
                alone = _gpu_encode(torch, enc, dims, np.ascontiguousarray(emb[sl[i]]), [s])
                e = rel_err(alone, full[sl[i]])
                _say(f"  alone vs packed, seq {i}: {e:.3e}")
                assert e <= TOL_LAYER
        for perm in ([2, 0, 1], [1, 2, 0]):
            idx = np.concatenate([np.arange(sl[i].start, sl[i].stop) for i in perm])
            out = _gpu_encode(torch, enc, dims, np.ascontiguousarray(emb[idx]), [layouts[i] for i in perm])
            if exact:
                np.testing.assert_array_equal(out, full[idx])
            else:
                e = rel_err(out, full[idx])
                _say(f"  permuted {perm} vs packed: {e:.3e}")
                assert e <= TOL_LAYER
    enc.close()


def test_graph_capture_replays_match_eager(torch):
    """mte_encode performs no host sync or allocation: it captures into a graph."""
    from paper_2606_05981_amd.encoder import build_positions
    dims = W.DIMS_FULL.with_(n_layers=2)
    layouts = (W.FRAME_96,) * 3
    emb = W.embeddings(dims, layouts)
    enc = make_encoder(dims)
    x = torch.from_numpy(emb).to("cuda", torch.bfloat16)
    pos = build_positions(layout_tuples(layouts))
    lens = W.seq_lens(layouts)
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
        assert bool(torch.isfinite(out).all()), r
        assert torch.equal(out, eager), r
        enc.encode(x, pos, lens)   # eager work between replays
        torch.cuda.synchronize()
    enc.close()

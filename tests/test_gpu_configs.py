"""Parity of supported model shapes beyond the default Qwen3-VL-2B layer, in bf16 storage
(fp16 matrix-core operands): head_dim 64, plain multi-head attention (one query head per kv
head), wider query groups (4, 8 and 16 query heads per kv head; 16 is beyond the LDS-staged
attention's 4- or 8-wave workgroups and takes the register-streaming kernel, with its key
split at this small batch), and the interleaved M-RoPE layout with QK-norm off at full width. Each runs one layer from the oracle's input (per-layer
bar) and a two-layer stack (stack bar) over a ragged packed batch."""
import sys

import numpy as np
import pytest

from oracle import te_oracle as O
from synth import workloads as W
from tests.gpu_common import layout_tuples, make_encoder, oracle_encode, rel_err

pytestmark = pytest.mark.gpu

TOL_LAYER = 1e-2
TOL_STACK = 3e-2

CASES = {
    "hd64": W.Dims(n_layers=2, hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=64, ffn=2816,
                   mrope_section=(12, 10, 10)),
    "mha": W.Dims(n_layers=2, hidden=1024, n_q_heads=8, n_kv_heads=8, head_dim=128, ffn=2048),
    "gqa4": W.Dims(n_layers=2, hidden=2048, n_q_heads=16, n_kv_heads=4, head_dim=128, ffn=4096),
    "gqa8": W.Dims(n_layers=2, hidden=2048, n_q_heads=16, n_kv_heads=2, head_dim=128, ffn=4096),
    "gqa16": W.Dims(n_layers=2, hidden=2048, n_q_heads=16, n_kv_heads=1, head_dim=128, ffn=4096),
    "interleaved_noqknorm": W.DIMS_FULL.with_(n_layers=2, mrope_layout=1, qk_norm=0),
}
LAYOUTS = (W.FRAME_96, W.SeqLayout(0, 1, 6, 5, 21), W.SeqLayout(3, 1, 9, 8, 40))


@pytest.mark.parametrize("case", sorted(CASES))
def test_shape_variants(case):
    import torch
    from paper_2606_05981_amd.encoder import build_positions
    assert torch.cuda.is_available(), "no GPU"
    dims = CASES[case]
    emb = W.embeddings(dims, LAYOUTS)
    lens = W.seq_lens(LAYOUTS)
    pos = O.positions(LAYOUTS)
    print(case, "T =", sum(lens), file=sys.stderr, flush=True)
    enc = make_encoder(dims, max_tokens=1024, max_batch=8, max_seq=512)
    pos_g = build_positions(layout_tuples(LAYOUTS))
    h = enc.encode_layers(torch.from_numpy(emb.astype(np.float32)).cuda(), pos_g, lens, 0, 1)
    out = enc.encode(torch.from_numpy(emb).to("cuda", torch.bfloat16), pos_g, lens)
    torch.cuda.synchronize()
    enc.close()
    from tests.gpu_common import layer_w
    e1 = rel_err(h.cpu().numpy(), O.layer_forward(emb, pos, lens, layer_w(dims, 0), dims))
    e2 = rel_err(out.float().cpu().numpy(), oracle_encode(dims, emb, LAYOUTS))
    print(f"  {case}: one layer {e1:.3e}, two layers {e2:.3e}", file=sys.stderr, flush=True)
    assert e1 <= TOL_LAYER
    assert e2 <= TOL_STACK


def test_long_sequences_one_layer():
    """Long sequences at full width, one layer from the oracle's input: a 2048-token sequence
    (a 32x32 image grid and 1024 text tokens; 64 causal query tiles, keys staged in LDS in 16
    rounds of four tiles) packed with a 1003-token one whose last key tile is partial."""
    import torch
    from paper_2606_05981_amd.encoder import build_positions
    assert torch.cuda.is_available(), "no GPU"
    dims = W.DIMS_FULL.with_(n_layers=1)
    layouts = (W.SeqLayout(0, 1, 32, 32, 1024), W.SeqLayout(11, 1, 28, 30, 152))
    emb = W.embeddings(dims, layouts)
    lens = W.seq_lens(layouts)
    print("long sequences", lens, file=sys.stderr, flush=True)
    enc = make_encoder(dims, max_tokens=sum(lens), max_batch=2, max_seq=max(lens))
    h_in = torch.from_numpy(emb.astype(np.float32)).cuda()
    h = enc.encode_layers(h_in, build_positions(layout_tuples(layouts)), lens, 0, 1)
    torch.cuda.synchronize()
    enc.close()
    ref = O.layer_forward(emb, O.positions(layouts), lens, W.layer_weights(dims, 0), dims)
    got = h.cpu().numpy()
    err = rel_err(got, ref)
    print("  err", err, file=sys.stderr, flush=True)
    assert err <= TOL_LAYER
    s = lens[0]
    assert rel_err(got[:s], ref[:s]) <= TOL_LAYER and rel_err(got[s:], ref[s:]) <= TOL_LAYER

"""Shared-prefix encode (mte_encode_prefixed) against the oracle on the full sequences.

Every frame's sequence starts with the same text prefix (the paper's system prompt and
chat template, Sec. V). The prefix is encoded once and its per-layer keys / values are
cached; each frame's own tokens attend to them and to themselves. The result must equal
the encoder run on the full sequences [prefix ++ frame tokens]: prefix rows and frame rows
are compared with the fp64 oracle of the full sequences.
"""
import sys

import numpy as np
import pytest

from oracle import te_oracle as O
from synth import workloads as W
from tests.gpu_common import make_encoder, oracle_encode, rel_err

pytestmark = pytest.mark.gpu

TOL_STACK = 3e-2


# Staged attention: an 80-token prefix (3 prefix tiles + 3 own) takes two LDS rounds, the
# first all prefix; a 16-token prefix (1 + 3 tiles) and (24, 4, 4) (20 own tokens after 24
# prefix keys: one prefix tile and one own tile) one round holding both key sources.
@pytest.mark.parametrize("prefix,hw,after,frames,n_layers",
                         [(80, 8, 32, 3, 4), (16, 8, 32, 2, 4), (80, 8, 32, 1, 28), (24, 4, 4, 2, 2)])
def test_prefixed_equals_full_sequences(prefix, hw, after, frames, n_layers):
    import torch
    assert torch.cuda.is_available(), "no GPU"
    dims = W.DIMS_FULL.with_(n_layers=n_layers)
    full = tuple(W.SeqLayout(prefix, 1, hw, hw, after) for _ in range(frames))
    L = full[0].length
    emb = W.embeddings(dims, full)            # text rows come first and are shared by all frames
    pos = O.positions(full)
    for f in range(1, frames):
        assert np.array_equal(emb[f * L:f * L + prefix], emb[:prefix])
    own = np.concatenate([np.arange(f * L + prefix, (f + 1) * L) for f in range(frames)])
    print("prefix", prefix, "frames", frames, "layers", n_layers, file=sys.stderr, flush=True)
    enc = make_encoder(dims, max_tokens=1024, max_batch=8, max_seq=512)
    enc.reserve_prefix(128)
    dt = torch.bfloat16
    out_p, out = enc.encode_prefixed(
        torch.from_numpy(np.ascontiguousarray(emb[:prefix])).to("cuda", dt),
        torch.from_numpy(np.ascontiguousarray(pos[:, :prefix])).to("cuda", torch.int32),
        torch.from_numpy(np.ascontiguousarray(emb[own])).to("cuda", dt),
        torch.from_numpy(np.ascontiguousarray(pos[:, own])).to("cuda", torch.int32),
        [L - prefix] * frames)
    torch.cuda.synchronize()
    enc.close()
    ref = oracle_encode(dims, emb, full)
    e_own = rel_err(out.float().cpu().numpy(), ref[own])
    e_pre = rel_err(out_p.float().cpu().numpy(), ref[:prefix])
    print(f"  own rows err {e_own:.3e}, prefix rows err {e_pre:.3e}", file=sys.stderr, flush=True)
    assert e_own <= TOL_STACK and e_pre <= TOL_STACK


def test_prefixed_rejects_missing_reservation_and_capacity():
    """Host-side checks of mte_encode_prefixed: no reservation, a prefix longer than the
    reservation, and prefix + sequence beyond max_seq are refused before any launch."""
    import torch
    from paper_2606_05981_amd import binding as B
    dims = W.DIMS_FULL.with_(n_layers=1)
    enc = make_encoder(dims, max_tokens=256, max_batch=4, max_seq=150)
    x = torch.zeros((96, dims.hidden), dtype=torch.bfloat16, device="cuda")
    xp = torch.zeros((80, dims.hidden), dtype=torch.bfloat16, device="cuda")
    p = torch.zeros((3, 96), dtype=torch.int32, device="cuda")
    pp = torch.zeros((3, 80), dtype=torch.int32, device="cuda")
    with pytest.raises(B.MteError) as ei:
        enc.encode_prefixed(xp, pp, x, p, [96])          # no reservation yet
    assert ei.value.status == -1
    enc.reserve_prefix(64)
    with pytest.raises(B.MteError) as ei:
        enc.encode_prefixed(xp, pp, x, p, [96])          # prefix longer than the reservation
    assert ei.value.status == -2
    enc.reserve_prefix(128)
    with pytest.raises(B.MteError) as ei:
        enc.encode_prefixed(xp, pp, x, p, [96])          # 80 + 96 tokens > max_seq 150
    assert ei.value.status == -2
    enc.close()

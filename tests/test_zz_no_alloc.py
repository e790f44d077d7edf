"""mte_encode_static: the encoder forward with its activations in the library's static
device array (no allocation in the call), against mte_encode through the C ABI -- two calls
in a row on one encoder, the second with a smaller batch -- and against the fp64 oracle;
oversized batches are rejected on the host."""
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests.gpu_common import layout_tuples, make_encoder, oracle_encode, rel_err, seq_slices

pytestmark = pytest.mark.gpu

TOL_STACK = 3e-2


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def test_static_scratch_matches_encode_twice():
    import torch
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import build_positions
    assert torch.cuda.is_available(), "no GPU"
    dims = W.DIMS_FULL.with_(n_layers=2)
    enc = make_encoder(dims, max_tokens=2048, max_batch=64, max_seq=1024)
    st = torch.cuda.current_stream().cuda_stream
    calls = [(W.FRAME_96, W.SeqLayout(0, 1, 8, 8, 33), W.SeqLayout(2, 1, 4, 4, 5)),   # 96 + 97 + 23 tokens
             (W.SeqLayout(0, 1, 4, 4, 17),)]                                          # then 33 tokens
    for n, layouts in enumerate(calls):
        lens = W.seq_lens(layouts)
        T = sum(lens)
        _say(f"call {n}: lens {lens}")
        emb = W.embeddings(dims, layouts)
        x = torch.from_numpy(emb).to("cuda", torch.bfloat16)
        pos = build_positions(layout_tuples(layouts))
        ref_gpu = torch.empty((T, dims.hidden), dtype=torch.float32, device="cuda")
        got = torch.full((T, dims.hidden), float("nan"), dtype=torch.float32, device="cuda")
        B.mte_encode(enc.handle, x.data_ptr(), pos.data_ptr(), lens, len(lens), ref_gpu.data_ptr(), st)
        B.mte_encode_static(enc.handle, x.data_ptr(), pos.data_ptr(), lens, len(lens), got.data_ptr(), st)
        torch.cuda.synchronize()
        g = got.cpu().numpy()
        assert np.isfinite(g).all()
        # same kernels and the same launch plan: identical to mte_encode bit for bit
        np.testing.assert_array_equal(g, ref_gpu.cpu().numpy())
        ref = oracle_encode(dims, emb, layouts)
        for i, sl in enumerate(seq_slices(layouts)):
            e = rel_err(g[sl], ref[sl])
            _say(f"  seq {i} (L={lens[i]}): {e:.3e}")
            assert e <= TOL_STACK
    # beyond the static array: rejected before any HIP call, nothing written
    big = [96] * 8                                                  # 768 tokens > ~736
    x = torch.zeros((sum(big), dims.hidden), dtype=torch.bfloat16, device="cuda")
    pos = torch.zeros((3, sum(big)), dtype=torch.int32, device="cuda")
    out = torch.zeros((sum(big), dims.hidden), dtype=torch.float32, device="cuda")
    with pytest.raises(B.MteError) as ei:
        B.mte_encode_static(enc.handle, x.data_ptr(), pos.data_ptr(), big, len(big), out.data_ptr(), st)
    assert ei.value.status == -2
    torch.cuda.synchronize()
    assert not bool(out.any())
    enc.close()

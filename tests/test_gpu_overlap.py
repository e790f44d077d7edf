"""The encoder on a side stream beside other GPU work (the paper's pipelining: the text
encoder runs on a side stream while the main stream denoises, Alg. 1). A captured encode
graph replays on a side stream while the main stream runs a GEMM load; its output must match
the fp64 oracle (stack bar) and be bit-identical to a solo run (the kernels' arithmetic does
not depend on what else runs)."""
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests.gpu_common import layout_tuples, make_encoder, oracle_encode, rel_err, seq_slices

pytestmark = pytest.mark.gpu


def test_side_stream_graph_concurrent_with_main_stream_load():
    import torch
    from paper_2606_05981_amd.encoder import build_positions
    assert torch.cuda.is_available(), "no GPU"
    dims = W.DIMS_FULL.with_(n_layers=2)
    layouts = (W.FRAME_96,) * 4
    emb = W.embeddings(dims, layouts)
    enc = make_encoder(dims)
    x = torch.from_numpy(emb).to("cuda", torch.bfloat16)
    pos = build_positions(layout_tuples(layouts))
    lens = W.seq_lens(layouts)
    solo = enc.encode(x, pos, lens).clone()
    torch.cuda.synchronize()
    ref = oracle_encode(dims, emb, layouts)
    out = torch.empty_like(solo)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(main)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            enc.encode(x, pos, lens, out=out, stream=side)
    main.wait_stream(side)
    a = torch.randn(2048, 2048, device="cuda", dtype=torch.float16)
    c = torch.empty_like(a)
    for r in range(3):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        side.wait_stream(main)
        with torch.cuda.stream(side):
            g.replay()
        for _ in range(8):
            torch.mm(a, a, out=c)                 # main-stream load meanwhile
        main.wait_stream(side)
        torch.cuda.synchronize()
        print("replay", r, file=sys.stderr, flush=True)
        got = out.cpu().numpy()
        for i, sl in enumerate(seq_slices(layouts)):
            e = rel_err(got[sl], ref[sl])
            assert e <= 3e-2, (r, i, e)
        assert torch.equal(out, solo), r
    enc.close()

"""Parity of the vision tower (mte_vision_*, through the C ABI) with the fp64
oracle (oracle/vit_oracle.py). Error = max|gpu - oracle| / rms(oracle) over
all image tokens. fp32 configuration <= 1e-4; bf16 weights with fp16
matrix-core operands and fp32 accumulation <= 1e-2 for two blocks and the
merger, <= 3e-2 for the 24-block tower (the decoder's bars)."""
import functools
import sys

import numpy as np
import pytest

from oracle import vit_oracle as V
from synth import vision as SV
from tests.gpu_common import rel_err

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_SHORT = 1e-2
TOL_DEEP = 3e-2


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "no GPU"
    return t


@functools.lru_cache(maxsize=None)
def _bw(v, l):
    return SV.block_weights(v, l)


@functools.lru_cache(maxsize=None)
def _ow(v):
    return SV.outer_weights(v)


def _encoder(v, max_images=4, max_side=256, out_dtype=None):
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import VisionEncoder
    dt = B.MTE_BF16 if v.dtype == "bf16" else B.MTE_F32
    cfg = B.make_vision_config(v.depth, v.hidden, v.n_heads, v.head_dim, v.ffn, patch=v.patch, merge=v.merge,
                               in_channels=v.in_channels, out_hidden=v.out_hidden, ln_eps=v.ln_eps,
                               rope_theta=v.rope_theta, dtype=dt, out_dtype=B.MTE_F32 if out_dtype is None else out_dtype,
                               max_images=max_images, max_side=max_side)
    return VisionEncoder.from_host(cfg, _ow(v), [_bw(v, l) for l in range(v.depth)])


def _run(torch, enc, v, img, raw=False):
    dt = torch.bfloat16 if v.dtype == "bf16" else torch.float32
    out = enc.encode(torch.from_numpy(img).to("cuda", dt))
    torch.cuda.synchronize()
    return out.cpu() if raw else out.float().cpu().numpy()


def _oracle(v, img):
    return V.encode(img, v, lambda l: _bw(v, l), _ow(v))


@pytest.mark.parametrize("n,h,w", [(2, 64, 96), (1, 64, 64), (3, 32, 32)])
def test_vision_tiny_fp32(torch, n, h, w):
    v = SV.VDIMS_TINY
    img = SV.images(v, n, h, w)
    _say("vision tiny fp32", n, h, w)
    enc = _encoder(v, max_side=96)
    got = _run(torch, enc, v, img)
    enc.close()
    ref = _oracle(v, img)
    assert got.shape == ref.shape
    err = rel_err(got, ref)
    _say("  err", err)
    assert err <= TOL_F32


def test_vision_bf16_two_blocks(torch):
    v = SV.VDIMS_FULL.with_(depth=2)
    img = SV.images(v, 2, 256, 256)
    _say("vision bf16, 2 blocks, 2 images of 256x256")
    enc = _encoder(v)
    got = _run(torch, enc, v, img)
    ref = _oracle(v, img)
    err = rel_err(got, ref)
    _say("  err", err)
    assert err <= TOL_SHORT
    for i in range(2):
        assert rel_err(got[64 * i:64 * (i + 1)], ref[64 * i:64 * (i + 1)]) <= TOL_SHORT
    # a bf16 output is the fp32 result rounded to nearest even
    from paper_2606_05981_amd import binding as B
    e16 = _encoder(v, out_dtype=B.MTE_BF16)
    y16 = _run(torch, e16, v, img, raw=True)
    y32 = _run(torch, enc, v, img, raw=True)
    enc.close(); e16.close()
    assert y16.dtype == torch.bfloat16 and torch.equal(y16, y32.to(torch.bfloat16))


def test_vision_bf16_512_source(torch):
    """A 512x512 source (1024 patches, 256 image tokens: the 16x16 grid of the long-sequence
    decoder configuration), two full-width blocks: attention over 1024 keys."""
    v = SV.VDIMS_FULL.with_(depth=2)
    img = SV.images(v, 1, 512, 512)
    _say("vision bf16, 2 blocks, one 512x512 image")
    enc = _encoder(v, max_images=1, max_side=512)
    got = _run(torch, enc, v, img)
    enc.close()
    ref = _oracle(v, img)
    assert got.shape == (256, v.out_hidden)
    err = rel_err(got, ref)
    _say("  err", err)
    assert err <= TOL_SHORT


def test_vision_bf16_unaligned_patch_counts(torch):
    """Images whose patch counts are not multiples of the 32-key attention tile (224x224:
    196 patches, 49 image tokens each): every image after the first starts its key range
    inside a tile and every range ends inside one, so the LDS-staged attention masks the
    first and last tiles of each range, which the aligned sizes above never need."""
    v = SV.VDIMS_FULL.with_(depth=2)
    img = SV.images(v, 3, 224, 224)
    _say("vision bf16, 2 blocks, 3 images of 224x224")
    enc = _encoder(v)
    got = _run(torch, enc, v, img)
    enc.close()
    ref = _oracle(v, img)
    assert got.shape == (3 * 49, v.out_hidden)
    for i in range(3):
        err = rel_err(got[49 * i:49 * (i + 1)], ref[49 * i:49 * (i + 1)])
        _say("  image", i, "err", err)
        assert err <= TOL_SHORT


def test_vision_bf16_full_depth(torch):
    v = SV.VDIMS_FULL
    img = SV.images(v, 1, 256, 256)
    _say("vision bf16, 24 blocks, one 256x256 image")
    enc = _encoder(v, max_images=16)
    got = _run(torch, enc, v, img)
    enc.close()
    ref = _oracle(v, img)
    err = rel_err(got, ref)
    _say("  err", err)
    assert err <= TOL_DEEP


def test_vision_strided_output_lands_in_place(torch):
    """Image tokens written at a row stride into a prefilled buffer (the layout of a packed
    text-encoder input): the token rows equal the dense output bit for bit, the rows between
    images keep their contents."""
    v = SV.VDIMS_TINY
    img = SV.images(v, 3, 64, 96)
    enc = _encoder(v, max_side=96)
    dense = enc.encode(torch.from_numpy(img).cuda())
    tpi, stride = 6, 11
    buf = torch.full(((3 - 1) * stride + tpi + 2, v.out_hidden), 7.0, device="cuda")
    enc.encode(torch.from_numpy(img).cuda(), out=buf, image_stride=stride)
    torch.cuda.synchronize()
    enc.close()
    for i in range(3):
        assert torch.equal(buf[i * stride:i * stride + tpi], dense[i * tpi:(i + 1) * tpi])
        if i < 2:
            assert bool((buf[i * stride + tpi:(i + 1) * stride] == 7.0).all())
    assert bool((buf[2 * stride + tpi:] == 7.0).all())


def test_vision_rejects_bad_shapes_and_capacity(torch):
    """Host-side checks of mte_vision_encode with a live encoder: nothing is enqueued."""
    from paper_2606_05981_amd import binding as B
    v = SV.VDIMS_TINY
    enc = _encoder(v, max_images=2, max_side=64)
    px = torch.zeros((3, 3, 64, 64), dtype=torch.float32, device="cuda")
    out = torch.empty((64, v.out_hidden), dtype=torch.float32, device="cuda")
    h, p, o = enc.handle, px.data_ptr(), out.data_ptr()
    assert B.lib.mte_vision_encode(h, p, 3, 64, 64, o, None) == -2        # more images than max_images
    assert B.lib.mte_vision_encode(h, p, 1, 96, 64, o, None) == -2        # taller than max_side
    assert B.lib.mte_vision_encode(h, p, 1, 48, 64, o, None) == -1        # not a multiple of patch * merge
    assert B.lib.mte_vision_encode(h, p, 0, 64, 64, o, None) == -1        # no images
    assert B.lib.mte_vision_encode(h, None, 1, 64, 64, o, None) == -1
    assert B.lib.mte_vision_encode_strided(h, p, 2, 64, 64, o, 3, None) == -1   # stride below 4 tokens
    # one 32x32 image: a single image token, a single merge group
    img = SV.images(v, 1, 32, 32)
    got = enc.encode(torch.from_numpy(img).cuda())
    torch.cuda.synchronize()
    enc.close()
    ref = _oracle(v, img)
    assert got.shape == (1, v.out_hidden) and rel_err(got.cpu().numpy(), ref) <= TOL_F32


def test_vision_graph_replays_match_eager(torch):
    """mte_vision_encode only enqueues work: captured once, every replay (with eager work in
    between) reproduces the eager result bit for bit, also when written strided."""
    v = SV.VDIMS_FULL.with_(depth=2)
    img = torch.from_numpy(SV.images(v, 2, 256, 256)).to("cuda", torch.bfloat16)
    enc = _encoder(v)
    eager = enc.encode(img).clone()
    out = torch.empty((2 * 96, v.out_hidden), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            enc.encode(img, out=out, image_stride=96, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    for r in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for i in range(2):
            assert torch.equal(out[96 * i:96 * i + 64], eager[64 * i:64 * (i + 1)]), (r, i)
        assert bool(torch.isnan(out[64:96]).all())          # rows between images untouched
        enc.encode(img)                                      # eager work between replays
        torch.cuda.synchronize()
    enc.close()

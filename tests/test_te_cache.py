"""TECache: the optional text-encoder caching modes (Sec. III-B) as host logic around an
encoder -- which rows are encoded, how often, and what each frame receives. Runs on the CPU
with a stand-in encoder; the GPU test is in test_gpu_te_cache.py."""
import pytest
import torch

from paper_2606_05981_amd.encoder import TECache

D = 8


class _Enc:
    """Records every encode call and returns a value that identifies its input rows."""

    def __init__(self):
        self.calls = []

    def encode(self, embeds, pos_thw, seq_lens, stream=None):
        assert pos_thw.is_contiguous() and pos_thw.shape == (3, embeds.shape[0])
        assert sum(seq_lens) == embeds.shape[0]
        self.calls.append((embeds.clone(), pos_thw.clone(), list(seq_lens)))
        return embeds.float() * 2 + pos_thw[0].float()[:, None]


def _batch(lens, seed=0):
    g = torch.Generator().manual_seed(seed)
    T = sum(lens)
    return torch.randn(T, D, generator=g), torch.arange(3 * T, dtype=torch.int32).reshape(3, T)


def test_plain_encodes_the_whole_batch_every_call():
    enc, lens = _Enc(), [4, 4, 4]
    c = TECache(enc)
    for i in range(3):
        e, p = _batch(lens, i)
        out = c(e, p, lens)
        assert torch.equal(out, e * 2 + p[0].float()[:, None])
    assert len(enc.calls) == 3 and c.encodes == 3


def test_batch_one_encodes_the_first_frame_and_broadcasts_it():
    enc, lens = _Enc(), [5, 5, 5, 5]
    e, p = _batch(lens)
    out = TECache(enc, batch_one=True)(e, p, lens)
    (ce, cp, cl), = enc.calls
    assert cl == [5] and torch.equal(ce, e[:5]) and torch.equal(cp, p[:, :5])
    assert out.shape == (4, 5, D)
    one = e[:5] * 2 + p[0, :5].float()[:, None]
    for f in range(4):
        assert torch.equal(out[f], one)
    assert out.stride(0) == 0                   # a view of the one encoded frame, not copies


def test_refresh_every_reuses_the_result_between_refreshes():
    enc, lens = _Enc(), [3, 3]
    c = TECache(enc, batch_one=True, refresh_every=3)
    outs = []
    for i in range(7):
        e, p = _batch(lens, i)
        outs.append(c(e, p, lens))
    assert c.encodes == 3 and len(enc.calls) == 3        # calls 0, 3 and 6
    assert outs[1] is outs[0] and outs[2] is outs[0]
    assert outs[4] is outs[3] and outs[5] is outs[3]
    assert outs[3] is not outs[0] and outs[6] is not outs[3]
    e3, p3 = _batch(lens, 3)
    assert torch.equal(enc.calls[1][0], e3[:3])


def test_bad_arguments():
    with pytest.raises(ValueError):
        TECache(_Enc(), refresh_every=0)
    e, p = _batch([2])
    with pytest.raises(ValueError):
        TECache(_Enc())(e, p, [0, 2])

"""The torch wrapper rejects tensors the kernels cannot take -- on the host, on another
device, of the wrong dtype or shape, or not contiguous -- with ValueError before any call
into the library (runs without a GPU: the checks never reach the C ABI)."""
import pytest
import torch

from paper_2606_05981_amd import binding as B
from paper_2606_05981_amd.encoder import TextEncoder

D = 256


class _Lib:
    """Stands in for the C ABI: any call into it fails the test."""

    def __getattr__(self, name):
        raise AssertionError(f"{name} reached the library")


@pytest.fixture
def enc(monkeypatch):
    import paper_2606_05981_amd.encoder as E
    monkeypatch.setattr(E, "B", _Lib())
    e = object.__new__(TextEncoder)
    e.cfg = B.make_config(2, D, 4, 2, 64, 768, mrope_section=(12, 10, 10), dtype=B.MTE_BF16,
                          out_dtype=B.MTE_F32)
    e.dtype, e.out_dtype = torch.bfloat16, torch.float32
    e.device = torch.device("cuda:0")
    e.handle = None
    return e


LENS = [5, 3]
T = sum(LENS)


def test_host_embeddings_rejected(enc):
    with pytest.raises(ValueError, match="embeds"):
        enc.encode(torch.zeros(T, D, dtype=torch.bfloat16), torch.zeros(3, T, dtype=torch.int32), LENS)


def test_host_positions_rejected_for_layers(enc):
    with pytest.raises(ValueError, match="h_in"):
        enc.encode_layers(torch.zeros(T, D), torch.zeros(3, T, dtype=torch.int32), LENS, 0, 1)


def test_bad_lengths_rejected(enc):
    for lens in ([], [3, 0], [-1]):
        with pytest.raises(ValueError, match="seq_lens"):
            enc.encode(torch.zeros(1, D, dtype=torch.bfloat16), torch.zeros(3, 1, dtype=torch.int32), lens)


def test_check_helper_rules():
    from paper_2606_05981_amd.encoder import _check
    dev = torch.device("cuda:0")
    with pytest.raises(ValueError, match="on cuda:0"):
        _check("x", torch.zeros(2, 3), torch.float32, (2, 3), dev)
    with pytest.raises(ValueError, match="torch.Tensor"):
        _check("x", [[0.0] * 3] * 2, torch.float32, (2, 3), dev)
    meta = torch.empty((2, 3), device="meta")
    with pytest.raises(ValueError, match="on cuda:0"):
        _check("x", meta, torch.float32, (2, 3), dev)


def test_prefixed_rejects_host_tensors(enc):
    with pytest.raises(ValueError, match="prefix_embeds"):
        enc.encode_prefixed(torch.zeros(4, D, dtype=torch.bfloat16), torch.zeros(3, 4, dtype=torch.int32),
                            torch.zeros(T, D, dtype=torch.bfloat16), torch.zeros(3, T, dtype=torch.int32), LENS)

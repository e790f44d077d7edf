"""Torch-facing wrapper of the C ABI: tensors in, tensors out.

PyTorch only provides device memory and streams here; every step of the
encoder runs in libmte's HIP kernels. Nothing falls back to another
implementation: a missing library raises at import, a failing call raises
MteError.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import torch

from . import binding as B

WEIGHT_KEYS = ("attn_norm", "w_q", "w_k", "w_v", "q_norm", "k_norm", "w_o", "mlp_norm",
               "w_gate", "w_up", "w_down")
TORCH_DTYPE = {B.MTE_F32: torch.float32, B.MTE_BF16: torch.bfloat16}


def _stream(stream: Optional[torch.cuda.Stream]) -> int:
    return (stream or torch.cuda.current_stream()).cuda_stream


def _check(name: str, t, dtype: torch.dtype, shape, device: torch.device) -> None:
    """Raises ValueError unless t is a contiguous tensor of `dtype` and exactly `shape` on
    `device`: the C ABI takes bare addresses, so a host tensor or a short buffer would
    otherwise reach the kernels."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor")
    if not t.is_cuda or t.device != device:
        raise ValueError(f"{name}: expected a tensor on {device}, got one on {t.device}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: expected dtype {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")


def _total(seq_lens: Sequence[int]) -> int:
    lens = [int(x) for x in seq_lens]
    if not lens or min(lens) <= 0:
        raise ValueError("seq_lens must be a non-empty list of positive lengths")
    return sum(lens)


class TextEncoder:
    """Owns one mte_encoder. Weights are copied into the library at creation."""

    def __init__(self, cfg: B.mte_config, layers: Sequence[Dict[str, torch.Tensor]],
                 final_norm: torch.Tensor, stream: Optional[torch.cuda.Stream] = None):
        self.cfg = cfg
        self.dtype = TORCH_DTYPE[cfg.dtype]
        self.out_dtype = TORCH_DTYPE[cfg.out_dtype]
        if not final_norm.is_cuda:
            raise ValueError("final_norm: expected a tensor on the GPU")
        # the encoder lives on the device its weights are on (mte_encoder_create
        # allocates on the current device, made that one here)
        self.device = final_norm.device
        for L in layers:
            for k, t in L.items():
                if t is not None and (t.dtype != self.dtype or t.device != self.device or not t.is_contiguous()):
                    raise ValueError(f"weight {k}: expected contiguous {self.dtype} on {self.device}")
        ptrs = [{k: (L[k].data_ptr() if L.get(k) is not None else None) for k in WEIGHT_KEYS}
                for L in layers]
        with torch.cuda.device(self.device):
            self.handle = B.mte_encoder_create(cfg, ptrs, final_norm.data_ptr(), _stream(stream))

    @classmethod
    def from_host(cls, cfg: B.mte_config, layer_arrays, final_norm, device="cuda",
                  stream: Optional[torch.cuda.Stream] = None) -> "TextEncoder":
        """Creates the encoder from host arrays (numpy or CPU tensors), one layer at a time
        on the device, so peak device memory is one layer beyond the library's copy."""
        dt = TORCH_DTYPE[cfg.dtype]
        layers: List[Dict[str, torch.Tensor]] = []
        for arrs in layer_arrays:
            layers.append({k: torch.as_tensor(arrs[k]).to(device=device, dtype=dt).contiguous()
                           for k in WEIGHT_KEYS if k in arrs})
        fn = torch.as_tensor(final_norm).to(device=device, dtype=dt).contiguous()
        enc = cls(cfg, layers, fn, stream)
        torch.cuda.synchronize()
        return enc

    def encode(self, embeds: torch.Tensor, pos_thw: torch.Tensor, seq_lens: Sequence[int],
               out: Optional[torch.Tensor] = None,
               stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        T = _total(seq_lens)
        D = self.cfg.hidden
        _check("embeds", embeds, self.dtype, (T, D), self.device)
        _check("pos_thw", pos_thw, torch.int32, (3, T), self.device)
        if out is None:
            out = torch.empty((T, D), dtype=self.out_dtype, device=self.device)
        _check("out", out, self.out_dtype, (T, D), self.device)
        B.mte_encode(self.handle, embeds.data_ptr(), pos_thw.data_ptr(), list(seq_lens),
                     len(seq_lens), out.data_ptr(), _stream(stream))
        return out

    def encode_layers(self, h_in: torch.Tensor, pos_thw: torch.Tensor, seq_lens: Sequence[int],
                      layer_begin: int, layer_end: int, h_out: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        T = _total(seq_lens)
        D = self.cfg.hidden
        _check("h_in", h_in, torch.float32, (T, D), self.device)
        _check("pos_thw", pos_thw, torch.int32, (3, T), self.device)
        if h_out is None:
            h_out = torch.empty_like(h_in)
        _check("h_out", h_out, torch.float32, (T, D), self.device)
        B.mte_encode_layers(self.handle, h_in.data_ptr(), pos_thw.data_ptr(), list(seq_lens),
                            len(seq_lens), layer_begin, layer_end, h_out.data_ptr(), _stream(stream))
        return h_out

    def reserve_prefix(self, max_prefix: int) -> None:
        B.mte_encoder_reserve_prefix(self.handle, max_prefix)

    def encode_prefixed(self, prefix_embeds: torch.Tensor, prefix_pos: torch.Tensor,
                        embeds: torch.Tensor, pos_thw: torch.Tensor, seq_lens: Sequence[int],
                        stream: Optional[torch.cuda.Stream] = None):
        """Sequences sharing a prefix -> (prefix rows [P, D], own rows [T, D])."""
        T = _total(seq_lens)
        D = self.cfg.hidden
        if not isinstance(prefix_embeds, torch.Tensor) or prefix_embeds.dim() != 2:
            raise ValueError("prefix_embeds: expected a 2-D tensor")
        P = int(prefix_embeds.shape[0])
        _check("prefix_embeds", prefix_embeds, self.dtype, (P, D), self.device)
        _check("embeds", embeds, self.dtype, (T, D), self.device)
        _check("prefix_pos", prefix_pos, torch.int32, (3, P), self.device)
        _check("pos_thw", pos_thw, torch.int32, (3, T), self.device)
        out_p = torch.empty((P, D), dtype=self.out_dtype, device=self.device)
        out = torch.empty((T, D), dtype=self.out_dtype, device=self.device)
        B.mte_encode_prefixed(self.handle, prefix_embeds.data_ptr(), prefix_pos.data_ptr(), P,
                              embeds.data_ptr(), pos_thw.data_ptr(), list(seq_lens), len(seq_lens),
                              out_p.data_ptr(), out.data_ptr(), _stream(stream))
        return out_p, out

    def close(self) -> None:
        if getattr(self, "handle", None):
            B.mte_encoder_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class TECache:
    """The optional text-encoder caching modes for streams whose instruction is fixed
    (Sec. III-B, optional TE caching modes), around a TextEncoder:

    - batch_one: encode only the batch's first frame (its rows 0 .. seq_lens[0] - 1) and
      hand every frame that frame's hidden states, as a [B, L0, D] broadcast view (no copy);
    - refresh_every = N: keep the result for N consecutive calls, encoding on the first of
      every N (counting from the first call).

    Both are approximations the caller opts into (the conditioning drifts from the frames it
    stands for); with neither, every call encodes the whole packed batch and returns [T, D].
    The cached tensor is returned as is until the next refresh."""

    def __init__(self, encoder: "TextEncoder", batch_one: bool = False, refresh_every: int = 1):
        if int(refresh_every) < 1:
            raise ValueError("refresh_every must be >= 1")
        self.encoder = encoder
        self.batch_one = bool(batch_one)
        self.refresh_every = int(refresh_every)
        self.calls = 0
        self.encodes = 0
        self._cached: Optional[torch.Tensor] = None

    def __call__(self, embeds: torch.Tensor, pos_thw: torch.Tensor, seq_lens: Sequence[int],
                 stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        lens = [int(x) for x in seq_lens]
        _total(lens)
        refresh = self._cached is None or self.calls % self.refresh_every == 0
        self.calls += 1
        if not refresh:
            return self._cached
        if self.batch_one:
            l0 = lens[0]
            one = self.encoder.encode(embeds[:l0], pos_thw[:, :l0].contiguous(), [l0], stream=stream)
            out = one.unsqueeze(0).expand(len(lens), l0, one.shape[1])
        else:
            out = self.encoder.encode(embeds, pos_thw, lens, stream=stream)
        self.encodes += 1
        self._cached = out
        return out


def build_positions(layouts: Sequence[Sequence[int]], device="cuda",
                    stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """(t, h, w) positions of packed sequences, built on the device -> int32 [3, T]."""
    T = sum(int(l[0]) + int(l[1]) * int(l[2]) * int(l[3]) + int(l[4]) for l in layouts)
    pos = torch.empty((3, T), dtype=torch.int32, device=device)
    B.mte_build_positions(layouts, pos.data_ptr(), _stream(stream))
    return pos


def quantize_e4m3_rows(w: torch.Tensor, stream: Optional[torch.cuda.Stream] = None):
    """OCP e4m3 codes and power-of-two row scales of a [rows, cols] bf16 / fp32
    device matrix (mte_quantize_e4m3_rows) -> (uint8 [rows, cols], float32 [rows])."""
    if w.dim() != 2 or not w.is_cuda or not w.is_contiguous() or w.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("w must be a contiguous 2-D bf16 or fp32 tensor on the GPU")
    rows, cols = w.shape
    codes = torch.empty((rows, cols), dtype=torch.uint8, device=w.device)
    scales = torch.empty((rows,), dtype=torch.float32, device=w.device)
    B.mte_quantize_e4m3_rows(w.data_ptr(), B.MTE_BF16 if w.dtype == torch.bfloat16 else B.MTE_F32, rows, cols,
                             codes.data_ptr(), scales.data_ptr(), _stream(stream))
    return codes, scales


class VisionEncoder:
    """Owns one mte_vision (include/mte_vision.h): images -> image-token embeddings."""

    def __init__(self, cfg: B.mte_vision_config, outer: Dict[str, torch.Tensor],
                 layers: Sequence[Dict[str, torch.Tensor]], stream: Optional[torch.cuda.Stream] = None):
        self.cfg = cfg
        self.dtype = TORCH_DTYPE[cfg.dtype]
        self.out_dtype = TORCH_DTYPE[cfg.out_dtype]
        for t in list(outer.values()) + [t for L in layers for t in L.values()]:
            if t.dtype != self.dtype or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"vision weights: expected contiguous {self.dtype} tensors on the GPU")
        self.handle = B.mte_vision_create(cfg, {k: outer[k].data_ptr() for k in B.VISION_OUTER_FIELDS},
                                          [{k: L[k].data_ptr() for k in B.VISION_LAYER_FIELDS} for L in layers],
                                          _stream(stream))
        torch.cuda.synchronize()

    @classmethod
    def from_host(cls, cfg: B.mte_vision_config, outer, layer_arrays, device="cuda"):
        dt = TORCH_DTYPE[cfg.dtype]
        put = lambda a: torch.as_tensor(a).to(device=device, dtype=dt).contiguous()
        return cls(cfg, {k: put(outer[k]) for k in B.VISION_OUTER_FIELDS},
                   [{k: put(L[k]) for k in B.VISION_LAYER_FIELDS} for L in layer_arrays])

    def encode(self, pixels: torch.Tensor, out: Optional[torch.Tensor] = None,
               stream: Optional[torch.cuda.Stream] = None, image_stride: Optional[int] = None) -> torch.Tensor:
        """pixels [n, C, H, W] of the config dtype -> [n * tokens per image, out_hidden], or with
        image_stride image i's tokens at rows i*image_stride.. of `out` (mte_vision_encode_strided)."""
        c = self.cfg
        if pixels.dim() != 4 or pixels.dtype != self.dtype or not pixels.is_contiguous() or \
                pixels.shape[1] != c.in_channels:
            raise ValueError("pixels must be a contiguous [n, C, H, W] tensor of the encoder dtype")
        n, _, h, w = pixels.shape
        s = c.patch * c.merge
        tpi = (h // s) * (w // s)
        stride = tpi if image_stride is None else int(image_stride)
        rows = (n - 1) * stride + tpi
        if out is None:
            out = torch.empty((rows, c.out_hidden), dtype=self.out_dtype, device=pixels.device)
        if out.dtype != self.out_dtype or not out.is_contiguous() or out.dim() != 2 or \
                out.shape[1] != c.out_hidden or out.shape[0] < rows:
            raise ValueError("out must be a contiguous [rows, out_hidden] tensor of the output dtype")
        B.mte_vision_encode_strided(self.handle, pixels.data_ptr(), n, h, w, out.data_ptr(), stride,
                                    _stream(stream))
        return out

    def close(self) -> None:
        if getattr(self, "handle", None):
            B.mte_vision_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

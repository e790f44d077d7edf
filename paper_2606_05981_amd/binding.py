"""ctypes binding of libmte (include/mte.h): argument marshalling only.

Every function keeps the C name and returns what the C call returns, except
that a negative status raises MteError. Device buffers are passed as integer
addresses (``tensor.data_ptr()``) and streams as ``hipStream_t`` handles
(``torch.cuda.current_stream().cuda_stream``). There is no fallback: if the
library is not built, importing this module raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmte.so")

MTE_F32, MTE_BF16 = 0, 1
MTE_MROPE_SECTIONS, MTE_MROPE_INTERLEAVED = 0, 1
MTE_WEIGHTS_DTYPE, MTE_WEIGHTS_E4M3 = 0, 1
STATUS = {0: "MTE_OK", -1: "MTE_E_INVALID", -2: "MTE_E_CAPACITY", -3: "MTE_E_HIP",
          -4: "MTE_E_OOM", -5: "MTE_E_UNSUPPORTED"}
KERNEL_CLASSES = {"qkv_gemm": 0, "attention": 1, "o_gemm": 2, "gate_up_gemm": 3, "down_gemm": 4}


class MteError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({mte_status_string(status)})")


class mte_config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("mrope_section", C.c_int32 * 3), ("mrope_layout", C.c_int32),
                ("qk_norm", C.c_int32), ("dtype", C.c_int32), ("out_dtype", C.c_int32),
                ("max_tokens", C.c_int32), ("max_batch", C.c_int32), ("max_seq", C.c_int32),
                ("weight_format", C.c_int32)]


class mte_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "w_q", "w_k", "w_v", "q_norm", "k_norm",
                                          "w_o", "mlp_norm", "w_gate", "w_up", "w_down")]


class mte_weights(C.Structure):
    _fields_ = [("layers", C.POINTER(mte_layer_weights)), ("final_norm", C.c_void_p)]


class mte_seq_layout(C.Structure):
    _fields_ = [("n_text_before", C.c_int32), ("grid_t", C.c_int32), ("grid_h", C.c_int32),
                ("grid_w", C.c_int32), ("n_text_after", C.c_int32)]


class mte_vision_config(C.Structure):
    _fields_ = [("depth", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32), ("head_dim", C.c_int32),
                ("ffn", C.c_int32), ("patch", C.c_int32), ("merge", C.c_int32), ("in_channels", C.c_int32),
                ("out_hidden", C.c_int32), ("ln_eps", C.c_float), ("rope_theta", C.c_float),
                ("dtype", C.c_int32), ("out_dtype", C.c_int32), ("max_images", C.c_int32),
                ("max_side", C.c_int32)]


VISION_LAYER_FIELDS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o", "ln2_g", "ln2_b", "w_fc1", "b_fc1",
                       "w_fc2", "b_fc2")
VISION_OUTER_FIELDS = ("patch_w", "patch_b", "merge_ln_g", "merge_ln_b", "merge_w1", "merge_b1", "merge_w2",
                       "merge_b2")


class mte_vision_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in VISION_LAYER_FIELDS]


class mte_vision_weights(C.Structure):
    _fields_ = [("patch_w", C.c_void_p), ("patch_b", C.c_void_p),
                ("layers", C.POINTER(mte_vision_layer_weights)),
                ("merge_ln_g", C.c_void_p), ("merge_ln_b", C.c_void_p), ("merge_w1", C.c_void_p),
                ("merge_b1", C.c_void_p), ("merge_w2", C.c_void_p), ("merge_b2", C.c_void_p)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_05981_amd.build`")
lib = C.CDLL(LIB_PATH)

_P = C.c_void_p
_sig = {
    "mte_config_validate": (C.c_int, [C.POINTER(mte_config)]),
    "mte_check_batch": (C.c_int, [C.POINTER(mte_config), C.POINTER(C.c_int32), C.c_int32,
                                  C.POINTER(C.c_int32)]),
    "mte_encoder_create": (C.c_int, [C.POINTER(mte_config), C.POINTER(mte_weights), _P,
                                     C.POINTER(_P)]),
    "mte_encode": (C.c_int, [_P, _P, _P, C.POINTER(C.c_int32), C.c_int32, _P, _P]),
    "mte_encode_static": (C.c_int, [_P, _P, _P, C.POINTER(C.c_int32), C.c_int32, _P, _P]),
    "mte_encode_layers": (C.c_int, [_P, _P, _P, C.POINTER(C.c_int32), C.c_int32, C.c_int32,
                                    C.c_int32, _P, _P]),
    "mte_build_positions": (C.c_int, [C.POINTER(mte_seq_layout), C.c_int32, _P, _P]),
    "mte_encoder_reserve_prefix": (C.c_int, [_P, C.c_int32]),
    "mte_encode_prefixed": (C.c_int, [_P, _P, _P, C.c_int32, _P, _P, C.POINTER(C.c_int32), C.c_int32, _P,
                                      _P, _P]),
    "mte_encoder_destroy": (None, [_P]),
    "mte_status_string": (C.c_char_p, [C.c_int]),
    "mte_timing_enable": (C.c_int, [_P, C.c_int32, C.c_int32]),
    "mte_timing_read": (C.c_int, [_P, C.POINTER(C.c_int32), C.POINTER(C.c_double)]),
    "mte_timing_disable": (C.c_int, [_P]),
    "mte_quantize_e4m3_rows": (C.c_int, [_P, C.c_int32, C.c_int32, C.c_int32, _P, _P, _P]),
    "mte_vision_config_validate": (C.c_int, [C.POINTER(mte_vision_config)]),
    "mte_vision_create": (C.c_int, [C.POINTER(mte_vision_config), C.POINTER(mte_vision_weights), _P,
                                    C.POINTER(_P)]),
    "mte_vision_encode": (C.c_int, [_P, _P, C.c_int32, C.c_int32, C.c_int32, _P, _P]),
    "mte_vision_encode_strided": (C.c_int, [_P, _P, C.c_int32, C.c_int32, C.c_int32, _P, C.c_int32, _P]),
    "mte_vision_destroy": (None, [_P]),
}
for _name, (_res, _args) in _sig.items():
    _f = getattr(lib, _name)
    _f.restype, _f.argtypes = _res, _args


def _check(st: int, where: str) -> int:
    if st < 0:
        raise MteError(st, where)
    return st


def _i32(values: Sequence[int]):
    return (C.c_int32 * len(values))(*[int(v) for v in values])


def make_config(n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, rms_eps=1e-6,
                rope_theta=5e6, mrope_section=(24, 20, 20), mrope_layout=0, qk_norm=1,
                dtype=MTE_BF16, out_dtype=None, max_tokens=4096, max_batch=64,
                max_seq=4096, weight_format=MTE_WEIGHTS_DTYPE) -> mte_config:
    c = mte_config()
    c.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads = n_layers, hidden, n_q_heads, n_kv_heads
    c.head_dim, c.ffn, c.rms_eps, c.rope_theta = head_dim, ffn, rms_eps, rope_theta
    c.mrope_section[:] = list(mrope_section)
    c.mrope_layout, c.qk_norm, c.dtype = mrope_layout, qk_norm, dtype
    c.out_dtype = dtype if out_dtype is None else out_dtype
    c.max_tokens, c.max_batch, c.max_seq = max_tokens, max_batch, max_seq
    c.weight_format = weight_format
    return c


def mte_status_string(status: int) -> str:
    return lib.mte_status_string(int(status)).decode()


def mte_config_validate(cfg: mte_config) -> int:
    return lib.mte_config_validate(C.byref(cfg))


def mte_check_batch(cfg: Optional[mte_config], seq_lens: Optional[Sequence[int]],
                    batch: Optional[int] = None):
    """Returns (status, total_tokens)."""
    tot = C.c_int32(-1)
    arr = _i32(seq_lens) if seq_lens is not None else None
    n = len(seq_lens) if batch is None else batch
    st = lib.mte_check_batch(C.byref(cfg) if cfg is not None else None, arr, n, C.byref(tot))
    return st, tot.value


def mte_encoder_create(cfg: mte_config, layers: Sequence[dict], final_norm: int, stream: int) -> int:
    """layers: per layer a dict of device addresses keyed like mte_layer_weights."""
    arr = (mte_layer_weights * max(1, len(layers)))()
    for i, L in enumerate(layers):
        for k, v in L.items():
            setattr(arr[i], k, v)
    w = mte_weights(arr if layers else None, final_norm)
    h = _P()
    _check(lib.mte_encoder_create(C.byref(cfg), C.byref(w), stream, C.byref(h)), "mte_encoder_create")
    return h.value


def mte_encode(enc: int, embeds: int, pos_thw: int, seq_lens: Sequence[int], batch: int,
               out_hidden: int, stream: int) -> int:
    return _check(lib.mte_encode(enc, embeds, pos_thw, _i32(seq_lens), batch, out_hidden, stream),
                  "mte_encode")


def mte_encode_static(enc: int, embeds: int, pos_thw: int, seq_lens: Sequence[int], batch: int,
                      out_hidden: int, stream: int) -> int:
    return _check(lib.mte_encode_static(enc, embeds, pos_thw, _i32(seq_lens), batch, out_hidden, stream),
                  "mte_encode_static")


def mte_encode_layers(enc: int, h_in: int, pos_thw: int, seq_lens: Sequence[int], batch: int,
                      layer_begin: int, layer_end: int, h_out: int, stream: int) -> int:
    return _check(lib.mte_encode_layers(enc, h_in, pos_thw, _i32(seq_lens), batch, layer_begin,
                                        layer_end, h_out, stream), "mte_encode_layers")


def mte_build_positions(layouts: Sequence[Sequence[int]], pos_thw: int, stream: int) -> int:
    arr = (mte_seq_layout * max(1, len(layouts)))()
    for i, s in enumerate(layouts):
        arr[i] = mte_seq_layout(*[int(v) for v in s])
    return _check(lib.mte_build_positions(arr, len(layouts), pos_thw, stream), "mte_build_positions")


def mte_encoder_reserve_prefix(enc: int, max_prefix: int) -> int:
    return _check(lib.mte_encoder_reserve_prefix(enc, max_prefix), "mte_encoder_reserve_prefix")


def mte_encode_prefixed(enc: int, prefix_embeds: int, prefix_pos: int, prefix_len: int, embeds: int,
                        pos_thw: int, seq_lens: Sequence[int], batch: int, out_prefix: int,
                        out_hidden: int, stream: int) -> int:
    return _check(lib.mte_encode_prefixed(enc, prefix_embeds, prefix_pos, prefix_len, embeds, pos_thw,
                                          _i32(seq_lens), batch, out_prefix, out_hidden, stream),
                  "mte_encode_prefixed")


def mte_encoder_destroy(enc: int) -> None:
    lib.mte_encoder_destroy(enc)


def mte_timing_enable(enc: int, kernel_class: int, capacity: int) -> int:
    return _check(lib.mte_timing_enable(enc, kernel_class, capacity), "mte_timing_enable")


def mte_timing_read(enc: int):
    n, ms = C.c_int32(0), C.c_double(0.0)
    _check(lib.mte_timing_read(enc, C.byref(n), C.byref(ms)), "mte_timing_read")
    return n.value, ms.value


def mte_timing_disable(enc: int) -> int:
    return _check(lib.mte_timing_disable(enc), "mte_timing_disable")


def mte_quantize_e4m3_rows(src: int, src_dtype: int, rows: int, cols: int, codes: int, scales: int,
                           stream: int) -> int:
    return _check(lib.mte_quantize_e4m3_rows(src, src_dtype, rows, cols, codes, scales, stream),
                  "mte_quantize_e4m3_rows")


def make_vision_config(depth, hidden, n_heads, head_dim, ffn, patch=16, merge=2, in_channels=3, out_hidden=2048,
                       ln_eps=1e-6, rope_theta=10000.0, dtype=MTE_BF16, out_dtype=None, max_images=16,
                       max_side=256) -> mte_vision_config:
    c = mte_vision_config()
    c.depth, c.hidden, c.n_heads, c.head_dim, c.ffn = depth, hidden, n_heads, head_dim, ffn
    c.patch, c.merge, c.in_channels, c.out_hidden = patch, merge, in_channels, out_hidden
    c.ln_eps, c.rope_theta, c.dtype = ln_eps, rope_theta, dtype
    c.out_dtype = dtype if out_dtype is None else out_dtype
    c.max_images, c.max_side = max_images, max_side
    return c


def mte_vision_config_validate(cfg: mte_vision_config) -> int:
    return lib.mte_vision_config_validate(C.byref(cfg))


def mte_vision_create(cfg: mte_vision_config, outer: dict, layers: Sequence[dict], stream: int) -> int:
    """outer: device addresses keyed like VISION_OUTER_FIELDS; layers: per block keyed like
    VISION_LAYER_FIELDS."""
    arr = (mte_vision_layer_weights * max(1, len(layers)))()
    for i, L in enumerate(layers):
        for k, v in L.items():
            setattr(arr[i], k, v)
    w = mte_vision_weights()
    for k in VISION_OUTER_FIELDS:
        setattr(w, k, outer[k])
    w.layers = arr if layers else None
    h = _P()
    _check(lib.mte_vision_create(C.byref(cfg), C.byref(w), stream, C.byref(h)), "mte_vision_create")
    return h.value


def mte_vision_encode(enc: int, pixels: int, n_images: int, height: int, width: int, out: int,
                      stream: int) -> int:
    return _check(lib.mte_vision_encode(enc, pixels, n_images, height, width, out, stream), "mte_vision_encode")


def mte_vision_destroy(enc: int) -> None:
    lib.mte_vision_destroy(enc)


def mte_vision_encode_strided(enc: int, pixels: int, n_images: int, height: int, width: int, out: int,
                              image_stride: int, stream: int) -> int:
    return _check(lib.mte_vision_encode_strided(enc, pixels, n_images, height, width, out, image_stride, stream),
                  "mte_vision_encode_strided")


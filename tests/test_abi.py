"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects bad arguments before any HIP call (runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def B():
    from paper_2606_05981_amd import binding
    return binding


def _declared_functions():
    src = "".join(open(os.path.join(ROOT, "include", f)).read() for f in ("mte.h", "mte_vision.h"))
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\**\s*(mte_[a-z0-9_]+)\s*\(", src, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for n in ("mte_encoder_create", "mte_encode", "mte_build_positions", "mte_encoder_destroy",
              "mte_status_string", "mte_config_validate", "mte_check_batch", "mte_encode_layers",
              "mte_encoder_reserve_prefix", "mte_encode_prefixed", "mte_quantize_e4m3_rows",
              "mte_vision_config_validate", "mte_vision_create", "mte_vision_encode", "mte_vision_destroy",
              "mte_vision_encode_strided"):
        assert n in names


def test_library_exports_every_declared_symbol(B):
    lib = ctypes.CDLL(B.LIB_PATH)
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def _full(B, **kw):
    args = dict(n_layers=28, hidden=2048, n_q_heads=16, n_kv_heads=8, head_dim=128, ffn=6144)
    args.update(kw)
    return B.make_config(**args)


def test_valid_configs(B):
    assert B.mte_config_validate(_full(B)) == 0
    assert B.mte_config_validate(_full(B, n_layers=0)) == 0
    tiny = B.make_config(2, 256, 4, 2, 64, 768, mrope_section=(12, 10, 10), dtype=B.MTE_F32)
    assert B.mte_config_validate(tiny) == 0
    assert B.mte_config_validate(_full(B, mrope_layout=1, qk_norm=0)) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(n_q_heads=16, n_kv_heads=5), -1),          # Hq % Hkv != 0
    (dict(mrope_section=(24, 20, 19)), -1),          # sections do not sum to d/2
    (dict(mrope_section=(-1, 45, 20)), -1),
    (dict(hidden=0), -1), (dict(n_layers=-1), -1), (dict(ffn=-256), -1),
    (dict(max_tokens=0), -1), (dict(max_batch=0), -1), (dict(max_seq=-3), -1),
    (dict(rms_eps=0.0), -1), (dict(rope_theta=-1.0), -1), (dict(rms_eps=float("nan")), -1),
    (dict(dtype=7), -1), (dict(out_dtype=2), -1), (dict(mrope_layout=3), -1), (dict(qk_norm=2), -1),
    (dict(head_dim=96, mrope_section=(16, 16, 16)), -5),   # head_dim not built
    (dict(hidden=2000), -5), (dict(ffn=6000), -5),
    (dict(n_q_heads=12, n_kv_heads=4), -5),          # group of 3 query heads
    (dict(max_tokens=1 << 24), -5),
    (dict(max_tokens=400_000), -5),                  # 400k x 6144 fp16 activations exceed 4 GiB
    (dict(max_tokens=200_000, dtype=0), -5),         # ... in fp32 already at 200k
    (dict(max_tokens=300_000), 0),
    (dict(weight_format=2), -1), (dict(weight_format=-1), -1),
    (dict(weight_format=1, dtype=0), -5),           # e4m3 weights need bf16 storage
])
def test_invalid_configs(B, kw, status):
    assert B.mte_config_validate(_full(B, **kw)) == status


def test_null_config(B):
    assert B.lib.mte_config_validate(None) == -1


def test_check_batch(B):
    cfg = _full(B, max_tokens=1000, max_batch=4, max_seq=320)
    assert B.mte_check_batch(cfg, [96, 320, 1]) == (0, 417)
    assert B.mte_check_batch(cfg, [96, 0])[0] == -1           # empty sequence
    assert B.mte_check_batch(cfg, [96, -4])[0] == -1
    assert B.mte_check_batch(cfg, [321])[0] == -2             # longer than max_seq
    assert B.mte_check_batch(cfg, [1] * 5)[0] == -2           # more than max_batch
    assert B.mte_check_batch(cfg, [320, 320, 320, 100])[0] == -2  # more than max_tokens
    assert B.mte_check_batch(cfg, [96], batch=0)[0] == -1
    assert B.mte_check_batch(None, [96])[0] == -1
    assert B.mte_check_batch(cfg, None, batch=1)[0] == -1


def test_encode_rejects_null_encoder(B):
    assert B.lib.mte_encode(None, 1, 1, B._i32([4]), 1, 1, None) == -1
    assert B.lib.mte_encode_layers(None, 1, 1, B._i32([4]), 1, 0, 1, 1, None) == -1
    assert B.lib.mte_timing_enable(None, 0, 4) == -1
    assert B.lib.mte_encoder_reserve_prefix(None, 80) == -1
    assert B.lib.mte_encode_prefixed(None, 1, 1, 80, 1, 1, B._i32([96]), 1, 1, 1, None) == -1
    B.lib.mte_encoder_destroy(None)  # no-op


def test_create_rejects_bad_arguments_before_hip(B):
    bad = _full(B, n_q_heads=16, n_kv_heads=5)
    h = ctypes.c_void_p()
    w = B.mte_weights(None, None)
    assert B.lib.mte_encoder_create(ctypes.byref(bad), ctypes.byref(w), None, ctypes.byref(h)) == -1
    good = _full(B)
    # null weights / null layer array / null final norm
    assert B.lib.mte_encoder_create(ctypes.byref(good), None, None, ctypes.byref(h)) == -1
    assert B.lib.mte_encoder_create(ctypes.byref(good), ctypes.byref(w), None, ctypes.byref(h)) == -1
    layers = (B.mte_layer_weights * 28)()
    w2 = B.mte_weights(layers, 1234)
    assert B.lib.mte_encoder_create(ctypes.byref(good), ctypes.byref(w2), None, ctypes.byref(h)) == -1
    assert h.value is None


@pytest.mark.parametrize("layouts", [
    [(0, 1, 8, 8, -1)],           # negative count
    [(0, 1, 0, 8, 32)],           # partially empty grid
    [(0, 0, 0, 0, 0)],            # empty sequence
    [(0, 1, 8, 8, 32), (-2, 0, 0, 0, 5)],
    [(0, 1, 4096, 4096, 0)],      # 2^24 tokens
])
def test_build_positions_rejects_bad_layouts(B, layouts):
    arr = (B.mte_seq_layout * len(layouts))(*[B.mte_seq_layout(*l) for l in layouts])
    assert B.lib.mte_build_positions(arr, len(layouts), 4096, None) == -1


def test_build_positions_rejects_null(B):
    arr = (B.mte_seq_layout * 1)(B.mte_seq_layout(0, 1, 2, 2, 1))
    assert B.lib.mte_build_positions(None, 1, 4096, None) == -1
    assert B.lib.mte_build_positions(arr, 1, None, None) == -1
    assert B.lib.mte_build_positions(arr, 0, 4096, None) == -1


def test_e4m3_config_valid(B):
    assert B.mte_config_validate(_full(B, weight_format=B.MTE_WEIGHTS_E4M3)) == 0
    assert ctypes.sizeof(B.mte_config) == 4 * 19   # 19 four-byte fields, as in mte.h


def test_probe_is_not_in_the_encoder_library(B):
    """The matrix-core probe is a benchmark instrument in its own library, not part of the
    encoder's ABI; it rejects bad arguments before any HIP call."""
    assert not hasattr(ctypes.CDLL(B.LIB_PATH), "mte_probe_mfma")
    probe = ctypes.CDLL(os.path.join(os.path.dirname(B.LIB_PATH), "libmte_probe.so"))
    probe.mte_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    assert probe.mte_probe_mfma(0, 10, 4096, None) == -1
    assert probe.mte_probe_mfma(4, 0, 4096, None) == -1
    assert probe.mte_probe_mfma(4, 10, None, None) == -1


def test_quantize_rejects_bad_arguments(B):
    q = B.lib.mte_quantize_e4m3_rows
    assert q(None, 1, 4, 4, 4096, 8192, None) == -1       # null source
    assert q(4096, 1, 4, 4, None, 8192, None) == -1       # null codes
    assert q(4096, 1, 4, 4, 4096, None, None) == -1       # null scales
    assert q(4096, 1, 0, 4, 4096, 8192, None) == -1       # no rows
    assert q(4096, 1, 4, -1, 4096, 8192, None) == -1      # no columns
    assert q(4096, 5, 4, 4, 4096, 8192, None) == -1       # bad dtype


def test_status_strings(B):
    for s in (0, -1, -2, -3, -4, -5, 17):
        assert isinstance(B.mte_status_string(s), str) and B.mte_status_string(s)


def _vision(B, **kw):
    args = dict(depth=24, hidden=1024, n_heads=16, head_dim=64, ffn=4096)
    args.update(kw)
    return B.make_vision_config(**args)


def test_vision_configs(B):
    assert B.mte_vision_config_validate(_vision(B)) == 0
    assert B.mte_vision_config_validate(_vision(B, depth=2, hidden=128, n_heads=2, ffn=256, out_hidden=256,
                                                dtype=0)) == 0
    assert B.lib.mte_vision_config_validate(None) == -1
    for kw, st in [(dict(hidden=1000), -1),                 # hidden != heads * head_dim
                   (dict(n_heads=10, hidden=960, head_dim=96), -5),
                   (dict(ffn=4000), -5), (dict(out_hidden=2000), -5),
                   (dict(patch=10), -5),                    # 3*10*10 not a multiple of 64
                   (dict(depth=-1), -1), (dict(max_images=0), -1), (dict(max_side=16), -1),
                   (dict(ln_eps=0.0), -1), (dict(dtype=3), -1),
                   (dict(hidden=8192, n_heads=64, head_dim=128), -5),
                   (dict(max_images=2100), -5),             # 2100 x 256 patches x 4096 fp16 exceed 4 GiB
                   (dict(max_images=2000), 0)]:
        assert B.mte_vision_config_validate(_vision(B, **kw)) == st, kw


def test_vision_rejects_bad_arguments(B):
    assert B.lib.mte_vision_encode(None, 4096, 1, 256, 256, 8192, None) == -1
    assert B.lib.mte_vision_encode_strided(None, 4096, 1, 256, 256, 8192, 96, None) == -1
    h = ctypes.c_void_p()
    good = _vision(B)
    w = B.mte_vision_weights()
    assert B.lib.mte_vision_create(ctypes.byref(good), ctypes.byref(w), None, ctypes.byref(h)) == -1
    assert B.lib.mte_vision_create(ctypes.byref(good), None, None, ctypes.byref(h)) == -1
    B.lib.mte_vision_destroy(None)

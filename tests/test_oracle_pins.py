"""Pins of the fp64 CPU oracle against things other than itself.

Each check compares the oracle with a closed form worked by hand (fixtures in
tests/golden), a brute-force scalar implementation written differently (the
rotary embedding as complex multiplication, attention over the whole packed
batch with an explicit block-diagonal causal mask), or an invariant of the
mathematics. The last group plants mistakes in the oracle (on the CPU) and
asserts that at least one pin catches each of them.
"""
import cmath
import json
import math
import os

import numpy as np
import pytest

from oracle import te_oracle as O
from synth import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ------------------------------------------------------------- brute force
def bf_linear(Wm, x):
    return [sum(Wm[i][k] * x[k] for k in range(len(x))) for i in range(len(Wm))]


def bf_rms(x, g, eps):
    s = sum(v * v for v in x) / len(x)
    r = 1.0 / math.sqrt(s + eps)
    return [v * r * gi for v, gi in zip(x, g)]


def bf_rotate(z, pos3, section, theta):
    """Rotary embedding as complex multiplication, contiguous t/h/w sections."""
    d = len(z)
    half = d // 2
    out = [0.0] * d
    for j in range(half):
        axis = 0 if j < section[0] else (1 if j < section[0] + section[1] else 2)
        ang = pos3[axis] * theta ** (-2.0 * j / d)
        c = complex(z[j], z[j + half]) * cmath.exp(1j * ang)
        out[j], out[j + half] = c.real, c.imag
    return out


def bf_layer(x, pos, seq_ids, w, dims):
    """One decoder layer over a packed batch with scalar Python loops."""
    T, D = len(x), len(x[0])
    hq, hkv, hd = dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    eps = dims.rms_eps
    L = {k: v.astype(float).tolist() for k, v in w.items()}
    q, k, v = [], [], []
    for i in range(T):
        a = bf_rms(x[i], L["attn_norm"], eps)
        qi, ki, vi = bf_linear(L["w_q"], a), bf_linear(L["w_k"], a), bf_linear(L["w_v"], a)
        qh = [qi[h * hd:(h + 1) * hd] for h in range(hq)]
        kh = [ki[h * hd:(h + 1) * hd] for h in range(hkv)]
        vh = [vi[h * hd:(h + 1) * hd] for h in range(hkv)]
        if dims.qk_norm:
            qh = [bf_rms(z, L["q_norm"], eps) for z in qh]
            kh = [bf_rms(z, L["k_norm"], eps) for z in kh]
        p3 = [int(pos[0][i]), int(pos[1][i]), int(pos[2][i])]
        qh = [bf_rotate(z, p3, dims.mrope_section, dims.rope_theta) for z in qh]
        kh = [bf_rotate(z, p3, dims.mrope_section, dims.rope_theta) for z in kh]
        q.append(qh); k.append(kh); v.append(vh)
    out = []
    for i in range(T):
        o = []
        for h in range(hq):
            g = h // (hq // hkv)
            allowed = [j for j in range(T) if seq_ids[j] == seq_ids[i] and j <= i]
            sc = [sum(q[i][h][c] * k[j][g][c] for c in range(hd)) / math.sqrt(hd) for j in allowed]
            m = max(sc)
            e = [math.exp(s - m) for s in sc]
            z = sum(e)
            o += [sum(e[n] / z * v[j][g][c] for n, j in enumerate(allowed)) for c in range(hd)]
        y = bf_linear(L["w_o"], o)
        xi = [x[i][c] + y[c] for c in range(D)]
        m = bf_rms(xi, L["mlp_norm"], eps)
        gt, up = bf_linear(L["w_gate"], m), bf_linear(L["w_up"], m)
        act = [gg / (1.0 + math.exp(-gg)) * uu for gg, uu in zip(gt, up)]
        dn = bf_linear(L["w_down"], act)
        out.append([xi[c] + dn[c] for c in range(D)])
    return out


MICRO = W.Dims(n_layers=2, hidden=12, n_q_heads=2, n_kv_heads=1, head_dim=6, ffn=10,
               mrope_section=(1, 1, 1), rope_theta=10.0, dtype="f32")


def _micro_weights(dims, layer, scale=0.4):
    rng = np.random.default_rng(100 + layer)
    d, hq, hkv, hd, f = dims.hidden, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.ffn
    g = lambda n: 1.0 + rng.uniform(-0.5, 0.5, n)
    return {
        "attn_norm": g(d), "w_q": rng.normal(0, scale, (hq * hd, d)),
        "w_k": rng.normal(0, scale, (hkv * hd, d)), "w_v": rng.normal(0, scale, (hkv * hd, d)),
        "q_norm": g(hd), "k_norm": g(hd), "w_o": rng.normal(0, scale, (d, hq * hd)),
        "mlp_norm": g(d), "w_gate": rng.normal(0, scale, (f, d)),
        "w_up": rng.normal(0, scale, (f, d)), "w_down": rng.normal(0, scale, (d, f)),
    }


def _micro_inputs(lens=(3, 2), seed=5):
    rng = np.random.default_rng(seed)
    T = sum(lens)
    x = rng.normal(0, 1, (T, MICRO.hidden))
    pos = rng.integers(0, 9, (3, T))
    ids = sum(([s] * L for s, L in enumerate(lens)), [])
    return x, pos, ids, list(lens)


# ------------------------------------------------------------------ checks
def check_layer_brute_force(qk_norm=1):
    dims = MICRO.with_(qk_norm=qk_norm)
    x, pos, ids, lens = _micro_inputs()
    w = _micro_weights(dims, 0)
    ref = np.array(bf_layer(x.tolist(), pos.tolist(), ids, w, dims))
    got = O.layer_forward(x, pos, lens, w, dims)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


def check_rmsnorm_closed_form():
    for c in _gold("closed_forms.json")["rmsnorm"]:
        y = O.rmsnorm(np.array(c["x"], float), np.array(c["g"], float), c["eps"])
        np.testing.assert_allclose(y, c["y"], rtol=1e-14, atol=0)


def check_silu_closed_form():
    c = _gold("closed_forms.json")["silu"]
    np.testing.assert_allclose(O.silu(np.array(c["z"], float)), c["y"], rtol=1e-14, atol=1e-300)


def check_attention_two_tokens():
    c = _gold("closed_forms.json")["attention_two_tokens"]
    q = np.array(c["q"], float)[:, None, :]
    k = np.array(c["k"], float)[:, None, :]
    v = np.array(c["v"], float)[:, None, :]
    np.testing.assert_allclose(O.causal_attention(q, k, v)[:, 0, :], c["o"], rtol=1e-14)


def check_rotary_closed_form():
    c = _gold("closed_forms.json")["rotary"]
    d = 64
    z = np.zeros((1, 1, d)); z[0, 0, 0] = 1.0
    pos = np.array([[1], [1], [1]])
    r = O.mrope(z, pos, d, c["theta"], (12, 10, 10), 0)
    np.testing.assert_allclose([r[0, 0, 0], r[0, 0, d // 2]], c["pair0_unit_at_pos1"], rtol=1e-14)
    np.testing.assert_allclose(O.inv_freq(d, c["theta"])[d // 4], c["pair_quarter_inv_freq"], rtol=1e-13)


def check_axis_only_positions(layout=0):
    """Position (p,0,0) turns exactly the t pairs, (0,p,0) the h pairs, (0,0,p) the w pairs."""
    d, sec = 64, (12, 10, 10)
    if layout == 0:
        expect = {0: set(range(0, 12)), 1: set(range(12, 22)), 2: set(range(22, 32))}
    else:  # interleaved: h at j%3==1 (j<30), w at j%3==2 (j<30), t elsewhere
        expect = {1: {j for j in range(32) if j % 3 == 1 and j < 30},
                  2: {j for j in range(32) if j % 3 == 2 and j < 30}}
        expect[0] = set(range(32)) - expect[1] - expect[2]
    rng = np.random.default_rng(3)
    z = rng.normal(size=(1, 1, d))
    for axis in range(3):
        pos = np.zeros((3, 1), np.int64); pos[axis, 0] = 3
        r = O.mrope(z, pos, d, 5e6, sec, layout)
        moved = {j for j in range(d // 2)
                 if abs(r[0, 0, j] - z[0, 0, j]) + abs(r[0, 0, j + d // 2] - z[0, 0, j + d // 2]) > 1e-12}
        assert moved == expect[axis], (axis, sorted(moved))


def check_positions_golden():
    for c in _gold("positions.json")["cases"]:
        s = W.SeqLayout(*c["layout"])
        p = O.positions([s])
        if "t" in c:
            assert p[0].tolist() == c["t"] and p[1].tolist() == c["h"] and p[2].tolist() == c["w"]
        else:
            ts = c["text_start"]
            assert p[0, ts] == c["text_positions_first"] and p[0, -1] == c["text_positions_last"]
            assert (p[:, ts:] == p[0, ts:]).all()
            assert p[1, 19] == c["image_h_of_token_19"] and p[2, 19] == c["image_w_of_token_19"]
            assert (p[0, :ts] == 0).all()


def check_gqa_grouping():
    """Query heads 0,1 read kv head 0; heads 2,3 read kv head 1 (contiguous groups)."""
    rng = np.random.default_rng(4)
    L, d = 5, 8
    q = rng.normal(size=(L, 4, d)); k = rng.normal(size=(L, 2, d))
    v = np.zeros((L, 2, d)); v[:, 1, :] = 1.0
    o = O.causal_attention(q, k, v)
    np.testing.assert_allclose(o[:, :2, :], 0.0, atol=1e-15)
    np.testing.assert_allclose(o[:, 2:, :], 1.0, rtol=1e-14)


def check_causal_prefix():
    rng = np.random.default_rng(6)
    L, d = 7, 8
    q, k, v = (rng.normal(size=(L, 2, d)) for _ in range(3))
    o1 = O.causal_attention(q, k, v)
    k2, v2 = k.copy(), v.copy(); k2[4:] += 3.0; v2[4:] -= 2.0
    o2 = O.causal_attention(q, k2, v2)
    np.testing.assert_array_equal(o1[:4], o2[:4])
    assert np.abs(o1[4:] - o2[4:]).max() > 1e-3


# -------------------------------------------------------------- the pins
def test_layer_matches_scalar_brute_force():
    check_layer_brute_force(qk_norm=1)
    check_layer_brute_force(qk_norm=0)


def test_rmsnorm_closed_form():
    check_rmsnorm_closed_form()


def test_silu_closed_form():
    check_silu_closed_form()


def test_attention_two_token_closed_form():
    check_attention_two_tokens()


def test_rotary_closed_form():
    check_rotary_closed_form()


@pytest.mark.parametrize("layout", [0, 1])
def test_axis_only_positions_turn_their_pairs(layout):
    check_axis_only_positions(layout)


def test_positions_golden():
    check_positions_golden()


def test_gqa_contiguous_grouping():
    check_gqa_grouping()


def test_causal_prefix_invariance():
    check_causal_prefix()


def test_attention_single_token_is_v():
    rng = np.random.default_rng(1)
    q, k, v = (rng.normal(size=(1, 4, 16)) for _ in range(3))
    k, v = k[:, :2], v[:, :2]
    o = O.causal_attention(q, k, v)
    np.testing.assert_allclose(o, np.repeat(v, 2, axis=1), rtol=1e-15)


def test_attention_identical_keys_prefix_mean():
    rng = np.random.default_rng(2)
    L, d = 6, 8
    q = rng.normal(size=(L, 2, d)); k = np.repeat(rng.normal(size=(1, 1, d)), L, 0).repeat(2, 1)
    v = rng.normal(size=(L, 2, d))
    o = O.causal_attention(q, k, v)
    mean = np.cumsum(v, axis=0) / np.arange(1, L + 1)[:, None, None]
    np.testing.assert_allclose(o, mean, rtol=1e-12)


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(8)
    L, d = 9, 16
    q, k = rng.normal(size=(L, 4, d)) * 3, rng.normal(size=(L, 2, d)) * 3
    o = O.causal_attention(q, k, np.ones((L, 2, d)))
    np.testing.assert_allclose(o, 1.0, rtol=1e-14)


def test_gqa_equals_mha_with_duplicated_kv():
    rng = np.random.default_rng(9)
    L, d = 6, 8
    q = rng.normal(size=(L, 6, d)); k, v = rng.normal(size=(L, 2, d)), rng.normal(size=(L, 2, d))
    o = O.causal_attention(q, k, v)
    for h in range(6):
        ref = O.causal_attention(q[:, h:h + 1], k[:, h // 3:h // 3 + 1], v[:, h // 3:h // 3 + 1])
        np.testing.assert_allclose(o[:, h:h + 1], ref, rtol=1e-14)


@pytest.mark.parametrize("layout", [0, 1])
def test_rotary_preserves_pair_norms_and_zero_is_identity(layout):
    rng = np.random.default_rng(10)
    d = 128
    z = rng.normal(size=(7, 3, d))
    pos = rng.integers(0, 400, size=(3, 7))
    r = O.mrope(z, pos, d, 5e6, (24, 20, 20), layout)
    nz = z[..., :64] ** 2 + z[..., 64:] ** 2
    nr = r[..., :64] ** 2 + r[..., 64:] ** 2
    np.testing.assert_allclose(nr, nz, rtol=1e-12)
    r0 = O.mrope(z, np.zeros((3, 7), np.int64), d, 5e6, (24, 20, 20), layout)
    np.testing.assert_array_equal(r0, z)


@pytest.mark.parametrize("layout", [0, 1])
def test_mrope_with_equal_axes_is_1d_rope(layout):
    rng = np.random.default_rng(12)
    d = 64
    z = rng.normal(size=(5, 2, d))
    p = rng.integers(0, 300, size=5)
    r = O.mrope(z, np.stack([p, p, p]), d, 5e6, (12, 10, 10), layout)
    for i in range(5):
        for h in range(2):
            ref = bf_rotate(z[i, h].tolist(), [p[i]] * 3, (32, 0, 0), 5e6)
            np.testing.assert_allclose(r[i, h], ref, rtol=1e-10, atol=1e-12)


def test_relative_position_property():
    """q(m).k(n) depends only on per-axis position differences."""
    rng = np.random.default_rng(13)
    d = 64
    q, k = rng.normal(size=(1, 1, d)), rng.normal(size=(1, 1, d))
    pm, pn = np.array([[5], [2], [7]]), np.array([[1], [4], [3]])
    s = np.array([[11], [3], [6]])
    rot = lambda z, p: O.mrope(z, p, d, 5e6, (12, 10, 10), 0)
    a = np.sum(rot(q, pm) * rot(k, pn))
    b = np.sum(rot(q, pm + s) * rot(k, pn + s))
    assert abs(a - b) < 1e-12 * (1 + abs(a))


def _stack_case(lens=(4, 3, 5), n_layers=2, seed=21):
    dims = MICRO.with_(n_layers=n_layers)
    rng = np.random.default_rng(seed)
    x = rng.normal(0, 1, (sum(lens), dims.hidden))
    layouts = [W.SeqLayout(0, 1, 1, 2, L - 2) for L in lens]
    pos = O.positions(layouts)
    g = 1.0 + rng.uniform(-0.5, 0.5, dims.hidden)
    return dims, x, pos, list(lens), g


def _run(dims, x, pos, lens, g, n_layers=None, wfn=None):
    return O.encode(x, pos, lens, dims, wfn or (lambda l: _micro_weights(dims, l)), g, n_layers=n_layers)


def test_packed_batch_equals_each_sequence_alone():
    dims, x, pos, lens, g = _stack_case()
    full = _run(dims, x, pos, lens, g)
    start = 0
    for L in lens:
        sl = slice(start, start + L)
        np.testing.assert_allclose(full[sl], _run(dims, x[sl], pos[:, sl], [L], g), rtol=1e-12, atol=1e-12)
        start += L


def test_batch_permutation_equivariance():
    dims, x, pos, lens, g = _stack_case()
    full = _run(dims, x, pos, lens, g)
    starts = np.cumsum([0] + lens)
    perm = [2, 0, 1]
    idx = np.concatenate([np.arange(starts[i], starts[i + 1]) for i in perm])
    out = _run(dims, x[idx], pos[:, idx], [lens[i] for i in perm], g)
    np.testing.assert_allclose(out, full[idx], rtol=1e-12, atol=1e-12)


def test_zero_layers_is_final_norm():
    dims, x, pos, lens, g = _stack_case()
    out = _run(dims, x, pos, lens, g, n_layers=0)
    ms = np.mean(x * x, axis=1, keepdims=True)
    np.testing.assert_allclose(out, x / np.sqrt(ms + dims.rms_eps) * g, rtol=1e-14)


def test_zero_output_projections_make_layers_identity():
    dims, x, pos, lens, g = _stack_case()

    def wz(l):
        w = _micro_weights(dims, l)
        w["w_o"] = np.zeros_like(w["w_o"]); w["w_down"] = np.zeros_like(w["w_down"])
        return w
    np.testing.assert_allclose(_run(dims, x, pos, lens, g, wfn=wz), _run(dims, x, pos, lens, g, n_layers=0), rtol=1e-14)


def test_uniform_position_shift_invariance():
    dims, x, pos, lens, g = _stack_case(lens=(6,))
    a = _run(dims, x, pos, lens, g)
    b = _run(dims, x, pos + 17, lens, g)
    np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)


# ---------------------------------------------------- planted mistakes
def _mut_rope_sign(z, pos, head_dim, theta, section, layout, _orig=O.mrope):
    return _orig(z, -pos, head_dim, theta, section, layout)


def _mut_inv_freq(head_dim, theta):
    j = np.arange(head_dim // 2, dtype=float)
    return np.power(float(theta), -1.0 * j / head_dim)


def _mut_pair_axis(head_dim, section, layout, _orig=O.pair_axis):
    return _orig(head_dim, section, layout)[::-1].copy()


def _mut_rms_no_gain(x, g, eps):
    x = x.astype(float)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def _mut_silu_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def _mut_attn_scale(q, k, v, _orig=O.causal_attention):
    return _orig(q / math.sqrt(q.shape[-1]), k, v)


def _mut_attn_nomask(q, k, v):
    L, hq, d = q.shape
    rep = hq // k.shape[1]
    o = np.empty_like(q)
    for h in range(hq):
        s = q[:, h] @ k[:, h // rep].T / math.sqrt(d)
        p = np.exp(s - s.max(1, keepdims=True)); p /= p.sum(1, keepdims=True)
        o[:, h] = p @ v[:, h // rep]
    return o


def _mut_attn_grouping(q, k, v):
    L, hq, d = q.shape
    hkv = k.shape[1]
    o = np.empty_like(q)
    mask = np.triu(np.ones((L, L), bool), 1)
    for h in range(hq):
        s = np.where(mask, -np.inf, q[:, h] @ k[:, h % hkv].T / math.sqrt(d))
        p = np.exp(s - s.max(1, keepdims=True)); p /= p.sum(1, keepdims=True)
        o[:, h] = p @ v[:, h % hkv]
    return o


def _mut_positions(layouts, _orig=O.positions):
    p = _orig(layouts)
    return p[[0, 2, 1]]


def _all_pins():
    for f in (check_layer_brute_force, check_rmsnorm_closed_form, check_silu_closed_form,
              check_attention_two_tokens, check_rotary_closed_form, check_axis_only_positions,
              check_positions_golden, check_gqa_grouping, check_causal_prefix):
        f()


@pytest.mark.parametrize("name,mutant", [
    ("mrope", _mut_rope_sign), ("inv_freq", _mut_inv_freq), ("pair_axis", _mut_pair_axis),
    ("rmsnorm", _mut_rms_no_gain), ("silu", _mut_silu_sigmoid),
    ("causal_attention", _mut_attn_scale), ("causal_attention", _mut_attn_nomask),
    ("causal_attention", _mut_attn_grouping), ("positions", _mut_positions),
])
def test_planted_mistake_is_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(O, name, mutant)
    with pytest.raises(AssertionError):
        _all_pins()


def test_planted_transposed_projection_is_caught(monkeypatch):
    orig = O.layer_forward

    def lf(x, pos, seq_lens, w, dims):
        w = dict(w); w["w_q"] = np.ascontiguousarray(w["w_q"].T)
        return orig(x, pos, seq_lens, w, dims)
    monkeypatch.setattr(O, "layer_forward", lf)
    with pytest.raises(AssertionError):
        check_layer_brute_force()


def test_planted_dropped_residual_is_caught(monkeypatch):
    orig = O.layer_forward

    def lf(x, pos, seq_lens, w, dims):
        return orig(x, pos, seq_lens, w, dims) - x
    monkeypatch.setattr(O, "layer_forward", lf)
    with pytest.raises(AssertionError):
        check_layer_brute_force()

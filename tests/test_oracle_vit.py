"""Pins of the vision-tower oracle (oracle/vit_oracle.py) against things other
than itself: pixel bookkeeping checked by decoding tagged pixel values, the
merge-group structure, invariants of LayerNorm, the GELU identity
gelu(z) - gelu(-z) = z and its distance to the erf form, the relative-position
property of the 2-D rotary embedding and a hand rotation, attention by scalar
brute force and its permutation equivariance, equivariance of a whole block
under permuting patches with their positions, and the merger's gather by
explicit loops. The last test plants mistakes and checks that a pin fails."""
import math

import numpy as np
import pytest

from oracle import vit_oracle as V
from synth import vision as SV


def _tagged_images(n, C, h, w):
    # pixel value encodes (image, channel, y, x) exactly in float64
    i, c, y, x = np.meshgrid(np.arange(n), np.arange(C), np.arange(h), np.arange(w), indexing="ij")
    return (((i * C + c) * h + y) * w + x).astype(np.float64)


def test_patchify_pixel_bookkeeping():
    n, C, h, w, p, m = 2, 3, 64, 96, 16, 2
    img = _tagged_images(n, C, h, w)
    P = V.patchify(img, p, m)
    per = (h // p) * (w // p)
    assert P.shape == (n * per, C * p * p)
    gw = w // (p * m)
    for row in range(P.shape[0]):
        i, t = divmod(row, per)
        grp, inner = divmod(t, m * m)
        ph = (grp // gw) * m + inner // m
        pw = (grp % gw) * m + inner % m
        for k in (0, 17, 255, 256, 511, 767):
            c, ky, kx = k // (p * p), (k // p) % p, k % p
            code = int(P[row, k])
            xx = code % w; code //= w
            yy = code % h; code //= h
            cc = code % C; ii = code // C
            assert (ii, cc, yy, xx) == (i, c, ph * p + ky, pw * p + kx)


def test_patch_grid_is_merge_groups():
    rows, cols = V.patch_grid(64, 96, 16, 2)
    assert len(rows) == 24 and len(set(zip(rows, cols))) == 24          # every patch once
    for t in range(6):
        r4, c4 = rows[4 * t:4 * t + 4], cols[4 * t:4 * t + 4]
        a, b = divmod(t, 3)                                            # groups row-major
        assert list(r4) == [2 * a, 2 * a, 2 * a + 1, 2 * a + 1]
        assert list(c4) == [2 * b, 2 * b + 1, 2 * b, 2 * b + 1]


def test_layernorm_invariants_and_scalar():
    rng = np.random.default_rng(1)
    x = rng.normal(3.0, 2.0, (5, 64))
    g = rng.uniform(0.5, 1.5, 64)
    b = rng.normal(0, 0.1, 64)
    y = V.layernorm(x, g, b, 0.0)
    z = (y - b) / g
    assert np.allclose(z.mean(axis=1), 0, atol=1e-12)
    assert np.allclose((z * z).mean(axis=1), 1, atol=1e-12)
    assert np.allclose(V.layernorm(x + 7.5, g, b, 0.0), y, atol=1e-12)     # shift invariance
    assert np.allclose(V.layernorm(x * 4.0, g, b, 0.0), y, atol=1e-12)     # scale invariance
    v = [float(t) for t in x[2]]
    mu = sum(v) / 64
    var = sum((t - mu) ** 2 for t in v) / 64
    ref = [(t - mu) / math.sqrt(var + 1e-6) * gi + bi for t, gi, bi in zip(v, g, b)]
    assert np.allclose(V.layernorm(x[2:3], g, b, 1e-6)[0], ref, rtol=0, atol=1e-12)


def test_gelu_identity_and_erf_distance():
    z = np.linspace(-8, 8, 2001)
    gz = V.gelu_tanh(z)
    assert np.allclose(gz - V.gelu_tanh(-z), z, atol=1e-12)
    assert V.gelu_tanh(np.array([0.0]))[0] == 0.0
    erf = np.array([0.5 * t * (1 + math.erf(t / math.sqrt(2))) for t in z])
    assert np.max(np.abs(gz - erf)) < 1e-3                              # the tanh form's known accuracy
    assert abs(V.gelu_tanh(np.array([10.0]))[0] - 10.0) < 1e-12


def test_rope2d_relative_and_hand_rotation():
    rng = np.random.default_rng(2)
    d, th = 64, 10000.0
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, d))
    def dot(r1, c1, r2, c2):
        a = V.rope2d(q, np.array([r1]), np.array([c1]), d, th)
        b = V.rope2d(k, np.array([r2]), np.array([c2]), d, th)
        return float((a * b).sum())
    assert math.isclose(dot(3, 5, 1, 2), dot(7, 9, 5, 6), rel_tol=1e-12, abs_tol=1e-12)     # only (dr, dc) matters
    assert not math.isclose(dot(3, 5, 1, 2), dot(3, 6, 1, 2), rel_tol=1e-6)
    assert np.allclose(V.rope2d(q, np.array([0]), np.array([0]), d, th), q)
    # pair j = 3 (< d/4: row-driven) and j = 20 (column-driven), by complex multiplication
    z = V.rope2d(q, np.array([5]), np.array([11]), d, th)[0, 0]
    for j, p in ((3, 5), (20, 11)):
        w = complex(q[0, 0, j], q[0, 0, j + d // 2]) * complex(math.cos(p * th ** (-2 * j / d)),
                                                               math.sin(p * th ** (-2 * j / d)))
        assert math.isclose(z[j], w.real, abs_tol=1e-12) and math.isclose(z[j + d // 2], w.imag, abs_tol=1e-12)


def test_full_attention_brute_force_and_equivariance():
    rng = np.random.default_rng(3)
    L, H, d = 6, 2, 4
    q, k, v = (rng.standard_normal((L, H, d)) for _ in range(3))
    o = V.full_attention(q, k, v)
    for i in range(L):
        for h in range(H):
            s = [sum(q[i, h, t] * k[j, h, t] for t in range(d)) / math.sqrt(d) for j in range(L)]
            mx = max(s)
            e = [math.exp(t - mx) for t in s]
            ref = [sum(e[j] * v[j, h, t] for j in range(L)) / sum(e) for t in range(d)]
            assert np.allclose(o[i, h], ref, atol=1e-12)
    perm = rng.permutation(L)
    assert np.allclose(V.full_attention(q[perm], k[perm], v[perm]), o[perm], atol=1e-12)


def test_block_equivariant_under_patch_permutation():
    v = SV.VDIMS_TINY
    w = SV.block_weights(v, 0)
    rows, cols = V.patch_grid(64, 64, 16, 2)
    x = np.random.default_rng(4).standard_normal((16, v.hidden))
    y = V.block_forward(x, rows, cols, 16, w, v)
    perm = np.random.default_rng(5).permutation(16)
    y2 = V.block_forward(x[perm], rows[perm], cols[perm], 16, w, v)
    assert np.allclose(y2, y[perm], atol=1e-10)
    # positions matter: the same patches with their positions swapped give another result
    y3 = V.block_forward(x, cols, rows, 16, w, v)
    assert not np.allclose(y3, y, atol=1e-6)


def test_merger_gathers_groups_in_order():
    v = SV.VDIMS_TINY
    outer = SV.outer_weights(v)
    x = np.random.default_rng(6).standard_normal((8, v.hidden))
    got = V.merge_tokens(x, outer, v)
    y = V.layernorm(x, outer["merge_ln_g"], outer["merge_ln_b"], v.ln_eps)
    W1, b1 = outer["merge_w1"].astype(np.float64), outer["merge_b1"].astype(np.float64)
    W2, b2 = outer["merge_w2"].astype(np.float64), outer["merge_b2"].astype(np.float64)
    for t in range(2):
        u = np.zeros(4 * v.hidden)
        for j in range(4):
            for c in range(v.hidden):
                u[j * v.hidden + c] = y[4 * t + j, c]
        z = W1 @ u + b1
        ref = W2 @ (0.5 * z * (1 + np.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3)))) + b2
        assert np.allclose(got[t], ref, atol=1e-10)


def test_encode_shapes_and_image_independence():
    v = SV.VDIMS_TINY
    img = SV.images(v, 2, 64, 96)
    bw = lambda l: SV.block_weights(v, l)
    both = V.encode(img, v, bw, SV.outer_weights(v))
    assert both.shape == (2 * 6, v.out_hidden)
    one = V.encode(img[1:], v, bw, SV.outer_weights(v))
    assert np.allclose(both[6:], one, atol=1e-10)                      # images do not interact


def test_pins_catch_planted_mistakes(monkeypatch):
    rng = np.random.default_rng(7)
    x = rng.normal(3.0, 2.0, (5, 64))
    g, b = np.ones(64), np.zeros(64)
    # LayerNorm with the unbiased variance
    unbiased = lambda x, g, b, eps: (x - x.mean(-1, keepdims=True)) / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps) * g + b
    z = unbiased(x, g, b, 0.0)
    assert not np.allclose((z * z).mean(axis=1), 1, atol=1e-6)
    # gelu with the wrong cubic sign
    bad = lambda z: 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z - 0.044715 * z ** 3)))
    zz = np.linspace(-8, 8, 2001)
    erf = np.array([0.5 * t * (1 + math.erf(t / math.sqrt(2))) for t in zz])
    assert np.max(np.abs(bad(zz) - erf)) > 1e-3
    # rows and columns swapped inside the rotary embedding
    real = V.rope2d
    monkeypatch.setattr(V, "rope2d", lambda z, r, c, d, th: real(z, c, r, d, th))
    q = rng.standard_normal((1, 1, 64))
    zr = V.rope2d(q, np.array([5]), np.array([11]), 64, 10000.0)[0, 0]
    w = complex(q[0, 0, 3], q[0, 0, 35]) * complex(math.cos(5 * 10000.0 ** (-6 / 64)), math.sin(5 * 10000.0 ** (-6 / 64)))
    assert not math.isclose(zr[3], w.real, abs_tol=1e-9)
    monkeypatch.setattr(V, "rope2d", real)
    # causal attention breaks permutation equivariance
    L, H, d = 6, 2, 4
    q, k, v = (rng.standard_normal((L, H, d)) for _ in range(3))
    from oracle import te_oracle as O
    o = O.causal_attention(q, k, v)
    perm = rng.permutation(L)
    assert not np.allclose(O.causal_attention(q[perm], k[perm], v[perm]), o[perm], atol=1e-6)

"""Pins of the e4m3 weight-format oracle (oracle/e4m3.py) against things
other than itself: the format's defining constants, torch's own float8_e4m3fn
conversion (a library routine: decoding of every code, round-to-nearest-even
coding of in-range values), the definition of the row scale checked by brute
force, and the half-quantum error bound of rounding. The last group plants
mistakes in the oracle and asserts that a pin catches each."""
import numpy as np
import pytest
import torch

from oracle import e4m3 as Q


def _torch_codes(x):
    c = torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return np.where(c == 0x80, 0, c).astype(np.uint8)          # the oracle codes zero as +0


# ----------------------------------------------------------- format constants
def test_defining_values():
    t = Q.decode_table()
    assert t[0x7E] == 448.0 and t[0xFE] == -448.0                 # largest finite
    assert t[0x01] == 2.0 ** -9                                    # smallest subnormal
    assert t[0x07] == 7 * 2.0 ** -9                                # largest subnormal
    assert t[0x08] == 2.0 ** -6                                    # smallest normal
    assert t[0x38] == 1.0 and t[0x40] == 2.0 and t[0x39] == 1.125
    assert np.isnan(t[0x7F]) and np.isnan(t[0xFF])
    assert t[0x00] == 0.0 and t[0x80] == 0.0
    fin = np.isfinite(t)
    assert fin.sum() == 254
    assert np.array_equal(t[0x80:][fin[0x80:]], -t[:0x80][fin[:0x80]])   # sign symmetry


def test_decode_matches_torch():
    lib = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    t = Q.decode_table()
    fin = np.isfinite(lib)
    assert np.array_equal(np.isnan(t), np.isnan(lib))
    assert np.array_equal(t[fin], lib[fin])


# -------------------------------------------------------------------- coding
def test_round_trip_every_code():
    t = Q.decode_table()
    for c in range(256):
        if np.isfinite(t[c]):
            assert Q.encode(np.array(t[c]))[()] == (0 if c == 0x80 else c)


def test_ties_go_to_even_significand():
    # midpoints between neighbours: (1, 1.125) -> 1, (1.125, 1.25) -> 1.25,
    # (0, 2^-9) -> 0, (7, 8) * 2^-9 -> 2^-6, (416, 448) -> 448, (-1, -1.125) -> -1
    x = np.array([1.0625, 1.1875, 2.0 ** -10, 7.5 * 2.0 ** -9, 432.0, -1.0625])
    assert Q.encode(x).tolist() == [0x38, 0x3A, 0x00, 0x08, 0x7E, 0xB8]


def test_coding_matches_torch():
    rng = np.random.default_rng(5)
    # every binade of the range, plus exact midpoints and the ends
    x = np.concatenate([
        rng.uniform(-448, 448, 4000),
        np.sign(rng.standard_normal(4000)) * 2.0 ** rng.uniform(-12, np.log2(448), 4000),
        (Q.decode_table()[1:0x7E] + Q.decode_table()[2:0x7F]) / 2,          # midpoints
        np.array([0.0, -0.0, 448.0, -448.0, 2.0 ** -10, 2.0 ** -11]),
    ]).astype(np.float32)
    assert np.array_equal(Q.encode(x), _torch_codes(x))


def test_out_of_range_is_refused():
    with pytest.raises(ValueError):
        Q.encode(np.array([448.5]))
    with pytest.raises(ValueError):
        Q.encode(np.array([np.nan]))


# ---------------------------------------------------------------- row scales
def test_row_scale_is_the_smallest_power_of_two():
    rng = np.random.default_rng(6)
    amax = np.concatenate([2.0 ** rng.uniform(-30, 30, 500), [448.0, 449.0, 224.0, 1.0, 2.0 ** -20]])
    for a in amax:
        e = Q.row_scale_exponent(float(a))
        assert a <= 448.0 * 2.0 ** e and not a <= 448.0 * 2.0 ** (e - 1)
    assert Q.row_scale_exponent(0.0) == 0
    assert Q.row_scale_exponent(448.0) == 0 and Q.row_scale_exponent(449.0) == 1


def test_quantize_rows_error_bound():
    rng = np.random.default_rng(7)
    w = rng.normal(0, 0.02, (64, 256))
    w[3] = 0.0                                          # an all-zero row
    w[5] *= 1e-6                                        # a tiny row
    w[9, 17] = 3.0                                      # an outlier
    codes, scales = Q.quantize_rows(w)
    deq = Q.dequantize_rows(codes, scales)
    assert scales[3] == 1.0 and not codes[3].any()
    amax = np.abs(w).max(axis=1)
    assert np.all(amax[amax > 0] / scales[amax > 0] > 224) and np.all(amax / scales <= 448)
    # rounding to nearest: at most half a quantum, 2^-4 relative for
    # normals, 2^-10 * scale in the subnormal range
    bound = np.maximum(np.abs(w) * 2.0 ** -4, 2.0 ** -10 * scales[:, None])
    assert np.all(np.abs(deq - w) <= bound)
    # and it is the nearest: no other code of the row's scale is closer
    t = Q.decode_table()
    fin = t[np.isfinite(t)]
    for r in (0, 9, 5):
        cand = fin[None, :] * scales[r]
        best = np.min(np.abs(cand - w[r][:, None]), axis=1)
        assert np.all(np.abs(deq[r] - w[r]) == best)


# ------------------------------------------------------- planted mistakes
def test_pins_catch_planted_mistakes(monkeypatch):
    x = np.array([1.0625, 1.1875, 2.0 ** -10, 7.5 * 2.0 ** -9, 432.0, -1.0625])
    want = [0x38, 0x3A, 0x00, 0x08, 0x7E, 0xB8]
    real_decode = Q.decode
    # wrong exponent bias
    monkeypatch.setattr(Q, "decode", lambda c: real_decode(c) * (2.0 if (c >> 3) & 0xF else 1.0))
    assert Q.decode_table()[0x38] != 1.0
    monkeypatch.setattr(Q, "decode", real_decode)
    # subnormals scaled as normals: (1 + m/8) * 2^-7 at exponent 0
    monkeypatch.setattr(Q, "decode", lambda c: (real_decode(c) if (c >> 3) & 0xF else
                                                (1 + (c & 7) / 8) * 2.0 ** -7 * (-1 if c & 0x80 else 1)))
    lib = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()
    assert not np.array_equal(Q.decode_table()[1:8], lib[1:8])
    monkeypatch.setattr(Q, "decode", real_decode)
    # ties away from zero instead of to even
    real_encode = Q.encode

    def away(v):
        v = np.asarray(v, dtype=np.float64)
        t = Q.decode_table()[:0x7F]
        out = []
        for a in np.abs(v).ravel():
            d = np.abs(t - a)
            cand = np.flatnonzero(d == d.min())
            out.append(cand.max())
        mag = np.array(out)
        return (mag | np.where((v.ravel() < 0) & (mag != 0), 0x80, 0)).astype(np.uint8)
    assert away(x).tolist() != want
    # a row scale one binade too small overflows the range
    e = Q.row_scale_exponent(449.0)
    with pytest.raises(ValueError):
        real_encode(np.array([449.0 / 2.0 ** (e - 1)]))

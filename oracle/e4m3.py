"""Plain CPU oracle of the e4m3 weight format (OCP 8-bit floating point,
E4M3 variant): decoding, per-row power-of-two scaling and round-to-nearest
coding. TEST INFRASTRUCTURE ONLY, like the rest of ``oracle``: only the
tests, the smoke check and the benchmark's CPU-baseline leg may use it.

The paper leaves FP8 execution as an unverified direction (Sec. "Negative
Results and Case Studies", TensorRT FP16 paragraph); the format itself is
the OCP one: a sign bit, 4 exponent bits with bias 7 and 3 significand bits.
Exponent field 0 holds the subnormals m/8 * 2^-6; exponent fields 1..15 the
normals (1 + m/8) * 2^(E-7), except that exponent 15 with significand 7
(codes 0x7F, 0xFF) is NaN, so the largest finite value is 448 (0x7E).

Coding here is a nearest-value search over the table of all finite codes
(ties to the code with an even significand), written independently of any
bit arithmetic. Every value is held exactly in float64.
"""
from __future__ import annotations

import numpy as np


def decode(code: int) -> float:
    """Value of one e4m3 code (NaN codes give nan)."""
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 15 and m == 7:
        return float("nan")
    if e == 0:
        return s * (m / 8.0) * 2.0 ** -6
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


def decode_table() -> np.ndarray:
    """float64 [256]: the value of every code (NaN for 0x7F and 0xFF)."""
    return np.array([decode(c) for c in range(256)], dtype=np.float64)


def _positive_codes():
    """Codes 0x00..0x7E with their values, increasing (0x00 is zero)."""
    codes = np.arange(0x7F, dtype=np.int64)
    vals = np.array([decode(int(c)) for c in codes])
    assert np.all(np.diff(vals) > 0)
    return codes, vals


def encode(x: np.ndarray) -> np.ndarray:
    """e4m3 codes of x (|x| <= 448), nearest value, ties to the even
    significand; a zero result is coded +0 whatever the sign -> uint8."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.isnan(x)) or np.any(np.abs(x) > 448.0):
        raise ValueError("e4m3 coding needs |x| <= 448")
    codes, vals = _positive_codes()
    a = np.abs(x).ravel()
    hi = np.clip(np.searchsorted(vals, a, side="left"), 0, len(vals) - 1)   # first value >= a
    lo = np.clip(hi - 1, 0, len(vals) - 1)
    d_lo = a - vals[lo]
    d_hi = vals[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (codes[hi] % 2 == 0))
    mag = np.where(pick_hi, codes[hi], codes[lo])
    neg = (x.ravel() < 0) & (mag != 0)
    return (mag | np.where(neg, 0x80, 0)).astype(np.uint8).reshape(np.shape(x))


def row_scale_exponent(amax: float) -> int:
    """Smallest integer e with amax <= 448 * 2^e (0 when amax == 0)."""
    if amax == 0.0:
        return 0
    e = int(np.floor(np.log2(amax))) - 10
    while amax > 448.0 * 2.0 ** e:
        e += 1
    return e


def quantize_rows(w: np.ndarray):
    """Per row r: scale 2^e_r (row_scale_exponent of max |w[r]|) and the codes
    of w[r] / 2^e_r (exact division) -> (uint8 [rows, cols], float64 [rows])."""
    w = np.asarray(w, dtype=np.float64)
    amax = np.max(np.abs(w), axis=1)
    scales = np.array([2.0 ** row_scale_exponent(float(a)) for a in amax])
    return encode(w / scales[:, None]), scales


def dequantize_rows(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """decode(codes[r, c]) * scales[r] -> float64."""
    return decode_table()[codes.astype(np.int64)] * np.asarray(scales, dtype=np.float64)[:, None]

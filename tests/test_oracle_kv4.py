"""Pins for the oracle's KV4 quantizer (asymmetric 4-bit group quantization of
the KV cache: Sec. 3.2, and the setup of Sec. 6).

Pins, none of which re-types the oracle's steps:
  * hand-worked groups in tests/golden/kv4_examples.json;
  * an exact rational brute force: every fp32 step of the reading (range,
    range / 15, x - mn, (x - mn) / s) is rounded to the nearest binary32 by
    bisection over Fractions, the scale to the nearest binary16, codes to the
    nearest integer (ties to even); the packed bytes are unpacked by numpy;
  * invariants: the group minimum maps to code 0 and the maximum to 15; the
    reconstruction error is at most half a step (plus the final rounding).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "kv4_examples.json")


def to16(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def f32(x16):
    return np.asarray(x16, np.uint16).view(np.float16).astype(np.float32)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["note"][:40])
def test_kv4_golden(case):
    x = to16([case["x"]])
    codes, params = oracle.kv4_quantize(x, case["G"])
    assert codes[0].tolist() == case["bytes"]
    assert float(f32(params[0, 0, 0])) == case["s"]
    assert float(f32(params[0, 0, 1])) == case["mn"]
    q = np.stack([codes[0] & 15, codes[0] >> 4], axis=1).reshape(-1)
    assert q.tolist() == case["q"]
    xr = oracle.kv4_dequantize(codes, params, case["G"])
    assert f32(xr[0]).tolist() == [np.float32(v) for v in case["xr"]]


def _nearest_binary(r: Fraction, values):
    lo, hi = 0, len(values) - 1
    if r <= values[0]:
        return 0
    if r >= values[hi]:
        return hi
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if values[mid] <= r:
            lo = mid
        else:
            hi = mid
    dl, dh = r - values[lo], values[hi] - r
    if dl != dh:
        return lo if dl < dh else hi
    return lo if lo % 2 == 0 else hi


F16 = [Fraction(float(v)) for v in np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16)
       .view(np.float16).astype(np.float64)]


def fl32(r: Fraction) -> Fraction:
    """Nearest binary32 to r (ties to even significand), by exact comparison of the
    two binary32 neighbours of float(r)."""
    if r == 0:
        return Fraction(0)
    sign = -1 if r < 0 else 1
    a = abs(r)
    c = np.float32(float(a))
    cands = sorted({np.nextafter(c, np.float32(0)), c, np.nextafter(c, np.float32(np.inf))})
    best = None
    for v in cands:
        d = abs(Fraction(float(v)) - a)
        if best is None or d < best[0] or (d == best[0] and int(np.float32(v).view(np.uint32)) % 2 == 0):
            best = (d, v)
    return sign * Fraction(float(best[1]))


def rint_even(r: Fraction) -> int:
    f = r.numerator // r.denominator
    d = r - f
    if d != Fraction(1, 2):
        return f + (1 if d > Fraction(1, 2) else 0)
    return f if f % 2 == 0 else f + 1


def brute_group(xs):
    xs = [Fraction(float(v)) for v in xs]
    mn, mx = min(xs), max(xs)
    rng = fl32(mx - mn)
    s = F16[_nearest_binary(fl32(rng / 15), F16)]
    if s == 0:
        return s, mn, [0] * len(xs)
    q = [min(15, max(0, rint_even(fl32(fl32(x - mn) / s)))) for x in xs]
    return s, mn, q


@pytest.mark.parametrize("seed,T,C,G", [(0, 3, 256, 128), (1, 5, 128, 64), (2, 4, 96, 32),
                                        (3, 2, 64, 16)])
def test_kv4_brute_force(seed, T, C, G):
    X = synth.kv_rows(seed, T, C)
    codes, params = oracle.kv4_quantize(X, G)
    q = np.stack([codes & 15, codes >> 4], axis=2).reshape(T, C)
    xv = f32(X)
    for t in range(T):
        for g in range(C // G):
            s, mn, qb = brute_group(xv[t, g * G:(g + 1) * G])
            assert Fraction(float(f32(params[t, g, 0]))) == s
            assert Fraction(float(f32(params[t, g, 1]))) == mn
            assert q[t, g * G:(g + 1) * G].tolist() == qb


def test_kv4_invariants():
    T, C, G = 64, 1024, 128
    X = synth.kv_rows(11, T, C)
    codes, params = oracle.kv4_quantize(X, G)
    q = np.stack([codes & 15, codes >> 4], axis=2).reshape(T, C, order="C")
    xv = f32(X).reshape(T, C // G, G)
    qg = q.reshape(T, C // G, G)
    amin = xv.argmin(axis=2)
    amax = xv.argmax(axis=2)
    assert np.all(np.take_along_axis(qg, amin[..., None], 2) == 0)
    assert np.all(np.take_along_axis(qg, amax[..., None], 2) == 15)
    s = f32(params[..., 0]).astype(np.float64)
    xr = f32(oracle.kv4_dequantize(codes, params, G)).reshape(T, C // G, G).astype(np.float64)
    err = np.abs(xr - xv)
    ulp16 = np.abs(xr) * 2.0 ** -11 + 2.0 ** -24
    assert np.all(err <= 0.5 * s[..., None] * (1 + 2.0 ** -9) + ulp16)


def test_kv4_zero_minimum_is_positive_zero():
    # min over {+0, -0, 1}: stored as +0 whichever zero comes first
    for row in ([0x8000, 0x0000, 0x3C00, 0x3C00], [0x0000, 0x8000, 0x3C00, 0x3C00],
                [0x8000, 0x8000, 0x8000, 0x8000]):
        _, params = oracle.kv4_quantize(np.array([row], np.uint16), 4)
        assert int(params[0, 0, 1]) == 0x0000
    _, params = oracle.kv4_quantize(np.array([[0x8000, 0x0000, 0x8000, 0x0000]], np.uint16), 4)
    assert params[0, 0].tolist() == [0, 0]


def test_kv4_rejects_bad_arguments():
    X = synth.kv_rows(0, 2, 64)
    with pytest.raises(ValueError):
        oracle.kv4_quantize(X, 48)  # C % G != 0
    bad = X.copy()
    bad[1, 3] = 0x7C00  # +inf
    with pytest.raises(ValueError):
        oracle.kv4_quantize(bad, 32)

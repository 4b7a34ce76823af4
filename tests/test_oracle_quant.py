"""Pins for the oracle's block quantizer (FMPQ, Sec. 3.2 of the paper).

Pins used here, none of which re-types the oracle's own steps:
  * closed forms worked out by hand from the readings (symmetric, fp16 scale
    amax/qmax, nearest-even codes, clamp);
  * an exact rational brute force: the scale is the binary16 value nearest to
    amax/qmax and each code is the integer nearest to x/s (ties to even),
    both decided with Python Fractions from the candidate lists;
  * invariants that any correct symmetric quantizer satisfies.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle

F16_POS = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16)
F16_VAL = [Fraction(float(v)) for v in F16_POS.view(np.float16).astype(np.float64)]


def f16(x):
    return np.asarray(x, dtype=np.float16).astype(np.float32)


def nearest_f16_bits(r: Fraction) -> int:
    """binary16 pattern nearest to r >= 0, ties to even fraction (brute force by bisection)."""
    lo, hi = 0, len(F16_VAL) - 1
    if r >= F16_VAL[hi]:
        return hi
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if F16_VAL[mid] <= r:
            lo = mid
        else:
            hi = mid
    dlo, dhi = r - F16_VAL[lo], F16_VAL[hi] - r
    if dlo < dhi:
        return lo
    if dhi < dlo:
        return hi
    return lo if lo % 2 == 0 else hi


def round_half_even(r: Fraction) -> int:
    f = r.numerator // r.denominator
    d = r - f
    if d > Fraction(1, 2):
        return f + 1
    if d < Fraction(1, 2):
        return f
    return f if f % 2 == 0 else f + 1


def brute_force(v32, bits):
    qmax = 7 if bits == 4 else 127
    xs = [Fraction(float(x)) for x in v32]
    amax = max(abs(x) for x in xs)
    sb = nearest_f16_bits(amax / qmax)
    s = F16_VAL[sb]
    if s == 0:
        return sb, [0] * len(xs)
    return sb, [max(-qmax, min(qmax, round_half_even(x / s))) for x in xs]


def test_closed_form_unit_scale():
    # amax = qmax makes s = 1 exactly (fp16 0x3C00) and every integer keeps its value
    v = np.array([7, -7, 0, 3, -3, 1, -1, 5] * 16, dtype=np.float32)
    s, q = oracle.quantize_group(v, 4)
    assert s == 0x3C00 and np.array_equal(q, v.astype(np.int8))
    v8 = np.arange(-127, 129, 2, dtype=np.float32)[:128]
    v8[0] = 127
    s, q = oracle.quantize_group(v8, 8)
    assert s == 0x3C00 and np.array_equal(q, v8.astype(np.int8))


def test_closed_form_ties_go_to_even():
    v = np.zeros(128, np.float32)
    v[:8] = [7.0, 2.5, -2.5, 3.5, 0.5, -0.5, 1.5, -1.5]
    s, q = oracle.quantize_group(v, 4)
    assert s == 0x3C00
    assert q[:8].tolist() == [7, 2, -2, 4, 0, 0, 2, -2]


def test_closed_form_one_seventh():
    # amax = 1: 1/7 = 1.001001001001001...b * 2^-3; keeping 10 fraction bits and
    # rounding (next bits 01001.. < half) gives (1024 + 146) * 2^-13 -> 0x3092.
    v = np.zeros(128, np.float32)
    v[:4] = [1.0, -0.5, 0.25, -1.0]
    s, q = oracle.quantize_group(v, 4)
    assert s == 0x3092
    # 1/s = 8192/1170: codes are rint(1 * 7.0017) = 7, rint(-3.5009) = -4, rint(1.7504) = 2
    assert q[:4].tolist() == [7, -4, 2, -7]


def test_closed_form_scale_rounding_forces_clamp():
    # amax = 2^-20 (a binary16 subnormal): amax / 7 = 2.2857 * 2^-24 rounds to the
    # subnormal 2 * 2^-24, so x / s = 8 for the largest element, clamped to 7.
    v = np.zeros(128, np.float32)
    v[0] = 2.0 ** -20
    v[1] = -(2.0 ** -21)
    s, q = oracle.quantize_group(v, 4)
    assert s == 0x0002
    assert q[:2].tolist() == [7, -4]


def test_closed_form_tiny_and_zero_blocks():
    s, q = oracle.quantize_group(np.zeros(128, np.float32), 4)
    assert s == 0 and not q.any()
    v = np.zeros(128, np.float32)
    v[5] = 2.0 ** -24  # amax / 7 < 2^-25 rounds to a zero scale: all codes 0
    s, q = oracle.quantize_group(v, 4)
    assert s == 0 and not q.any()


def test_closed_form_outlier_block_8bit():
    # amax = 50: 50/127 = 0.3937007.. = 1.5748031 * 2^-2; 0.5748031 * 1024 = 588.6 -> 589,
    # s = 1613 * 2^-12 = 0.393798828125 -> bits (13 << 10) | 589 = 0x364D; 50 / s = 126.97 -> 127
    v = np.zeros(128, np.float32)
    v[0], v[1] = 50.0, -25.0
    s, q = oracle.quantize_group(v, 8)
    assert s == 0x364D
    assert q[:2].tolist() == [127, round_half_even(Fraction(-25) / Fraction(1613, 4096))]


@pytest.mark.parametrize("bits", [4, 8])
def test_brute_force_random_blocks(bits):
    rng = np.random.default_rng(7 + bits)
    dists = [
        lambda: rng.standard_normal(128),
        lambda: rng.standard_normal(128) * 50,
        lambda: rng.standard_t(2, 128),
        lambda: rng.standard_normal(128) * 1e-6,  # subnormal-sized scales
        lambda: np.round(rng.standard_normal(128) * 4) / 2,  # many exact ties
        lambda: rng.uniform(-65504, 65504, 128),
    ]
    for i in range(120):
        v = f16(dists[i % len(dists)]())
        s, q = oracle.quantize_group(v, bits)
        sb, qb = brute_force(v, bits)
        assert s == sb, (i, s, sb)
        assert q.tolist() == qb, i


@pytest.mark.parametrize("bits", [4, 8])
def test_invariants(bits):
    qmax = 7 if bits == 4 else 127
    rng = np.random.default_rng(11)
    for i in range(200):
        v = f16(rng.standard_normal(128) * (10.0 ** rng.uniform(-4, 3)))
        s16, q = oracle.quantize_group(v, bits)
        s = float(np.array([s16], np.uint16).view(np.float16)[0])
        qi = q.astype(np.int64)
        assert qi.min() >= -qmax and qi.max() <= qmax  # range; -8/-128 never emitted
        if np.abs(v).max() > 0 and s > 0:
            assert np.abs(qi).max() == qmax  # the largest element reaches qmax
        assert np.all((np.sign(qi) == np.sign(v)) | (qi == 0))  # sign kept
        err = np.abs(v.astype(np.float64) - s * qi)
        unclamped = np.abs(v.astype(np.float64)) <= qmax * s
        assert np.all(err[unclamped] <= s / 2 * (1 + 2.0 ** -20))  # nearest level
        # clamping happens only because the fp16 scale rounded below amax / qmax: the
        # excess is at most qmax times half a binary16 ulp at s (2^-25 for subnormals)
        half_ulp = max(s * 2.0 ** -11, 2.0 ** -25)
        assert np.all(err[~unclamped] <= qmax * half_ulp * (1 + 2.0 ** -20))


@pytest.mark.parametrize("bits", [4, 8])
def test_idempotent_on_dequantized_values(bits):
    # s * q is exact in fp32 (11-bit scale times <= 7-bit code): re-quantizing the
    # dequantized block gives back the same scale and codes
    rng = np.random.default_rng(3)
    for _ in range(100):
        v = f16(rng.standard_normal(128) * 3)
        s16, q = oracle.quantize_group(v, bits)
        s = np.float32(np.array([s16], np.uint16).view(np.float16)[0])
        deq = (q.astype(np.float32) * s).astype(np.float32)
        s2, q2 = oracle.quantize_group(deq, bits)
        assert s2 == s16 and np.array_equal(q2, q)


def test_rejects_non_finite():
    v = np.zeros(128, np.float32)
    v[3] = np.inf
    with pytest.raises(ValueError):
        oracle.quantize_group(v, 4)
    v[3] = np.nan
    with pytest.raises(ValueError):
        oracle.quantize_group(v, 8)


def test_quantize_act_layout_closed_form():
    # block (m, g) holds integers in [-qmax, qmax] times 2^j(m, g), with amax = qmax * 2^j,
    # so s = 2^j exactly and the codes are the integers; checks the [K/G][M] scale layout
    M, K, G = 5, 512, 128
    prec = np.array([4, 8, 4, 8], np.uint8)
    rng = np.random.default_rng(5)
    X = np.zeros((M, K), np.float32)
    codes = np.zeros((M, K), np.int64)
    exps = np.zeros((K // G, M), np.int64)
    for m in range(M):
        for g in range(K // G):
            qmax = 7 if prec[g] == 4 else 127
            c = rng.integers(-qmax, qmax + 1, G)
            c[rng.integers(G)] = qmax * (1 if rng.random() < 0.5 else -1)
            j = int(rng.integers(-6, 4))
            X[m, g * G:(g + 1) * G] = c * 2.0 ** j
            codes[m, g * G:(g + 1) * G] = c
            exps[g, m] = j
    X16 = X.astype(np.float16).view(np.uint16)
    qa, sa = oracle.quantize_act(X16, prec, G)
    assert np.array_equal(qa.astype(np.int64), codes)
    want = (2.0 ** exps).astype(np.float16).view(np.uint16)
    assert np.array_equal(sa, want)


def test_quantize_weight_is_4bit_blockwise():
    rng = np.random.default_rng(9)
    W = f16(rng.standard_normal((3, 256)) * 0.02)
    qw, sw = oracle.quantize_weight(W.astype(np.float16).view(np.uint16), 128)
    for n in range(3):
        for g in range(2):
            sb, qb = brute_force(W[n, g * 128:(g + 1) * 128], 4)
            assert sw[g, n] == sb and qw[n, g * 128:(g + 1) * 128].tolist() == qb

"""Pins for the oracle's binary16 conversions.

The oracle converts from the IEEE 754 definition; the pins are numpy's own
float16 conversions (an independent library routine), exhaustively for
fp16 -> fp32 and on a dense structured sweep for fp32 -> fp16.
"""
import numpy as np

import oracle


def test_f16_to_f32_exhaustive():
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.f32_from_f16(h)
    want = h.view(np.float16).astype(np.float32)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), want[~nan].view(np.uint32))


def _check(xf32):
    got = oracle.f16_from_f32(xf32)
    with np.errstate(over="ignore"):  # values past the fp16 range round to infinity
        want = xf32.astype(np.float16).view(np.uint16)
    nan = np.isnan(xf32)
    assert np.all((got[nan] & 0x7C00) == 0x7C00) and np.all((got[nan] & 0x3FF) != 0)
    bad = np.nonzero(got[~nan] != want[~nan])[0]
    assert bad.size == 0, (xf32[~nan][bad[:5]], got[~nan][bad[:5]], want[~nan][bad[:5]])


def test_f32_to_f16_ties_and_neighbours():
    # every finite fp16 value, the midpoints between neighbours (exact ties in fp32)
    # and the fp32 values one ulp either side of each midpoint
    h = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16)
    v = h.view(np.float16).astype(np.float64)
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    assert np.all(mids.astype(np.float64) == (v[:-1] + v[1:]) / 2)  # ties are exact in fp32
    up = np.nextafter(mids, np.float32(np.inf))
    dn = np.nextafter(mids, np.float32(0))
    top = np.array([65504.0, 65519.996, 65520.0, 65520.004, 1e6, np.inf], dtype=np.float32)
    x = np.concatenate([v.astype(np.float32), mids, up, dn, top])
    _check(x)
    _check(-x)


def test_f32_to_f16_strided_sweep():
    # every 97th fp32 bit pattern (44 M values; covers all exponents and NaN/inf)
    bits = np.arange(0, 1 << 32, 97, dtype=np.uint64).astype(np.uint32)
    for part in np.array_split(bits, 8):
        _check(part.view(np.float32))


def test_f32_to_f16_known_values():
    # binary16 encodings stated by the IEEE 754 format itself
    cases = {1.0: 0x3C00, -2.0: 0xC000, 65504.0: 0x7BFF, 2.0 ** -14: 0x0400,
             2.0 ** -24: 0x0001, 2.0 ** -25: 0x0000, 1.5 * 2.0 ** -25: 0x0001,
             0.5: 0x3800, 1.0 / 3.0: 0x3555}
    for x, h in cases.items():
        assert oracle.f16_from_f32(np.array([x], np.float32))[0] == h, x

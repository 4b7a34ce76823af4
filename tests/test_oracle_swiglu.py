"""Pins for the oracle's SwiGLU step (h = SiLU(gate) * up) and the next
layer's quantization of h (FMPQ, Sec. 3.2), which a fused GEMM epilogue
produces instead of the fp16 gate/up output.

Pins, none of which re-types the oracle's steps:
  * exp against Python's fp64 math.exp: within 2 ulps of the rounded true
    value on a dense grid, exact at 0, monotone, clamped outside [-87, 88];
  * SiLU against the fp64 definition x / (1 + e^-x); its limits (0 at 0,
    x for large x, -0 side for large -x);
  * fp16 SwiGLU against fp16(fp64 SiLU(g) * u): equal except within fp32
    rounding of an fp16 tie, and never more than one fp16 ulp apart;
  * the 2G-wide gate/up column grouping, checked by an index computation of
    its own, and the quantization of h against the pinned quantizer.
"""
import math

import numpy as np
import pytest

import oracle
import synth


def ulp32(v):
    return np.spacing(np.abs(np.float32(v))).astype(np.float64)


def test_exp_within_two_ulps():
    xs = np.linspace(-87.0, 88.0, 20001, dtype=np.float32)
    xs = np.concatenate([xs, np.float32([-1e-7, 0.0, 1e-7, 0.5, -0.5, 0.6931472, 1.0])])
    got = oracle.exp_f32(xs).astype(np.float64)
    want = np.array([math.exp(float(x)) for x in xs])
    assert np.all(np.abs(got - want) <= 2 * ulp32(want))
    assert oracle.exp_f32([0.0])[0] == 1.0
    s = np.sort(xs)
    assert np.all(np.diff(oracle.exp_f32(s).astype(np.float64)) >= 0)
    # clamped outside [-87, 88]
    assert oracle.exp_f32([1000.0])[0] == oracle.exp_f32([88.0])[0]
    assert oracle.exp_f32([-1000.0])[0] == oracle.exp_f32([-87.0])[0]


def test_silu_against_definition():
    xs = np.concatenate([np.linspace(-30, 30, 6001), [0.0, 1e-4, -1e-4, 5.5, -5.5]]).astype(np.float32)
    got = oracle.silu_f32(xs).astype(np.float64)
    want = np.array([float(x) / (1.0 + math.exp(-float(x))) for x in xs])
    assert np.all(np.abs(got - want) <= 4 * ulp32(want) + 1e-30)
    assert oracle.silu_f32([0.0])[0] == 0.0
    assert oracle.silu_f32([60000.0])[0] == np.float32(60000.0)
    assert abs(oracle.silu_f32([-60000.0])[0]) < 1e-30


def f16(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def test_swiglu_f16_against_fp64():
    rng = np.random.default_rng(3)
    g = f16(rng.normal(0, 3, 4000))
    u = f16(rng.normal(0, 2, 4000))
    h = oracle.swiglu_f16(g, u).view(np.float16).astype(np.float64)
    gv = g.view(np.float16).astype(np.float64)
    uv = u.view(np.float16).astype(np.float64)
    exact = gv / (1.0 + np.exp(-gv)) * uv
    ref = exact.astype(np.float16).astype(np.float64)
    diff = h != ref
    # where they differ, the exact value sits within fp32 rounding of an fp16 tie
    assert diff.mean() < 0.01
    sp = np.spacing(np.abs(ref.astype(np.float16))).astype(np.float64)
    assert np.all(np.abs(h - ref) <= sp)
    for i in np.flatnonzero(diff):
        mid = (h[i] + ref[i]) / 2
        assert abs(exact[i] - mid) <= 8 * ulp32(exact[i]) + 1e-12


def test_swiglu_f16_every_gate_value():
    """Every finite fp16 gate value with a few up values: the oracle's fp16 h is
    within one fp16 ulp of fp16 of the fp64 SwiGLU, and equal to it except where
    the fp64 value lies within fp32 rounding of an fp16 rounding boundary."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    gv_all = bits.view(np.float16)
    g = bits[np.isfinite(gv_all)]
    gv = g.view(np.float16).astype(np.float64)
    for upv in (1.0, -0.75, 3.0517578125e-05, 1000.0):
        u = np.full(g.shape, np.float16(upv)).view(np.uint16)
        with np.errstate(over="ignore", invalid="ignore"):
            exact = gv / (1.0 + np.exp(-gv)) * np.float64(np.float16(upv))
            ref = exact.astype(np.float16)
        h = oracle.swiglu_f16(g, u).view(np.float16)
        fin = np.isfinite(ref)
        # beyond the fp16 range both overflow to the same infinity
        assert np.array_equal(np.isinf(h[~fin]), np.isinf(ref[~fin]))
        hf, rf, ef = h[fin].astype(np.float64), ref[fin].astype(np.float64), exact[fin]
        with np.errstate(over="ignore"):  # above 65504 the next fp16 value is inf
            sp = np.spacing(np.abs(ref[fin])).astype(np.float64)
        assert np.all(np.abs(hf - rf) <= sp), upv
        diff = np.flatnonzero(hf != rf)
        assert diff.size <= 0.01 * hf.size, (upv, diff.size)
        for i in diff:
            mid = (hf[i] + rf[i]) / 2
            assert abs(ef[i] - mid) <= 8 * ulp32(ef[i]) + 1e-12, (upv, gv[fin][i])


@pytest.mark.parametrize("M,I,G", [(3, 256, 128), (5, 64, 16), (1, 128, 128)])
def test_swiglu_quantize_grouping(M, I, G):
    NG = I // G
    gu = synth.normal_fp16(M + I, 1, (M, 2 * I), 2.0)
    prec = synth.prec_map(NG, max(1, NG // 2), "random", seed=M)
    A, sa = oracle.swiglu_quantize(gu, prec, G)
    # gate column of channel c: (c // G) * 2G + c % G; up: + G
    c = np.arange(I)
    gcol = (c // G) * 2 * G + c % G
    h = np.stack([oracle.swiglu_f16(gu[m, gcol], gu[m, gcol + G]) for m in range(M)])
    qa, sa_ref = oracle.quantize_act(h, prec, G)
    assert np.array_equal(sa, sa_ref)
    assert np.array_equal(A, oracle.pack_act(qa, prec, G))

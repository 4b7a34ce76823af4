"""Host-side calibration map of libcomet (comet_plan_channel_perm, Sec. 3.2)
against the oracle, and argument checks of the permutation, calibration and
KV4 entry points (no device work: every call here fails its checks first).

The plan is integer and index work: perm, map and outlier count must be
identical to the oracle's.
"""
import ctypes
import json
import os

import numpy as np
import pytest

import oracle
import paper_2410_12168_amd as comet
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "plan_channel_perm.json")


def lib_plan(absmax, G, ratio, frac):
    return comet.plan_channel_perm(np.asarray(absmax, np.float32), G, ratio, frac)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["note"][:40])
def test_plan_golden(case):
    perm, prec, nout = lib_plan(case["absmax"], case["G"], case["ratio"], case["max_frac8"])
    assert perm.tolist() == case["perm"]
    assert prec.tolist() == case["prec"]
    assert nout == case["n_outliers"]


CASES = [
    # (K, n_out, ratio, frac, seed)
    (1024, 6, 8.0, 0.2, 0), (8192, 41, 8.0, 0.2, 1), (8192, 300, 8.0, 0.05, 2),
    (28672, 140, 8.0, 0.2, 3), (4096, 0, 8.0, 0.2, 4), (4096, 30, 0.0, 0.25, 5),
    (4096, 30, -1.0, 1.0, 6), (640, 5, 3.0, 1.0, 7),
]


@pytest.mark.parametrize("K,n_out,ratio,frac,seed", CASES)
def test_plan_matches_oracle(K, n_out, ratio, frac, seed):
    ch = synth.outlier_channels(K, n_out, seed=seed)
    a = oracle.channel_absmax(synth.calibration_activations(seed, 16, K, ch))
    want = oracle.plan_channel_perm(a, 128, ratio, frac)
    got = lib_plan(a, 128, ratio, frac)
    assert np.array_equal(got[0], want[0])
    assert np.array_equal(got[1], want[1])
    assert got[2] == want[2]


def test_plan_ties_match_oracle():
    # maxima drawn from a handful of values: long runs of ties at every rank
    rng = np.random.default_rng(5)
    for G in (1, 2, 16, 128):
        a = rng.choice(np.array([0.0, 1.0, 2.0, 50.0], np.float32), size=1024)
        for ratio, frac in ((4.0, 0.5), (0.0, 0.25), (1.0, 1.0)):
            want = oracle.plan_channel_perm(a, G, ratio, frac)
            got = lib_plan(a, G, ratio, frac)
            assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
            assert got[2] == want[2]


def test_plan_rejects_bad_arguments():
    a = np.ones(256, np.float32)
    for args in ((a, 100, 4.0, 0.2), (a, 128, 4.0, 1.5), (a, 128, 4.0, -0.5),
                 (a, 128, float("nan"), 0.2), (np.array([1.0, -2.0], np.float32), 1, 4.0, 0.5),
                 (np.array([1.0, np.inf], np.float32), 1, 4.0, 0.5)):
        with pytest.raises(comet.CometError) as e:
            lib_plan(*args)
        assert e.value.status == 1


FAKE = 1 << 20  # never dereferenced: every call below fails its argument checks


def p(x):
    return ctypes.c_void_p(x)


def test_device_entry_points_check_arguments():
    L = comet.lib()
    m = np.full(2, 4, np.uint8)
    mp = p(m.ctypes.data)
    # perm must be 16-byte aligned (NULL is allowed)
    assert L.comet_fmpq_quantize_act_perm(p(FAKE), p(FAKE + 4), mp, p(FAKE), p(FAKE), 4, 256, 128,
                                          None) == 1
    assert L.comet_pack_w4_perm(p(FAKE), p(FAKE + 8), p(FAKE), p(FAKE), 16, 256, 128, None) == 1
    assert L.comet_pack_w4_perm(p(FAKE), p(FAKE), p(FAKE), p(FAKE), 16, 256, 96, None) == 2
    # channel_absmax: K a positive multiple of 8, aligned pointers
    assert L.comet_channel_absmax(p(FAKE), p(FAKE), 4, 12, None) == 1
    assert L.comet_channel_absmax(p(FAKE), p(FAKE), 0, 16, None) == 1
    assert L.comet_channel_absmax(p(FAKE + 2), p(FAKE), 4, 16, None) == 1
    assert L.comet_channel_absmax(None, p(FAKE), 4, 16, None) == 1
    # KV4: G in {32, 64, 128}, C % G == 0, alignment
    assert L.comet_kv4_quantize(p(FAKE), p(FAKE), p(FAKE), 4, 256, 48, None) == 2
    assert L.comet_kv4_quantize(p(FAKE), p(FAKE), p(FAKE), 4, 96, 64, None) == 1
    assert L.comet_kv4_quantize(p(FAKE), p(FAKE), p(FAKE), 0, 128, 128, None) == 1
    assert L.comet_kv4_quantize(p(FAKE + 8), p(FAKE), p(FAKE), 4, 128, 128, None) == 1
    assert L.comet_kv4_quantize(p(FAKE), p(FAKE + 2), p(FAKE), 4, 128, 128, None) == 1
    assert L.comet_kv4_dequantize(p(FAKE), p(FAKE), p(FAKE), 4, 256, 256, None) == 2
    assert L.comet_kv4_dequantize(p(FAKE), p(FAKE), None, 4, 256, 128, None) == 1
    # SwiGLU entry points: N a multiple of 256, I of 128, aligned outputs
    W = p(FAKE)
    assert L.comet_w4ax_gemm_swiglu_quant(W, mp, W, W, W, 16, 384, 256, 128, mp, W, W, None) == 1
    assert L.comet_w4ax_gemm_swiglu_quant(W, mp, W, W, W, 16, 512, 256, 128, mp, p(FAKE + 4), W,
                                          None) == 1
    assert L.comet_w4ax_gemm_swiglu_quant(W, mp, W, W, W, 16, 512, 256, 128, mp, None, W,
                                          None) == 1
    assert L.comet_swiglu_quantize(W, mp, W, W, 4, 200, 128, None) == 1
    assert L.comet_swiglu_quantize(W, mp, W, W, 4, 256, 64, None) == 2
    assert L.comet_swiglu_quantize(W, mp, W, W, 0, 256, 128, None) == 1
    # the activation quantizer's row limit
    assert L.comet_fmpq_quantize_act_perm(p(FAKE), None, mp, p(FAKE), p(FAKE), 65535 * 32 + 1, 256,
                                          128, None) == 2
    assert comet.comet_last_error() != ""

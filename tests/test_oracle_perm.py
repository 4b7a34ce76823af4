"""Pins for the oracle's channel permutation and calibration map (Sec. 3.2).

The paper finds outlier channels by sampling activations, gathers them into a
few blocks with a channel permutation (the weight columns take the same
permutation, so the product is unchanged) and quantizes only those blocks to
8 bits.  Pins, none of which re-types the oracle's steps:
  * hand-worked cases in tests/golden/plan_channel_perm.json;
  * invariants any plan under the reading must satisfy (a permutation; the
    8-bit blocks hold exactly the largest maxima; every other channel stays
    put unless it moved up, and the displaced channels fill the gaps;
    the 8-bit share stays under the cap; every outlier is covered when the cap
    allows);
  * numpy brute force for the per-channel maxima and the column gather;
  * the defining property of the permutation: X W^T is unchanged (fp64);
  * the reason for it: on activations with scattered outlier channels the
    permuted mixed-precision result is far closer to X W^T than 4-bit
    quantization of the unpermuted activations, using one 8-bit block.
"""
import json
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "plan_channel_perm.json")


def f32(x16):
    return np.asarray(x16, np.uint16).view(np.float16).astype(np.float32)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["note"][:40])
def test_plan_golden(case):
    perm, prec, nout = oracle.plan_channel_perm(np.array(case["absmax"], np.float32), case["G"],
                                                case["ratio"], case["max_frac8"])
    assert perm.tolist() == case["perm"]
    assert prec.tolist() == case["prec"]
    assert nout == case["n_outliers"]


def check_plan(absmax, G, ratio, frac, perm, prec, nout):
    K = absmax.size
    NG = K // G
    assert sorted(perm.tolist()) == list(range(K))
    n8 = int((prec == 8).sum())
    assert prec.tolist() == [8] * n8 + [4] * (NG - n8)
    assert n8 <= int(np.floor(np.float64(frac) * NG))
    head = perm[: n8 * G]
    # the 8-bit blocks hold the n8*G largest maxima, in descending order
    assert np.array_equal(np.sort(absmax[head]), np.sort(absmax)[K - n8 * G:])
    assert np.all(np.diff(absmax[head].astype(np.float64)) <= 0)
    # later positions keep their channel unless it moved up; the vacated
    # positions take the displaced channels, ascending to ascending
    moved = np.zeros(K, bool)
    moved[head] = True
    pos = np.arange(n8 * G, K)
    keep = ~moved[pos]
    assert np.array_equal(perm[pos[keep]], pos[keep])
    displaced = np.array([c for c in range(n8 * G) if not moved[c]], dtype=np.int64)
    assert np.array_equal(perm[pos[~keep]], displaced)
    med = np.sort(absmax)[(K - 1) // 2]
    out = np.flatnonzero(absmax.astype(np.float64) > np.float64(ratio) * np.float64(med))
    if ratio > 0:
        assert nout == out.size
        if -(-out.size // G) <= int(np.floor(np.float64(frac) * NG)):
            assert set(out.tolist()) <= set(head.tolist())
            assert n8 == -(-out.size // G)


@pytest.mark.parametrize("K,n_out,ratio,frac", [(1024, 6, 8.0, 0.2), (4096, 40, 8.0, 0.2),
                                                (8192, 41, 8.0, 0.05), (8192, 300, 8.0, 0.05),
                                                (2048, 0, 8.0, 0.2), (2048, 10, 0.0, 0.25)])
def test_plan_invariants(K, n_out, ratio, frac):
    G = 128
    ch = synth.outlier_channels(K, n_out, seed=K + n_out)
    X = synth.calibration_activations(3, 64, K, ch)
    a = oracle.channel_absmax(X)
    perm, prec, nout = oracle.plan_channel_perm(a, G, ratio, frac)
    check_plan(a, G, ratio, frac, perm, prec, nout)
    if ratio > 0:
        assert nout >= n_out  # every planted channel is above 8 x median at 50x scale


def test_plan_edge_cases():
    a = np.arange(256, dtype=np.float32)
    perm, prec, _ = oracle.plan_channel_perm(a, 128, 4.0, 0.0)
    assert perm.tolist() == list(range(256)) and prec.tolist() == [4, 4]
    z = np.zeros(256, np.float32)
    perm, prec, nout = oracle.plan_channel_perm(z, 128, 10.0, 1.0)
    assert perm.tolist() == list(range(256)) and prec.tolist() == [4, 4] and nout == 0
    for bad in (dict(max_frac8=1.5), dict(max_frac8=-0.1), dict(max_frac8=float("nan"))):
        with pytest.raises(ValueError):
            oracle.plan_channel_perm(a, 128, 4.0, bad["max_frac8"])
    with pytest.raises(ValueError):
        oracle.plan_channel_perm(np.array([1.0, -1.0], np.float32), 2, 4.0, 0.5)
    with pytest.raises(ValueError):
        oracle.plan_channel_perm(np.array([1.0, np.inf], np.float32), 2, 4.0, 0.5)
    with pytest.raises(ValueError):
        oracle.plan_channel_perm(a, 100, 4.0, 0.5)  # K % G != 0


def test_channel_absmax_brute_force():
    X = synth.calibration_activations(1, 37, 384, [5, 200])
    want = np.abs(f32(X)).max(axis=0)
    assert np.array_equal(oracle.channel_absmax(X), want)
    # accumulating over two batches equals one pass over both
    Y = synth.calibration_activations(2, 11, 384, [7])
    acc = oracle.channel_absmax(Y, oracle.channel_absmax(X))
    assert np.array_equal(acc, np.abs(f32(np.concatenate([X, Y]))).max(axis=0))
    # -0.0 counts as 0
    neg0 = np.full((1, 8), 0x8000, np.uint16)
    assert np.array_equal(oracle.channel_absmax(neg0), np.zeros(8, np.float32))


def test_permute_columns_brute_force():
    X = synth.normal_fp16(4, 1, (9, 256))
    rng = np.random.default_rng(0)
    perm = rng.permutation(256).astype(np.int32)
    assert np.array_equal(oracle.permute_columns(X, perm), X[:, perm])
    with pytest.raises(ValueError):
        oracle.permute_columns(X, np.full(256, 256, np.int32))


def test_permutation_leaves_product_unchanged():
    K = 512
    ch = synth.outlier_channels(K, 5, seed=1)
    X = synth.calibration_activations(1, 8, K, ch)
    W = synth.weights(2, 16, K)
    perm, _, _ = oracle.plan_channel_perm(oracle.channel_absmax(X), 128, 8.0, 0.25)
    a = oracle.exact_gemm(X, W)
    b = oracle.exact_gemm(oracle.permute_columns(X, perm), oracle.permute_columns(W, perm))
    np.testing.assert_allclose(b, a, rtol=1e-12, atol=1e-12)


def activation_error(X, W, prec, perm=None):
    """Mean |quantized result - X (dequantized 4-bit W)^T|: the error that the
    activation quantization adds on top of the 4-bit weights."""
    if perm is not None:
        X = oracle.permute_columns(X, perm)
        W = oracle.permute_columns(W, perm)
    qa, sa = oracle.quantize_act(X, prec)
    qw, sw = oracle.quantize_weight(W)
    wd = qw.astype(np.float64) * np.repeat(f32(sw).astype(np.float64).T, 128, axis=1)
    ref = f32(X).astype(np.float64) @ wd.T
    return np.abs(oracle.dequant_gemm(qa, sa, qw, sw) - ref).mean()


def test_permutation_reduces_error_with_one_8bit_block():
    K, M, N = 1024, 64, 64
    ch = synth.outlier_channels(K, 6, seed=9)
    assert len({c // 128 for c in ch}) >= 4  # scattered over several blocks
    calib = synth.calibration_activations(5, 128, K, ch)
    perm, prec, nout = oracle.plan_channel_perm(oracle.channel_absmax(calib), 128, 8.0, 0.2)
    assert nout == 6 and prec.tolist() == [8] + [4] * 7
    X = synth.calibration_activations(6, M, K, ch, tid=synth.TID_X)
    W = synth.weights(7, N, K)
    e_perm = activation_error(X, W, prec, perm)
    e_all4 = activation_error(X, W, np.full(8, 4, np.uint8))
    # without the permutation the same 8-bit budget (one block) covers at most one outlier block
    e_same_budget = activation_error(X, W, np.array([8] + [4] * 7, np.uint8))
    # 8-bit on every block that holds an outlier, without the permutation
    blocks = sorted({int(c) // 128 for c in ch})
    cover = np.full(8, 4, np.uint8)
    cover[blocks] = 8
    e_cover = activation_error(X, W, cover)
    assert e_perm < 0.25 * e_all4
    assert e_perm < 0.25 * e_same_budget
    assert e_perm < 2.0 * e_cover

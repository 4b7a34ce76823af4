"""Pins for the oracle's W4Ax contraction (Sec. 4.1 and Sec. 5: O = WX over
blocks of 128 channels, integer products, per-block dequantization).

Pins: brute force with numpy int64 products on tiny shapes; the all-4-bit and
all-8-bit limiting cases against a textbook integer matmul; metamorphic
relations (block permutation, power-of-two token scaling); the
dequantize-first identity; and the closed-form quantization error bound
against the unquantized fp64 product.
"""
import numpy as np
import pytest

import oracle
import synth


def f16bits(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def f16val(h):
    return np.asarray(h, np.uint16).view(np.float16).astype(np.float64)


def make(M, N, K, prec, seed):
    X16 = synth.activations(seed, M, K, prec)
    W16 = synth.weights(seed, N, K)
    qa, sa = oracle.quantize_act(X16, prec)
    qw, sw = oracle.quantize_weight(W16)
    return X16, W16, qa, sa, qw, sw


@pytest.mark.parametrize("M,N,K", [(1, 1, 128), (2, 3, 256), (5, 2, 384), (3, 5, 128)])
def test_group_acc_brute_force(M, N, K):
    rng = np.random.default_rng(M * 100 + N * 10 + K)
    prec = rng.choice(np.array([4, 8], np.uint8), K // 128)
    _, _, qa, sa, qw, sw = make(M, N, K, prec, seed=int(rng.integers(1000)))
    acc = oracle.group_acc(qa, qw)
    a = qa.astype(np.int64).reshape(M, K // 128, 128)
    w = qw.astype(np.int64).reshape(N, K // 128, 128)
    want = np.einsum("mgc,ngc->mng", a, w)
    assert np.array_equal(acc.astype(np.int64), want)
    # worst-case magnitudes fit int32 with room: 128 * 127 * 7 for 8-bit blocks
    assert np.abs(acc).max() <= 128 * 127 * 7


@pytest.mark.parametrize("bits", [4, 8])
def test_limiting_case_uniform_precision(bits):
    M, N, K = 4, 6, 512
    prec = np.full(K // 128, bits, np.uint8)
    _, _, qa, sa, qw, sw = make(M, N, K, prec, seed=bits)
    qmax = 7 if bits == 4 else 127
    assert np.abs(qa.astype(int)).max() == qmax
    acc = oracle.group_acc(qa, qw)
    for g in range(K // 128):
        a = qa[:, g * 128:(g + 1) * 128].astype(np.int64)
        w = qw[:, g * 128:(g + 1) * 128].astype(np.int64)
        assert np.array_equal(acc[:, :, g].astype(np.int64), np.matmul(a, w.T))
    # the dequantized product is the plain scaled int GEMM summed over blocks
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    want = sum(np.matmul(qa[:, g * 128:(g + 1) * 128].astype(np.float64) * f16val(sa[g])[:, None],
                         (qw[:, g * 128:(g + 1) * 128].astype(np.float64) * f16val(sw[g])[:, None]).T)
               for g in range(K // 128))
    assert np.allclose(ref, want, rtol=1e-12, atol=0)


def test_block_permutation_is_equivariant():
    M, N, K = 3, 4, 512
    prec = np.array([4, 8, 4, 4], np.uint8)
    X16, W16, qa, sa, qw, sw = make(M, N, K, prec, seed=3)
    perm = np.array([2, 0, 3, 1])
    cols = np.concatenate([np.arange(g * 128, (g + 1) * 128) for g in perm])
    qa2, sa2 = oracle.quantize_act(X16[:, cols], prec[perm])
    qw2, sw2 = oracle.quantize_weight(W16[:, cols])
    acc = oracle.group_acc(qa, qw)
    acc2 = oracle.group_acc(qa2, qw2)
    assert np.array_equal(acc2, acc[:, :, perm])
    assert np.array_equal(sa2, sa[perm]) and np.array_equal(sw2, sw[perm])
    r1 = oracle.dequant_gemm(qa, sa, qw, sw)
    r2 = oracle.dequant_gemm(qa2, sa2, qw2, sw2)
    assert np.allclose(r1, r2, rtol=1e-13, atol=1e-15)


def test_power_of_two_token_scaling():
    M, N, K = 4, 3, 256
    prec = np.array([8, 4], np.uint8)
    X16, W16, qa, sa, qw, sw = make(M, N, K, prec, seed=5)
    X = f16val(X16)
    for j in (-3, 2):
        Xs = X.copy()
        Xs[1] *= 2.0 ** j
        qa2, sa2 = oracle.quantize_act(f16bits(Xs), prec)
        assert np.array_equal(qa2, qa)
        assert np.array_equal(f16val(sa2[:, 1]), f16val(sa[:, 1]) * 2.0 ** j)
        assert np.array_equal(sa2[:, [0, 2, 3]], sa[:, [0, 2, 3]])


def test_dequantize_first_identity_and_rows():
    M, N, K = 6, 5, 640
    prec = synth.prec_map(5, 2, "random", seed=9)
    X16, W16, qa, sa, qw, sw = make(M, N, K, prec, seed=9)
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    # dequantize each element first, then one fp64 dot product over all K
    sa_k = np.repeat(f16val(sa), 128, axis=0).T  # [M][K]
    sw_k = np.repeat(f16val(sw), 128, axis=0).T  # [N][K]
    deq = (qa * sa_k) @ (qw * sw_k).T
    assert np.allclose(ref, deq, rtol=1e-12, atol=1e-14 * np.abs(deq).max())
    rows = np.array([4, 0, 5])
    assert np.array_equal(oracle.dequant_gemm(qa, sa, qw, sw, rows=rows), ref[rows])


def test_quantization_error_bound_against_exact():
    M, N, K = 4, 8, 1024
    prec = synth.prec_map(8, 1)
    X16, W16, qa, sa, qw, sw = make(M, N, K, prec, seed=0)
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    exact = oracle.exact_gemm(X16, W16)
    X = f16val(X16)
    W = f16val(W16)
    ex = np.abs(X - qa * np.repeat(f16val(sa), 128, axis=0).T)
    ew = np.abs(W - qw * np.repeat(f16val(sw), 128, axis=0).T)
    bound = np.abs(X) @ ew.T + ex @ np.abs(W).T + ex @ ew.T
    assert np.all(np.abs(ref - exact) <= bound * (1 + 1e-9) + 1e-12)
    # and the error is a quantization error, not a broken contraction
    rel = np.linalg.norm(ref - exact) / np.linalg.norm(exact)
    assert 1e-3 < rel < 0.5

"""GPU parity sweep: seeded random shapes across every kernel regime.

Each case quantizes, packs and multiplies through the C ABI and checks the
per-block int32 sums of a window bit-exactly and the whole fp16 output
against the oracle's tolerance.  The shapes are drawn once from a fixed
seed, spread over the few-token (M <= 8), shared-activation (8 < M <= 32),
three-row-block few-token (32 < M <= 48), 128-row (48 < M <= 128) and
256-row tile (M > 128, up to several row tiles) kernels, with ragged M, N
and K, small column counts that make the tile kernels split every tile over
many workgroups, and all the precision-map kinds.  The oracle's cost bounds the sizes.
"""
import numpy as np
import pytest

import oracle
from parity import assert_out_close
from test_gpu_parity import host, host_u16, make_map, run_path

pytestmark = pytest.mark.gpu

REGIMES = [(1, 8), (9, 32), (33, 48), (49, 128), (129, 400), (401, 1100), (1101, 2100)]
KINDS = ["cfg0", "all4", "all8", "alternate", "random"]


def sweep_shapes(n_per_regime=6, seed=20241016, budget=2.5e8):
    rng = np.random.default_rng(seed)
    shapes = []
    for lo, hi in REGIMES:
        for _ in range(n_per_regime):
            while True:
                M = int(rng.integers(lo, hi + 1))
                N = 16 * int(rng.integers(1, 129))        # 16 .. 2048
                K = 128 * int(rng.integers(1, 33))        # 128 .. 4096
                if M * N * K <= budget:
                    break
            shapes.append((M, N, K, KINDS[len(shapes) % len(KINDS)]))
    return shapes


SHAPES = sweep_shapes()


@pytest.mark.parametrize("M,N,K,kind", SHAPES)
def test_sweep_matches_oracle(M, N, K, kind):
    prec = make_map(kind, K // 128, seed=M * 7 + N)
    win = (max(0, M - 20), M, 0, min(N, 48))
    r = run_path(M, N, K, prec, seed=M + 3 * N + K, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa[win[0]:win[1]], qw[win[2]:win[3]]))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"sweep {M}x{N}x{K}/{kind}")


@pytest.mark.parametrize("M", [1, 20, 100, 300])
def test_largest_k(M):
    # K = 65536 (512 blocks, the most the block map holds) in every kernel
    # regime: the K-block order table of the tile and mid-size kernels is full
    N, K = 64, 65536
    prec = make_map("random", K // 128, seed=M)
    win = (max(0, M - 8), M, N - 16, N)
    r = run_path(M, N, K, prec, seed=7 * M + 1, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa[win[0]:win[1]], qw[win[2]:win[3]]))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"largest K, M={M}")

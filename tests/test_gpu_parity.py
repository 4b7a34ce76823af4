"""GPU parity: libcomet (through its C ABI) against the CPU oracle.

Packed bytes, scales and the per-block int32 sums must be bit-identical; the
fp16 GEMM output must meet the elementwise tolerance of tests/parity.py.
Inputs are the seeded synthetic workloads of synth/.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_12168_amd as comet
import synth
from parity import act_rows, assert_out_close

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def dev_u16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.float16)


def host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy()


def host_u16(t: torch.Tensor) -> np.ndarray:
    return host(t.view(torch.int16)).view(np.uint16)


def run_path(M, N, K, prec, seed, diag_window=None):
    X16 = synth.activations(seed, M, K, prec)
    W16 = synth.weights(seed, N, K)
    X = dev_u16(X16)
    W = dev_u16(W16)
    A, sa = comet.quantize_act(X, prec)
    Wp, sw = comet.pack_w4(W)
    out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
    res = {"X16": X16, "W16": W16, "A": A, "sa": sa, "Wp": Wp, "sw": sw, "out": out}
    if diag_window is not None:
        res["acc"] = comet.w4ax_gemm_acc(A, prec, sa, Wp, sw, M, N, K, *diag_window)
    return res


SHAPES = [
    # (M, N, K, map kind) -- several tiles, ragged tails, both precisions
    (16, 1024, 1024, "cfg0"),
    (1, 16, 128, "all4"),
    (3, 48, 256, "all8"),
    (100, 272, 1152, "random"),
    (257, 400, 640, "alternate"),
    (130, 144, 384, "cfg0"),
    # 128-row tiles (64 < M <= 128): ragged rows and columns, both precisions
    (65, 528, 640, "alternate"),
    (128, 784, 1024, "all8"),
    (97, 4096, 2048, "random"),
]


def make_map(kind, NG, seed):
    if kind == "all4":
        return np.full(NG, 4, np.uint8)
    if kind == "all8":
        return np.full(NG, 8, np.uint8)
    if kind == "alternate":
        return np.array([4, 8] * NG, np.uint8)[:NG]
    if kind == "random":
        return synth.prec_map(NG, max(1, NG // 3), "random", seed)
    return synth.prec_map(NG, max(1, NG // 8))


@pytest.mark.parametrize("M,N,K,kind", SHAPES)
def test_quantize_and_pack_bit_exact(M, N, K, kind):
    prec = make_map(kind, K // 128, seed=M)
    r = run_path(M, N, K, prec, seed=M + N)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    assert np.array_equal(host_u16(r["sa"]), sa)
    assert np.array_equal(host(r["A"]), oracle.pack_act(qa, prec))
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host_u16(r["sw"]), sw)
    assert np.array_equal(host(r["Wp"]), oracle.pack_weight(qw))


@pytest.mark.parametrize("M,N,K,kind", SHAPES)
def test_gemm_matches_oracle(M, N, K, kind):
    prec = make_map(kind, K // 128, seed=M)
    win = (0, min(M, 37), max(0, N - 40), N)
    r = run_path(M, N, K, prec, seed=M + N, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    acc = oracle.group_acc(qa[win[0]:win[1]], qw[win[2]:win[3]])
    assert np.array_equal(host(r["acc"]), acc)
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"{M}x{N}x{K}/{kind}")


def test_gemm_run_twice_bit_identical():
    M, N, K = 130, 400, 1024
    prec = synth.prec_map(K // 128, 2, "random", 4)
    r = run_path(M, N, K, prec, seed=11)
    again = comet.w4ax_gemm(r["A"], prec, r["sa"], r["Wp"], r["sw"], M, N, K)
    assert torch.equal(r["out"].view(torch.int16), again.view(torch.int16))


def test_nondefault_stream():
    M, N, K = 64, 256, 512
    prec = synth.prec_map(4, 1)
    X16 = synth.activations(2, M, K, prec)
    W16 = synth.weights(2, N, K)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        X = dev_u16(X16)
        W = dev_u16(W16)
        A, sa = comet.quantize_act(X, prec)
        Wp, sw = comet.pack_w4(W)
        out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
    s.synchronize()
    qa, osa = oracle.quantize_act(X16, prec)
    qw, osw = oracle.quantize_weight(W16)
    assert_out_close(host_u16(out).view(np.float16), oracle.dequant_gemm(qa, osa, qw, osw))


def test_edge_values_quantize():
    # zero rows, tiny (subnormal-scale) rows, exact ties and +-65504
    M, K = 6, 256
    prec = np.array([4, 8], np.uint8)
    X = np.zeros((M, K), np.float32)
    X[1, :] = 2.0 ** -24
    X[2, :8] = [7.0, 2.5, -2.5, 3.5, 0.5, -0.5, 1.5, -1.5]
    X[3, :] = 65504.0 * np.cos(np.arange(K))
    X[4, ::3] = -(2.0 ** -20)
    X[5, 128:] = 127.0 * np.sin(np.arange(128))
    X16 = X.astype(np.float16).view(np.uint16)
    A, sa = comet.quantize_act(dev_u16(X16), prec)
    qa, osa = oracle.quantize_act(X16, prec)
    assert np.array_equal(host_u16(sa), osa)
    assert np.array_equal(host(A), oracle.pack_act(qa, prec))


@pytest.mark.parametrize("layer", ["qkv", "gate_up", "down"])
def test_llama3_70b_full_size_sampled_rows(layer):
    # full LLaMA-3-70B prefill shape (M = 4096); the oracle recomputes a seeded
    # sample of rows (quantization is per row), the weights in full
    K, N = synth.LLAMA3_70B[layer]
    M = 4096
    NG = K // 128
    prec = synth.prec_map(NG, NG // 16)
    r = run_path(M, N, K, prec, seed=0)
    rows = np.array([0, 1, 777, 2048, 4095])
    qa, sa = oracle.quantize_act(r["X16"][rows], prec)
    assert np.array_equal(act_rows(host(r["A"]), prec, M, rows), oracle.pack_act(qa, prec))
    assert np.array_equal(host_u16(r["sa"])[:, rows], sa)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host_u16(r["sw"]), sw)
    assert np.array_equal(host(r["Wp"]), oracle.pack_weight(qw))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    out = host_u16(r["out"]).view(np.float16)[rows]
    assert_out_close(out, ref, f"70B {layer}")


SKINNY = [
    # few-token shapes (weight-streaming kernel): ragged M, split-K, both precisions
    (1, 64, 256, "cfg0"),
    (5, 160, 1024, "random"),
    (16, 512, 512, "all8"),
    (33, 96, 1152, "alternate"),
    (64, 2048, 4096, "cfg0"),
    # four split-K slots per column block; shorter chunks for larger M
    (8, 512, 2048, "random"),
    (16, 256, 4096, "cfg0"),
    (40, 128, 2048, "all8"),
    # 8 < M <= 32 (activation operand shared through LDS): ragged M; column
    # blocks that leave the last workgroup partly idle; K-blocks that split
    # unevenly over two slots (9 blocks: 4 + 5, so one slot runs dead steps)
    (9, 80, 1152, "random"),
    (17, 208, 2048, "alternate"),
    (24, 1040, 4096, "cfg0"),
    (31, 336, 1536, "all8"),
    # two split-K slots (N = 8192) with uneven halves: 4 + 5 and 8 + 9 blocks
    (20, 8192, 1152, "random"),
    (12, 8192, 2176, "alternate"),
]


@pytest.mark.parametrize("M,N,K,kind", SKINNY)
def test_skinny_gemm_matches_oracle(M, N, K, kind):
    prec = make_map(kind, K // 128, seed=M + 1)
    win = (0, M, max(0, N - 48), N)
    r = run_path(M, N, K, prec, seed=3 * M + N, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa, qw[win[2]:win[3]]))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"{M}x{N}x{K}/{kind}")
    again = comet.w4ax_gemm(r["A"], prec, r["sa"], r["Wp"], r["sw"], M, N, K)
    assert torch.equal(r["out"].view(torch.int16), again.view(torch.int16))


@pytest.mark.parametrize("M", [1, 8, 32])
def test_llama3_70b_decode_full_size(M):
    # LLaMA-3-70B gate_up at decode sizes: every output row checked
    K, N = synth.LLAMA3_70B["gate_up"]
    prec = synth.prec_map(K // 128, K // 128 // 16)
    r = run_path(M, N, K, prec, seed=M)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"decode M={M}")


@pytest.mark.parametrize("layer,M", [("qkv", 1), ("qkv", 8), ("o", 1), ("o", 8), ("down", 1),
                                     ("down", 8)])
def test_llama3_70b_decode_other_layers_full_size(layer, M):
    # the other LLaMA-3-70B layers at decode sizes (per-wave few-token kernel
    # for qkv's 640 panels, the stream kernel for o and down with two panels
    # per CU): every output row checked
    K, N = synth.LLAMA3_70B[layer]
    prec = synth.prec_map(K // 128, K // 128 // 16)
    r = run_path(M, N, K, prec, seed=M + 7)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"decode {layer} M={M}")


@pytest.mark.parametrize("M", [40, 96, 128])
def test_llama3_70b_decode_128_row_tiles_sampled_rows(M):
    # LLaMA-3-70B gate_up with 128-row tiles (at M = 40 too: its 224 column
    # tiles are wide enough to take it from the few-token kernel); a sample of
    # rows on both halves of the tile checked against the oracle
    K, N = synth.LLAMA3_70B["gate_up"]
    prec = synth.prec_map(K // 128, K // 128 // 16)
    r = run_path(M, N, K, prec, seed=M)
    rows = np.unique(np.clip([0, 1, 63, 64, M - 1], 0, M - 1))
    qa, sa = oracle.quantize_act(r["X16"][rows], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16)[rows], ref, f"decode M={M}")


def test_wrappers_reject_strided_and_mistyped_tensors():
    X = torch.zeros((256, 128), dtype=torch.float16, device=DEV)
    with pytest.raises(ValueError, match="strided"):
        comet.quantize_act(X.t(), [4, 8])
    with pytest.raises(ValueError, match="float32"):
        comet.pack_w4(X.float())
    A, sa = comet.quantize_act(X[:, :128].contiguous(), [4])
    Wp, sw = comet.pack_w4(X[:16].contiguous())
    with pytest.raises(ValueError, match="a_scales"):
        comet.w4ax_gemm(A, [4], sa.view(torch.int16), Wp, sw, 256, 16, 128)

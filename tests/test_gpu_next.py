"""GPU parity of the calibration step, the channel permutation and the KV4
quantizer (Sec. 3.2; Sec. 6 setup) against the CPU oracle, through the C ABI.

All of it is integer, byte or exactly-defined fp work: maxima, packed codes,
scales, permutations and KV4 codes/params/reconstructions must be
bit-identical.  The end-to-end permuted GEMM meets the tolerance of
tests/parity.py against the oracle on the permuted operands.
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


def dev_u16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.float16)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def host_u16(t):
    return host(t.view(torch.int16)).view(np.uint16)


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


# --- per-channel maxima ---------------------------------------------------------

@pytest.mark.parametrize("M,K", [(1, 8), (37, 384), (1000, 1032), (33, 4104), (4096, 8192)])
def test_channel_absmax_bit_exact(M, K):
    print(f"channel_absmax M={M} K={K}", flush=True)
    ch = synth.outlier_channels(K, max(1, K // 200), seed=M)
    X16 = synth.calibration_activations(M, M, K, ch)
    got = host(comet.channel_absmax(dev_u16(X16)))
    assert np.array_equal(got.view(np.uint32), oracle.channel_absmax(X16).view(np.uint32))


def test_channel_absmax_accumulates():
    K = 2048
    X1 = synth.calibration_activations(1, 300, K, [3, 900])
    X2 = synth.calibration_activations(2, 77, K, [1500])
    a = comet.channel_absmax(dev_u16(X1))
    comet.channel_absmax(dev_u16(X2), a)
    want = oracle.channel_absmax(X2, oracle.channel_absmax(X1))
    assert np.array_equal(host(a), want)


# --- permuted quantization and packing -----------------------------------------

def random_perm(K, seed):
    return np.random.default_rng(seed).permutation(K).astype(np.int32)


PERM_SHAPES = [(1, 128, "random"), (16, 1024, "planned"), (100, 1152, "random"),
               (257, 640, "planned"), (3, 256, "identity")]


def perm_for(kind, X16, K, seed):
    if kind == "identity":
        return np.arange(K, dtype=np.int32), np.full(K // 128, 4, np.uint8)
    if kind == "random":
        return random_perm(K, seed), synth.prec_map(K // 128, max(1, K // 384), "random", seed)
    perm, prec, _ = oracle.plan_channel_perm(oracle.channel_absmax(X16), 128, 8.0, 0.25)
    return perm, prec


@pytest.mark.parametrize("M,K,kind", PERM_SHAPES)
def test_quantize_act_perm_bit_exact(M, K, kind):
    print(f"quantize_act_perm M={M} K={K} {kind}", flush=True)
    ch = synth.outlier_channels(K, 3, seed=K)
    X16 = synth.calibration_activations(M + 1, M, K, ch)
    perm, prec = perm_for(kind, X16, K, M)
    A, sa = comet.quantize_act(dev_u16(X16), prec, perm=dev_i32(perm))
    qa, sa_ref = oracle.quantize_act(oracle.permute_columns(X16, perm), prec)
    assert np.array_equal(host_u16(sa), sa_ref)
    assert np.array_equal(host(A), oracle.pack_act(qa, prec))


@pytest.mark.parametrize("N,K,kind", [(16, 128, "random"), (48, 1024, "planned"),
                                      (400, 640, "random")])
def test_pack_w4_perm_bit_exact(N, K, kind):
    print(f"pack_w4_perm N={N} K={K} {kind}", flush=True)
    W16 = synth.weights(N, N, K)
    X16 = synth.calibration_activations(5, 32, K, synth.outlier_channels(K, 3, seed=1))
    perm, _ = perm_for(kind, X16, K, N)
    Wp, sw = comet.pack_w4(dev_u16(W16), perm=dev_i32(perm))
    qw, sw_ref = oracle.quantize_weight(oracle.permute_columns(W16, perm))
    assert np.array_equal(host_u16(sw), sw_ref)
    assert np.array_equal(host(Wp), oracle.pack_weight(qw))


def test_perm_null_equals_unpermuted():
    M, K = 40, 512
    X16 = synth.activations(3, M, K, np.array([4, 8, 4, 4], np.uint8))
    prec = np.array([4, 8, 4, 4], np.uint8)
    X = dev_u16(X16)
    A0, s0 = comet.quantize_act(X, prec)
    A1, s1 = comet.quantize_act(X, prec, perm=dev_i32(np.arange(K)))
    assert torch.equal(A0, A1) and torch.equal(s0.view(torch.int16), s1.view(torch.int16))


def test_perm_out_of_range_reads_last_channel():
    M, K = 8, 256
    X16 = synth.normal_fp16(9, 1, (M, K))
    perm = random_perm(K, 2)
    perm[[3, 100, 200]] = [K, -1, 1 << 30]
    prec = np.array([8, 4], np.uint8)
    A, sa = comet.quantize_act(dev_u16(X16), prec, perm=dev_i32(perm))
    clamped = np.where((perm < 0) | (perm >= K), K - 1, perm).astype(np.int32)
    qa, sa_ref = oracle.quantize_act(oracle.permute_columns(X16, clamped), prec)
    assert np.array_equal(host_u16(sa), sa_ref)
    assert np.array_equal(host(A), oracle.pack_act(qa, prec))


@pytest.mark.parametrize("M,N,K", [(64, 256, 1024), (5, 96, 2048)])
def test_calibrated_gemm_end_to_end(M, N, K):
    """Sample -> plan -> permuted quantize/pack -> W4Ax GEMM, against the oracle on
    the permuted operands; and the permutation's purpose: a smaller error than
    all-4-bit quantization of the unpermuted activations."""
    print(f"calibrated gemm M={M} N={N} K={K}", flush=True)
    ch = synth.outlier_channels(K, 7, seed=K)
    calib = synth.calibration_activations(11, 256, K, ch)
    absmax = comet.channel_absmax(dev_u16(calib))
    perm, prec, nout = comet.plan_channel_perm(absmax, 128, 8.0, 0.2)
    assert nout >= 7 and (prec == 8).sum() == 1
    X16 = synth.calibration_activations(12, M, K, ch, tid=synth.TID_X)
    W16 = synth.weights(13, N, K)
    pd = dev_i32(perm)
    A, sa = comet.quantize_act(dev_u16(X16), prec, perm=pd)
    Wp, sw = comet.pack_w4(dev_u16(W16), perm=pd)
    out = host_u16(comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)).view(np.float16)
    qa, sa_r = oracle.quantize_act(oracle.permute_columns(X16, perm), prec)
    qw, sw_r = oracle.quantize_weight(oracle.permute_columns(W16, perm))
    ref = oracle.dequant_gemm(qa, sa_r, qw, sw_r)
    assert_out_close(out, ref)
    exact = oracle.exact_gemm(X16, W16)
    all4 = np.full(K // 128, 4, np.uint8)
    A4, sa4 = comet.quantize_act(dev_u16(X16), all4)
    Wp4, sw4 = comet.pack_w4(dev_u16(W16))
    out4 = host_u16(comet.w4ax_gemm(A4, all4, sa4, Wp4, sw4, M, N, K)).view(np.float16)
    e_perm = np.abs(out.astype(np.float64) - exact).mean()
    e_all4 = np.abs(out4.astype(np.float64) - exact).mean()
    assert e_perm < 0.7 * e_all4


def test_llama3_70b_permuted_quantize_full_size_sampled_rows():
    """K = 8192 hidden size, 4096 tokens, a planned permutation; rows sampled."""
    M, K = 4096, 8192
    print(f"permuted quantize full size M={M} K={K}", flush=True)
    ch = synth.outlier_channels(K, 41, seed=70)
    X16 = synth.calibration_activations(70, M, K, ch)
    absmax = comet.channel_absmax(dev_u16(X16[:512]))
    perm, prec, _ = comet.plan_channel_perm(absmax, 128, 8.0, 0.2)
    A, sa = comet.quantize_act(dev_u16(X16), prec, perm=dev_i32(perm))
    rows = np.array([0, 1, 777, 2048, 4095])
    qa, sa_ref = oracle.quantize_act(oracle.permute_columns(X16[rows], perm), prec)
    assert np.array_equal(host_u16(sa)[:, rows], sa_ref)
    assert np.array_equal(act_rows(host(A), prec, M, rows), oracle.pack_act(qa, prec))


# --- KV4 ---------------------------------------------------------------------------

KV_SHAPES = [(1, 128, 128), (7, 1024, 128), (5, 96, 32), (33, 320, 64), (4096, 1024, 128),
             (3, 64, 64)]


@pytest.mark.parametrize("T,C,G", KV_SHAPES)
def test_kv4_bit_exact(T, C, G):
    print(f"kv4 T={T} C={C} G={G}", flush=True)
    X16 = synth.kv_rows(T, T, C)
    codes, params = comet.kv4_quantize(dev_u16(X16), G)
    c_ref, p_ref = oracle.kv4_quantize(X16, G)
    assert np.array_equal(host(codes), c_ref)
    assert np.array_equal(host_u16(params), p_ref)
    xr = comet.kv4_dequantize(codes, params, G)
    assert np.array_equal(host_u16(xr), oracle.kv4_dequantize(c_ref, p_ref, G))


def test_kv4_edge_values():
    C, G = 256, 128
    rows = [np.zeros(C), np.full(C, 3.5), np.linspace(-65504, 65504, C),
            np.where(np.arange(C) % 2 == 0, 65504.0, -65504.0), np.full(C, -0.0),
            np.linspace(0, 6e-8, C),
            np.where(np.arange(C) % 3 == 0, 0.0, np.where(np.arange(C) % 3 == 1, -0.0, 1.0)),
            np.where(np.arange(C) % 3 == 0, -0.0, np.where(np.arange(C) % 3 == 1, 0.0, -0.0))]
    X16 = np.stack([np.asarray(r, np.float32).astype(np.float16).view(np.uint16) for r in rows])
    codes, params = comet.kv4_quantize(dev_u16(X16), G)
    c_ref, p_ref = oracle.kv4_quantize(X16, G)
    assert np.array_equal(host(codes), c_ref)
    assert np.array_equal(host_u16(params), p_ref)
    assert np.array_equal(host_u16(comet.kv4_dequantize(codes, params, G)),
                          oracle.kv4_dequantize(c_ref, p_ref, G))


# --- SwiGLU + next-layer quantization ---------------------------------------------

@pytest.mark.parametrize("M,I,kind", [(1, 128, "all4"), (7, 384, "random"), (100, 1024, "random"),
                                      (33, 256, "all8")])
def test_swiglu_quantize_bit_exact(M, I, kind):
    print(f"swiglu_quantize M={M} I={I} {kind}", flush=True)
    NG = I // 128
    prec = {"all4": np.full(NG, 4, np.uint8), "all8": np.full(NG, 8, np.uint8),
            "random": synth.prec_map(NG, max(1, NG // 3), "random", M)}[kind]
    gu = synth.normal_fp16(M, 5, (M, 2 * I), 3.0)
    gu[0, :16] = [0, 0x8000, 0x6000, 0xE000, 0x3C00, 0xBC00, 1, 0x8001,
                  0x4900, 0xC900, 0x5640, 0xD640, 0x0400, 0x8400, 0x3555, 0xB555]
    A, sa = comet.swiglu_quantize(dev_u16(gu), prec)
    A_ref, sa_ref = oracle.swiglu_quantize(gu, prec)
    assert np.array_equal(host_u16(sa), sa_ref)
    assert np.array_equal(host(A), A_ref)


def gemm_inputs(M, N, K, seed):
    NG = K // 128
    prec = synth.prec_map(NG, max(1, NG // 8))
    X16 = synth.activations(seed, M, K, prec)
    W16 = synth.weights(seed, N, K)
    A, sa = comet.quantize_act(dev_u16(X16), prec)
    Wp, sw = comet.pack_w4(dev_u16(W16))
    return prec, A, sa, Wp, sw


# few-token (two-step), 128-row tiles, 256-row tiles, split tiles (320 tiles)
FUSED = [(8, 512, 1024), (100, 768, 1024), (300, 1024, 2048), (1024, 20480, 1024)]


@pytest.mark.parametrize("M,N,K", FUSED)
def test_fused_swiglu_matches_oracle_on_gemm_output(M, N, K):
    """The fused epilogue's quantized h is bit-identical to the oracle's SwiGLU
    quantization of the same GEMM's fp16 output (the plain entry point, same
    schedule, so the same fp16 gate/up values)."""
    print(f"fused swiglu M={M} N={N} K={K}", flush=True)
    I = N // 2
    prec, A, sa, Wp, sw = gemm_inputs(M, N, K, seed=M + N)
    out_map = synth.prec_map(I // 128, max(1, I // 128 // 4), "random", seed=N)
    A2, sa2 = comet.w4ax_gemm_swiglu_quant(A, prec, sa, Wp, sw, M, N, K, out_map)
    out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
    gu = host_u16(out)
    rows = np.arange(M) if M <= 300 else np.array([0, 1, 255, 256, 511, 777, M - 1])
    A_ref, sa_ref = oracle.swiglu_quantize(gu[rows], out_map)
    assert np.array_equal(host_u16(sa2)[:, rows], sa_ref)
    assert np.array_equal(act_rows(host(A2), out_map, M, rows), A_ref)
    # the standalone kernel on the same output agrees as well
    A3, sa3 = comet.swiglu_quantize(out, out_map)
    assert torch.equal(A2, A3) and torch.equal(sa2.view(torch.int16), sa3.view(torch.int16))


def test_fused_swiglu_llama3_70b_gate_up_sampled_rows():
    """LLaMA-3-70B gate_up (M = 4096, K = 8192 -> N = 2 x 28672) fused into the
    down projection's input (I = 28672, 1/16 of its blocks 8-bit)."""
    M, (K, N) = 4096, synth.LLAMA3_70B["gate_up"]
    print(f"fused swiglu 70B M={M} N={N} K={K}", flush=True)
    I = N // 2
    prec, A, sa, Wp, sw = gemm_inputs(M, N, K, seed=70)
    out_map = synth.prec_map(I // 128, I // 128 // 16)
    A2, sa2 = comet.w4ax_gemm_swiglu_quant(A, prec, sa, Wp, sw, M, N, K, out_map)
    out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
    rows = np.array([0, 1, 777, 2048, 4095])
    gu = host_u16(out[torch.from_numpy(rows).to(DEV)])
    A_ref, sa_ref = oracle.swiglu_quantize(gu, out_map)
    assert np.array_equal(host_u16(sa2)[:, rows], sa_ref)
    assert np.array_equal(act_rows(host(A2), out_map, M, rows), A_ref)


def test_fused_swiglu_few_tokens_across_workspace_growth():
    """The few-token fused path writes its fp16 gate/up output to a buffer kept
    per stream beside the split-K buffers.  Split GEMMs that grow those buffers
    in between (8 and then 32 split tiles) must leave the fused path exact, and
    the split GEMMs must match the oracle."""
    K = 1024
    steps = [("fused", 32, 1024), ("split", 512, 1024), ("fused", 40, 2048),
             ("split", 1024, 2048), ("fused", 24, 1024)]
    for kind, M, N in steps:
        print(f"workspace growth: {kind} M={M} N={N} K={K}", flush=True)
        NG = K // 128
        prec = synth.prec_map(NG, max(1, NG // 8))
        X16 = synth.activations(M + N, M, K, prec)
        W16 = synth.weights(M + N, N, K)
        A, sa = comet.quantize_act(dev_u16(X16), prec)
        Wp, sw = comet.pack_w4(dev_u16(W16))
        out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
        if kind == "split":
            rows = np.array([0, 1, 255, 256, M - 1])
            qa, osa = oracle.quantize_act(X16[rows], prec)
            qw, osw = oracle.quantize_weight(W16)
            ref = oracle.dequant_gemm(qa, osa, qw, osw)
            assert_out_close(host_u16(out).view(np.float16)[rows], ref, f"split {M}x{N}x{K}")
        else:
            out_map = synth.prec_map(N // 2 // 128, 1, "random", seed=N)
            A2, sa2 = comet.w4ax_gemm_swiglu_quant(A, prec, sa, Wp, sw, M, N, K, out_map)
            A_ref, sa_ref = oracle.swiglu_quantize(host_u16(out), out_map)
            assert np.array_equal(host_u16(sa2), sa_ref)
            assert np.array_equal(host(A2), A_ref)

"""GPU parity where it was thin: every row tile of the full-size layers, the
exact per-block sums of a split tile under the production schedule, the
quantizer's edge rows fed through the GEMM, the wide-N rule for 33-48 rows,
and the schedule modes (which must change nothing but the fp32 summation
order).  Everything is compared with the CPU oracle: packed bytes and int32
sums bit-exactly, fp16 outputs within the tolerance of tests/parity.py.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2410_12168_amd as comet
import synth
from parity import act_rows, assert_out_close
from test_gpu_parity import DEV, dev_u16, host, host_u16, run_path

pytestmark = pytest.mark.gpu


def tile_rows(M, tile=256, seed=0):
    """One token row inside every `tile`-row tile (at a seeded offset), plus
    the first and last rows."""
    rng = np.random.default_rng(seed)
    rows = [t * tile + int(rng.integers(0, tile)) for t in range((M + tile - 1) // tile)]
    return np.unique(np.clip(rows + [0, M - 1], 0, M - 1))


@pytest.mark.parametrize("model,layer", [("70b", "qkv"), ("70b", "o"), ("70b", "gate_up"),
                                         ("70b", "down"), ("8b", "qkv"), ("8b", "o"),
                                         ("8b", "gate_up"), ("8b", "down")])
def test_one_row_per_row_tile_full_size(model, layer):
    # one row in every row tile of the height the schedule picks (the 8B o
    # layer runs 128-row tiles, the others 256)
    shapes, M = (synth.LLAMA3_70B, 4096) if model == "70b" else (synth.LLAMA3_8B, 2048)
    K, N = shapes[layer]
    NG = K // 128
    prec = synth.prec_map(NG, NG // 16)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    tm = comet.comet_schedule_query(M, N, K, prec, num_cus=cus)["tile_m"]
    print(f"row tiles {model} {layer} M={M} N={N} K={K} tile_m={tm}", flush=True)
    r = run_path(M, N, K, prec, seed=21)
    rows = tile_rows(M, tile=tm, seed=NG)
    qa, sa = oracle.quantize_act(r["X16"][rows], prec)
    assert np.array_equal(act_rows(host(r["A"]), prec, M, rows), oracle.pack_act(qa, prec))
    qw, sw = oracle.quantize_weight(r["W16"])
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16)[rows], ref, f"{model} {layer}")


def test_split_tile_acc_window_production_plan():
    """LLaMA-3-70B qkv at M = 4096: 640 tiles on 256 CUs, so the default
    schedule splits the last wave.  The diagnostic entry point runs the same
    schedule; a window inside a split tile must hold the exact block sums."""
    K, N = synth.LLAMA3_70B["qkv"]
    M, NG = 4096, K // 128
    prec = synth.prec_map(NG, NG // 16)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    os.environ.pop("COMET_SCHED", None)
    q = comet.comet_schedule_query(M, N, K, prec, num_cus=cus)
    split = q["units"][q["units"][:, 4] > 1]
    assert len(split) > 0, "expected a split last wave"
    tile = int(split[len(split) // 2, 0])
    tiles_n = (N + 255) // 256
    m0, n0 = (tile // tiles_n) * 256, (tile % tiles_n) * 256
    win = (m0 + 100, m0 + 132, n0 + 200, n0 + 256)  # crosses wave quadrants
    print(f"split tile {tile} window {win}", flush=True)
    r = run_path(M, N, K, prec, seed=31, diag_window=win)
    rows = np.arange(win[0], win[1])
    qa, sa = oracle.quantize_act(r["X16"][rows], prec)
    qw, sw = oracle.quantize_weight(r["W16"][win[2]:win[3]])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa, qw))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    out = host_u16(r["out"]).view(np.float16)[win[0]:win[1], win[2]:win[3]]
    assert_out_close(out, ref, "split tile window")


@pytest.mark.parametrize("M,N,K", [(512, 8192, 8192), (2048, 4096, 14336)])
def test_split_tiles_sum_in_slot_order(M, N, K):
    """Plans whose tiles are split: 512 x 8192 x 8192 cuts each of its 64
    tiles into four slots (all partials added in slot order); the 8B down
    projection's 128 tiles into two (the finishing slot adds the other's
    partial to its registers).  The fp16 output must match the oracle and be
    bit-identical from run to run, whichever slot arrives last."""
    NG = K // 128
    prec = synth.prec_map(NG, NG // 16, "random", seed=M)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    q = comet.comet_schedule_query(M, N, K, prec, num_cus=cus)
    nslots = q["units"][:, 4].max()
    print(f"split slots M={M} N={N} K={K}: up to {nslots} slots per tile", flush=True)
    assert nslots >= 2
    r = run_path(M, N, K, prec, seed=41)
    rows = tile_rows(M, tile=q["tile_m"], seed=3)
    qa, sa = oracle.quantize_act(r["X16"][rows], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16)[rows], ref, f"split {M}x{N}x{K}")
    again = comet.w4ax_gemm(r["A"], prec, r["sa"], r["Wp"], r["sw"], M, N, K)
    assert torch.equal(r["out"].view(torch.int16), again.view(torch.int16))


@pytest.mark.parametrize("M,N", [(6, 64), (6, 512), (70, 256), (300, 512)])
def test_quantizer_edge_rows_through_gemm(M, N):
    """Zero blocks, subnormal-scale blocks, exact ties and +-65504 in an 8-bit
    block, quantized and contracted; every kernel regime (few-token, 128-row,
    256-row tiles) sees them."""
    K = 512
    prec = np.array([4, 8, 4, 8], np.uint8)
    rng = np.random.default_rng(M + N)
    X = rng.standard_normal((M, K)).astype(np.float32)
    X[0::6, :] = 0.0                           # all-zero rows
    X[1::6, :] = 2.0 ** -24                    # smallest subnormal: subnormal scales
    X[2::6, :128] = 0.0
    X[2::6, :8] = [7.0, 2.5, -2.5, 3.5, 0.5, -0.5, 1.5, -1.5]  # ties (scale 1)
    X[3::6, 128:256] *= 0.01
    X[3::6, 128:130] = [65504.0, -65504.0]     # 8-bit block at the fp16 limit
    X[4::6, 256:384] = 0.0                     # one zero block in a live row
    X[5::6, 384:] = -(2.0 ** -20)
    X16 = X.astype(np.float16).view(np.uint16)
    W16 = synth.weights(M, N, K)
    print(f"edge rows M={M} N={N}", flush=True)
    A, sa = comet.quantize_act(dev_u16(X16), prec)
    Wp, sw = comet.pack_w4(dev_u16(W16))
    out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
    acc = comet.w4ax_gemm_acc(A, prec, sa, Wp, sw, M, N, K, 0, M, 0, N)
    qa, osa = oracle.quantize_act(X16, prec)
    qw, osw = oracle.quantize_weight(W16)
    assert np.array_equal(host_u16(sa), osa)
    assert np.array_equal(host(A), oracle.pack_act(qa, prec))
    assert np.array_equal(host(acc), oracle.group_acc(qa, qw))
    ref = oracle.dequant_gemm(qa, osa, qw, osw)
    assert np.abs(ref).max() < 60000.0  # the reference itself fits fp16
    assert_out_close(host_u16(out).view(np.float16), ref, f"edge rows {M}x{N}")


@pytest.mark.parametrize("M", [33, 48])
def test_wide_n_mid_rows_acc_window(M):
    """33 and 48 rows at a gate_up-like width whose panels do not divide over
    256 CUs (N = 57600: 225 column tiles, wide) run on the 128-row tile
    kernel: exact block sums over every row and a column window across a
    tile boundary, and sampled fp16 rows."""
    K, N = 8192, 57600
    NG = K // 128
    assert comet.comet_gemm_kernel(M, N, K, 256) == 2
    prec = synth.prec_map(NG, NG // 16)
    win = (0, M, 256 * 100 - 24, 256 * 100 + 40)
    print(f"wide-N M={M} window {win}", flush=True)
    r = run_path(M, N, K, prec, seed=M, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa, qw[win[2]:win[3]]))
    rows = np.array([0, M // 2, M - 1])
    ref = oracle.dequant_gemm(qa[rows], sa[:, rows], qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16)[rows], ref, f"wide-N M={M}")


@pytest.mark.parametrize("N,kind", [(57344, "stream"), (57600, "mid")])
def test_fused_swiglu_wide_n_mid_rows(N, kind):
    """The fused SwiGLU entry point at M = 40, K = 8192: on the 70B gate_up
    shape (stream kernel, then the standalone SwiGLU quantizer) and at N =
    57600 (the 128-row kernel's fused epilogue), against the oracle's SwiGLU
    quantization of the same GEMM's fp16 output."""
    M, K = 40, 8192
    I = N // 2
    NG = K // 128
    assert comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, 256)] == kind
    print(f"fused swiglu wide-N M={M} N={N} ({kind})", flush=True)
    prec = synth.prec_map(NG, NG // 16)
    A, sa = comet.quantize_act(dev_u16(synth.activations(40, M, K, prec)), prec)
    Wp, sw = comet.pack_w4(dev_u16(synth.weights(40, N, K)))
    out_map = synth.prec_map(I // 128, I // 128 // 16, "random", seed=3)
    A2, sa2 = comet.w4ax_gemm_swiglu_quant(A, prec, sa, Wp, sw, M, N, K, out_map)
    out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
    A_ref, sa_ref = oracle.swiglu_quantize(host_u16(out), out_map)
    assert np.array_equal(host_u16(sa2), sa_ref)
    assert np.array_equal(host(A2), A_ref)


@pytest.mark.parametrize("M,N,K,placement", [(4096, 10240, 8192, "random"),
                                             (300, 1024, 4096, "contiguous"),
                                             (100, 2048, 2048, "random")])
def test_schedule_modes_agree(M, N, K, placement):
    """natural (map order, whole tiles), dp (precision-batched, whole tiles)
    and cost (precision-batched, split last wave) give bit-identical block
    sums and outputs within the oracle tolerance."""
    NG = K // 128
    prec = synth.prec_map(NG, NG // 4, placement, seed=K)
    X16 = synth.activations(7, M, K, prec)
    W16 = synth.weights(7, N, K)
    A, sa = comet.quantize_act(dev_u16(X16), prec)
    Wp, sw = comet.pack_w4(dev_u16(W16))
    win = (M - 20, M, N - 24, N)
    rows = np.array([0, M // 3, M - 1])
    qa, osa = oracle.quantize_act(X16[rows], prec)
    qw, osw = oracle.quantize_weight(W16)
    ref = oracle.dequant_gemm(qa, osa, qw, osw)
    qa_w, _ = oracle.quantize_act(X16[win[0]:win[1]], prec)
    acc_ref = oracle.group_acc(qa_w, qw[win[2]:win[3]])
    try:
        for mode in ("natural", "dp", "cost"):
            print(f"schedule mode {mode} M={M} N={N} K={K}", flush=True)
            os.environ["COMET_SCHED"] = mode
            out = comet.w4ax_gemm(A, prec, sa, Wp, sw, M, N, K)
            acc = comet.w4ax_gemm_acc(A, prec, sa, Wp, sw, M, N, K, *win)
            assert np.array_equal(host(acc), acc_ref), mode
            assert_out_close(host_u16(out).view(np.float16)[rows], ref, f"mode {mode}")
    finally:
        os.environ.pop("COMET_SCHED", None)


STREAM = [
    # (M, N, K, map kind): the persistent few-token stream kernel runs when
    # the 16-column panels divide evenly over the CUs (256 here)
    (1, 57344, 8192, "cfg0"),      # 70B gate_up: activations unpacked in LDS, 56 items per wave
    (8, 57344, 8192, "random"),
    (3, 8192, 8192, "alternate"),  # 70B o: activations from L2, 8 waves per panel
    (8, 8192, 28672, "cfg0"),      # 70B down: activations from L2 (too large for LDS)
    (5, 98304, 768, "random"),     # 1.5 panels per wave: complete and partial panels mixed
    (2, 65536, 1024, "all8"),      # one complete panel per wave
]


@pytest.mark.parametrize("M,N,K,kind", STREAM)
def test_stream_kernel_matches_oracle(M, N, K, kind):
    from test_gpu_parity import make_map

    NG = K // 128
    prec = make_map(kind, NG, seed=N)
    win = (0, M, N // 2 - 24, N // 2 + 40)
    print(f"stream kernel M={M} N={N} K={K} {kind}", flush=True)
    r = run_path(M, N, K, prec, seed=M + K, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa, qw[win[2]:win[3]]))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"stream {M}x{N}x{K}")
    again = comet.w4ax_gemm(r["A"], prec, r["sa"], r["Wp"], r["sw"], M, N, K)
    assert torch.equal(r["out"].view(torch.int16), again.view(torch.int16))


def test_quantizer_every_fp16_block_max():
    """Every positive finite fp16 value as a block's max |x|, in a 4-bit and
    an 8-bit block, with the other channels random fractions of it and exact
    ties: every scale the quantizers can produce meets the hardware
    reciprocal; codes and scales must equal the oracle's bit for bit."""
    amax = np.arange(1, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float32)
    M, K = amax.size, 256
    rng = np.random.default_rng(0)
    X = (rng.uniform(-1.0, 1.0, (M, K)).astype(np.float32) * amax[:, None])
    X[:, 0] = amax
    X[:, 128] = -amax
    X[:, 1] = amax * (2.5 / 7.0)      # near code midpoints of the 4-bit block
    X[:, 129] = amax * (64.5 / 127.0)  # and of the 8-bit block
    X16 = X.astype(np.float16).view(np.uint16)
    prec = np.array([4, 8], np.uint8)
    print(f"every fp16 block max: M={M}", flush=True)
    A, sa = comet.quantize_act(dev_u16(X16), prec)
    qa, osa = oracle.quantize_act(X16, prec)
    assert np.array_equal(host_u16(sa), osa)
    assert np.array_equal(host(A), oracle.pack_act(qa, prec))


CHUNK = [
    # (M, N, K, map kind): the chunked stream kernel (8 < M <= 64) runs when
    # the 16-column panels divide evenly over the CUs (256 here) with at
    # least three items per wave.  7 panels per workgroup: 3 or 4 items per
    # wave, panels split between waves at every offset within a chunk
    (9, 28672, 1152, "random"),       # one row block; last chunk partial (9 blocks)
    (16, 28672, 512, "cfg0"),         # one chunk
    (17, 28672, 1152, "alternate"),   # two row blocks, ragged rows
    (40, 65536, 1664, "all8"),        # 16 panels per workgroup: eight items per wave
    (64, 28672, 640, "random"),       # four row blocks
    (33, 57344, 384, "cfg0"),         # 14 panels per workgroup (LLaMA-3-70B gate_up width)
]


@pytest.mark.parametrize("M,N,K,kind", CHUNK)
def test_chunk_stream_kernel_matches_oracle(M, N, K, kind):
    from test_gpu_parity import make_map

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    NG = K // 128
    prec = make_map(kind, NG, seed=N + M)
    print(f"chunk stream kernel M={M} N={N} K={K} {kind}", flush=True)
    assert comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, cus)] == "stream"
    win = (max(0, M - 40), M, N // 2 - 24, N // 2 + 40)
    r = run_path(M, N, K, prec, seed=M + K, diag_window=win)
    qa, sa = oracle.quantize_act(r["X16"], prec)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host(r["acc"]), oracle.group_acc(qa[win[0]:win[1]], qw[win[2]:win[3]]))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16), ref, f"chunk {M}x{N}x{K}")
    again = comet.w4ax_gemm(r["A"], prec, r["sa"], r["Wp"], r["sw"], M, N, K)
    assert torch.equal(r["out"].view(torch.int16), again.view(torch.int16))

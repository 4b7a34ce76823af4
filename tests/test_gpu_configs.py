"""GPU parity at the benchmark configurations' full sizes.

LLaMA-3-8B linear layers at M = 2048 (K -> N: 4096 -> 6144, 4096 -> 4096,
4096 -> 28672, 14336 -> 4096; 1/16 of the activation blocks 8-bit), the
LLaMA-3-70B o projection at M = 4096 (the other 70B layers are in
test_gpu_parity.py), and the load-balance configuration's hardest point: the
70B down projection with half of its blocks 8-bit at seeded random positions.
The packed weights and scales are checked whole and bit-exactly; the oracle
recomputes a seeded sample of token rows (quantization is per row) and the
fp16 output rows must meet the oracle tolerance.
"""
import numpy as np
import pytest

import oracle
import synth
from parity import act_rows, assert_out_close
from test_gpu_parity import host, host_u16, run_path

pytestmark = pytest.mark.gpu


def check_sampled(M, N, K, prec, seed, rows, what):
    r = run_path(M, N, K, prec, seed=seed)
    qa, sa = oracle.quantize_act(r["X16"][rows], prec)
    assert np.array_equal(act_rows(host(r["A"]), prec, M, rows), oracle.pack_act(qa, prec))
    assert np.array_equal(host_u16(r["sa"])[:, rows], sa)
    qw, sw = oracle.quantize_weight(r["W16"])
    assert np.array_equal(host_u16(r["sw"]), sw)
    assert np.array_equal(host(r["Wp"]), oracle.pack_weight(qw))
    ref = oracle.dequant_gemm(qa, sa, qw, sw)
    assert_out_close(host_u16(r["out"]).view(np.float16)[rows], ref, what)


@pytest.mark.parametrize("layer", ["qkv", "o", "gate_up", "down"])
def test_llama3_8b_full_size_sampled_rows(layer):
    K, N = synth.LLAMA3_8B[layer]
    M, NG = 2048, K // 128
    check_sampled(M, N, K, synth.prec_map(NG, NG // 16), seed=11,
                  rows=np.array([0, 5, 1023, 1024, 2047]), what=f"8B {layer}")


def test_llama3_70b_o_full_size_sampled_rows():
    K, N = synth.LLAMA3_70B["o"]
    M, NG = 4096, K // 128
    check_sampled(M, N, K, synth.prec_map(NG, NG // 16), seed=12,
                  rows=np.array([0, 255, 256, 3000, 4095]), what="70B o")


def test_down_half_8bit_random_placement():
    K, N = synth.LLAMA3_70B["down"]
    M, NG = 4096, K // 128
    check_sampled(M, N, K, synth.prec_map(NG, NG // 2, "random", seed=5), seed=13,
                  rows=np.array([1, 511, 2600, 4094]), what="70B down, half 8-bit random")


def test_128_row_tiles_above_128_rows_ragged():
    # M = 1900 rows, N = K = 4096 on 256 CUs: 240 tiles of 128 rows (the last
    # row tile ragged, 108 rows) beat 128 split tiles of 256 rows, so the
    # 128-row kernel runs with many row tiles; rows on both sides of every
    # kind of boundary are checked
    import torch
    import paper_2410_12168_amd as comet
    M, N, K = 1900, 4096, 4096
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    if cus == 256:
        assert comet.KERNEL_NAMES[comet.comet_gemm_kernel(M, N, K, cus)] == "mid"
    NG = K // 128
    check_sampled(M, N, K, synth.prec_map(NG, 3, "random", seed=7), seed=14,
                  rows=np.array([0, 127, 128, 1023, 1791, 1792, 1899]),
                  what="128-row tiles, M = 1900")

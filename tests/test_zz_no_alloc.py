"""comet_w4ax_gemm_noalloc: the W4Ax GEMM over a fixed per-device workspace
(for callers that cannot allocate), against comet_w4ax_gemm and the oracle.

Two calls in a row, the second with a smaller input (a different schedule in
the shared workspace), on every kernel regime: the outputs must equal the
allocating entry point's bit for bit (same kernels, same schedule) and meet
the oracle tolerance on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_12168_amd as comet
import synth
from parity import assert_out_close
from test_gpu_parity import DEV, dev_u16, host_u16

pytestmark = pytest.mark.gpu


def operands(M, N, K, seed):
    NG = K // 128
    prec = synth.prec_map(NG, max(1, NG // 16), "random", seed=seed)
    X16, W16 = synth.activations(seed, M, K, prec), synth.weights(seed, N, K)
    A, sa = comet.quantize_act(dev_u16(X16), prec)
    Wp, sw = comet.pack_w4(dev_u16(W16))
    return dict(M=M, N=N, K=K, prec=prec, X16=X16, W16=W16, A=A, sa=sa, Wp=Wp, sw=sw)


def noalloc(o, out=None):
    if out is None:
        out = torch.empty((o["M"], o["N"]), dtype=torch.float16, device=DEV)
    comet.comet_w4ax_gemm_noalloc(o["A"], o["prec"], o["sa"], o["Wp"], o["sw"], out, o["M"],
                                  o["N"], o["K"])
    return out


def check(o, out):
    ref = comet.w4ax_gemm(o["A"], o["prec"], o["sa"], o["Wp"], o["sw"], o["M"], o["N"], o["K"])
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    M = o["M"]
    rows = np.unique(np.clip([0, 1, M // 2, M - 2, M - 1], 0, M - 1))
    qa, sa = oracle.quantize_act(o["X16"][rows], o["prec"])
    qw, sw = oracle.quantize_weight(o["W16"])
    assert_out_close(host_u16(out).view(np.float16)[rows], oracle.dequant_gemm(qa, sa, qw, sw),
                     f"noalloc {M}x{o['N']}x{o['K']}")


CASES = [
    # 256-row tiles: LLaMA-3-70B qkv (640 tiles, the last wave split: 64 MiB
    # of partials, the whole partial region), then a small GEMM
    ((4096, 10240, 8192), (300, 1024, 2048)),
    # LLaMA-3-8B o projection (128 tiles, all split), then a smaller split plan
    ((2048, 4096, 4096), (1024, 2048, 1024)),
    # 128-row tiles (70B gate_up at M = 128), then a ragged one
    ((128, 57344, 8192), (65, 512, 1024)),
    # few-token kernels (no workspace)
    ((8, 8192, 4096), (1, 256, 1024)),
]


@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_gemm_on_two_calls(first, second):
    print(f"noalloc {first} then {second}", flush=True)
    o1, o2 = operands(*first, seed=1), operands(*second, seed=2)
    out1 = noalloc(o1)
    out2 = noalloc(o2)
    torch.cuda.synchronize()
    check(o1, out1)
    check(o2, out2)
    # and back to the first shape: its schedule is uploaded again
    out3 = noalloc(o1)
    torch.cuda.synchronize()
    assert torch.equal(out3.view(torch.int16), out1.view(torch.int16))


def test_noalloc_allocates_nothing():
    """After the first calls (which load the kernels and look up the
    workspace), further calls with changing shapes leave the device's free
    memory unchanged."""
    print("noalloc free memory", flush=True)
    o1, o2 = operands(2048, 4096, 4096, seed=3), operands(128, 8192, 2048, seed=4)
    o3 = operands(8, 1024, 1024, seed=5)
    outs = [torch.empty((o["M"], o["N"]), dtype=torch.float16, device=DEV) for o in (o1, o2, o3)]
    for o, out in zip((o1, o2, o3), outs):
        noalloc(o, out)
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    for _ in range(3):
        for o, out in zip((o1, o2, o3), outs):
            noalloc(o, out)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0
    check(o1, outs[0])


def test_noalloc_refuses_oversized_schedule():
    """104,960 output tiles need a 2.1 MB schedule, more than the workspace's
    2 MiB plan region: refused before anything is enqueued (the buffers are
    real, so nothing could be read out of bounds either way)."""
    M, N, K = 65536, 256 * 410, 128
    print(f"noalloc oversized schedule {M}x{N}x{K}", flush=True)
    prec = [4]
    A = torch.empty(M * 64, dtype=torch.uint8, device=DEV)
    sa = torch.empty((1, M), dtype=torch.float16, device=DEV)
    Wp = torch.empty(N * K // 2, dtype=torch.uint8, device=DEV)
    sw = torch.empty((1, N), dtype=torch.float16, device=DEV)
    out = torch.empty((M, N), dtype=torch.float16, device=DEV)
    with pytest.raises(comet.CometError, match="no-allocation workspace"):
        comet.comet_w4ax_gemm_noalloc(A, prec, sa, Wp, sw, out, M, N, K)
    del out
    torch.cuda.empty_cache()

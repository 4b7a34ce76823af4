"""The C-ABI library loads, exports every symbol include/comet.h declares,
and rejects bad arguments before touching a device (CPU-only tests: no kernel
is launched)."""
import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

import paper_2410_12168_amd as comet

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "comet.h")
FAKE = 0x10000  # 16-byte aligned address that is never dereferenced


def declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(comet_[a-z0-9_]+)\s*\(", text)))


def test_header_compiles_as_c():
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-fsyntax-only", "-x", "c", HEADER],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_library_exports_declared_symbols():
    lib = comet.lib()
    names = declared()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    nm = subprocess.run(["nm", "-D", "--defined-only", comet.LIB_PATH], capture_output=True,
                        text=True).stdout
    for n in names:
        assert re.search(r"\bT " + n + r"\b", nm), n


def gemm(prec=(4, 8), M=16, N=32, K=256, G=128, A=FAKE, out=FAKE):
    m = np.asarray(prec, np.uint8)
    return comet.lib().comet_w4ax_gemm(ctypes.c_void_p(A), ctypes.c_void_p(m.ctypes.data),
                                       ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE),
                                       ctypes.c_void_p(FAKE), ctypes.c_void_p(out), M, N, K, G,
                                       None)


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), 1), (dict(N=0), 1), (dict(N=24), 1), (dict(K=200), 1), (dict(K=64), 1),
    (dict(G=64, K=256), 2), (dict(prec=(4, 5)), 1), (dict(A=0), 1), (dict(out=FAKE + 8), 1),
    (dict(K=65536 + 128, prec=(4,) * 513), 2), (dict(M=65535 * 32 + 1), 2),
])
def test_gemm_argument_errors(kw, status):
    assert gemm(**kw) == status
    assert comet.comet_last_error() != ""


def test_quantize_and_pack_argument_errors():
    L = comet.lib()
    m = np.array([4, 8], np.uint8)
    p = ctypes.c_void_p
    assert L.comet_fmpq_quantize_act(p(FAKE), p(m.ctypes.data), p(FAKE), p(FAKE), 0, 256, 128,
                                     None) == 1
    assert L.comet_fmpq_quantize_act(p(FAKE), None, p(FAKE), p(FAKE), 4, 256, 128, None) == 1
    assert L.comet_fmpq_quantize_act(p(FAKE + 2), p(m.ctypes.data), p(FAKE), p(FAKE), 4, 256, 128,
                                     None) == 1
    assert L.comet_pack_w4(p(FAKE), p(FAKE), p(FAKE), 16, 384, 96, None) == 2
    assert L.comet_pack_w4(p(FAKE), None, p(FAKE), 16, 256, 128, None) == 1


def test_acc_window_errors():
    L = comet.lib()
    m = np.array([4, 8], np.uint8)
    p = ctypes.c_void_p
    args = [p(FAKE), p(m.ctypes.data), p(FAKE), p(FAKE), p(FAKE), p(FAKE), 16, 32, 256, 128]
    assert L.comet_w4ax_gemm_acc(*args, 0, 17, 0, 32, None) == 1
    assert L.comet_w4ax_gemm_acc(*args, 4, 4, 0, 32, None) == 1
    assert L.comet_w4ax_gemm_acc(*args, 0, 16, -1, 32, None) == 1


def test_packed_bytes():
    assert comet.comet_act_packed_bytes([4, 8, 4], 10, 384) == 10 * (64 + 128 + 64)
    assert comet.comet_act_packed_bytes([4, 7], 10, 256) == 0
    assert comet.comet_act_packed_bytes([4], 10, 200) == 0


def _child(code: str, env: dict) -> str:
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       env={**os.environ, **env}, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    return r.stdout.strip()


def test_unsupported_architecture_is_reported():
    # valid arguments reach the device check; a forced non-gfx950 architecture
    # must give COMET_ERR_UNSUPPORTED before anything is enqueued
    code = ("import ctypes, numpy as np, paper_2410_12168_amd as c\n"
            "m = np.array([4, 8], np.uint8); p = ctypes.c_void_p\n"
            "print(c.lib().comet_w4ax_gemm(p(65536), p(m.ctypes.data), p(65536), p(65536),"
            " p(65536), p(65536), 16, 32, 256, 128, None), c.comet_last_error())")
    out = _child(code, {"COMET_TEST_FORCE_ARCH": "gfx942"})
    assert out.startswith("2 ") and "gfx950" in out


def test_status_strings():
    assert comet.comet_status_str(0) == "COMET_OK"
    assert comet.comet_status_str(2) == "COMET_ERR_UNSUPPORTED"


def test_wrappers_reject_host_tensors():
    # checked before any library call: the kernels read plain device memory
    import torch

    X = torch.zeros((4, 256), dtype=torch.float16)
    with pytest.raises(ValueError, match="CUDA tensor"):
        comet.quantize_act(X, [4, 8])
    with pytest.raises(ValueError, match="CUDA tensor"):
        comet.pack_w4(X)
    with pytest.raises(ValueError, match="CUDA tensor"):
        comet.kv4_quantize(X)
    with pytest.raises(ValueError, match="CUDA tensor"):
        comet.w4ax_gemm(X, [4, 8], X, X, X, 4, 16, 256)


def test_missing_library_raises(monkeypatch, tmp_path):
    # no fallback: without libcomet.so and with a failing build, the first
    # call raises the build's error
    import paper_2410_12168_amd.build as build_mod

    def failing_build(*a, **k):
        raise RuntimeError("hipcc failed (forced)")

    monkeypatch.setattr(comet, "_lib", None)
    monkeypatch.setattr(comet, "LIB_PATH", str(tmp_path / "libcomet.so"))
    monkeypatch.setattr(build_mod, "build", failing_build)
    with pytest.raises(RuntimeError, match="forced"):
        comet.comet_act_packed_bytes([4], 1, 128)

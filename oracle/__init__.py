"""Python access to the CPU oracle (test infrastructure only).

Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
use this module.  It loads ``oracle/liboracle.so`` (building it with gcc if it is
not there) and wraps each C function with numpy arrays.  Nothing here touches
the GPU library.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I = ctypes.c_int
    S = ctypes.c_size_t
    sig = {
        "orc_f16_from_f32": (ctypes.c_uint16, [ctypes.c_float]),
        "orc_f32_from_f16": (ctypes.c_float, [ctypes.c_uint16]),
        "orc_f16_from_f32_array": (None, [P, P, S]),
        "orc_f32_from_f16_array": (None, [P, P, S]),
        "orc_quantize_group": (I, [P, I, I, P, P]),
        "orc_quantize_act": (I, [P, P, I, I, I, P, P, I]),
        "orc_quantize_weight": (I, [P, I, I, I, P, P, I]),
        "orc_act_packed_bytes": (S, [P, I, I, I]),
        "orc_encode4": (None, [P, I, P]),
        "orc_encode8": (None, [P, I, P]),
        "orc_pack_act": (I, [P, P, I, I, I, P]),
        "orc_pack_weight": (I, [P, I, I, I, P]),
        "orc_group_acc": (None, [P, P, I, I, I, I, P]),
        "orc_dequant_gemm": (None, [P, P, P, P, I, I, I, I, P, I, P, I]),
        "orc_exact_gemm": (None, [P, P, I, I, I, P, I]),
        "orc_permute_columns": (I, [P, P, I, I, P]),
        "orc_channel_absmax": (None, [P, I, I, P]),
        "orc_plan_channel_perm": (I, [P, I, I, ctypes.c_float, ctypes.c_float, P, P, P]),
        "orc_kv4_quantize": (I, [P, I, I, I, P, P]),
        "orc_kv4_dequantize": (I, [P, P, I, I, I, P]),
        "orc_exp_f32": (ctypes.c_float, [ctypes.c_float]),
        "orc_silu_f32": (ctypes.c_float, [ctypes.c_float]),
        "orc_swiglu_f16": (ctypes.c_uint16, [ctypes.c_uint16, ctypes.c_uint16]),
        "orc_swiglu_quantize": (I, [P, I, I, I, P, P, P, I]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# --- fp16 ---------------------------------------------------------------------

def f16_from_f32(x) -> np.ndarray:
    """IEEE binary16 bit patterns (uint16) of fp32 values, round to nearest even."""
    x = _c(x, np.float32).reshape(-1)
    out = np.empty(x.size, dtype=np.uint16)
    _load().orc_f16_from_f32_array(_p(x), _p(out), x.size)
    return out


def f32_from_f16(h) -> np.ndarray:
    h = _c(h, np.uint16).reshape(-1)
    out = np.empty(h.size, dtype=np.float32)
    _load().orc_f32_from_f16_array(_p(h), _p(out), h.size)
    return out


# --- quantization ---------------------------------------------------------------

def quantize_group(v, bits: int):
    """Q(): returns (s16 uint16 bit pattern, int8 codes)."""
    v = _c(v, np.float32).reshape(-1)
    q = np.empty(v.size, dtype=np.int8)
    s = np.zeros(1, dtype=np.uint16)
    rc = _load().orc_quantize_group(_p(v), v.size, bits, _p(s), _p(q))
    if rc:
        raise ValueError("oracle rejected the block (non-finite input or bad bits)")
    return int(s[0]), q


def quantize_act(X16, prec, G: int = 128, nthreads: int = 0):
    """X16: uint16 fp16 bits [M][K]; prec: uint8 [K/G].  Returns (qa int8 [M][K], sa16 uint16 [K/G][M])."""
    X16 = _c(X16, np.uint16)
    prec = _c(prec, np.uint8)
    M, K = X16.shape
    qa = np.empty((M, K), dtype=np.int8)
    sa = np.empty((K // G, M), dtype=np.uint16)
    rc = _load().orc_quantize_act(_p(X16), _p(prec), M, K, G, _p(qa), _p(sa), nthreads)
    if rc:
        raise ValueError("oracle rejected the activations")
    return qa, sa


def quantize_weight(W16, G: int = 128, nthreads: int = 0):
    """W16: uint16 fp16 bits [N][K].  Returns (qw int8 [N][K], sw16 uint16 [K/G][N])."""
    W16 = _c(W16, np.uint16)
    N, K = W16.shape
    qw = np.empty((N, K), dtype=np.int8)
    sw = np.empty((K // G, N), dtype=np.uint16)
    rc = _load().orc_quantize_weight(_p(W16), N, K, G, _p(qw), _p(sw), nthreads)
    if rc:
        raise ValueError("oracle rejected the weights")
    return qw, sw


# --- encodings ------------------------------------------------------------------

def encode4(q) -> np.ndarray:
    q = _c(q, np.int8).reshape(-1)
    out = np.empty(q.size // 2, dtype=np.uint8)
    _load().orc_encode4(_p(q), q.size, _p(out))
    return out


def encode8(q) -> np.ndarray:
    q = _c(q, np.int8).reshape(-1)
    out = np.empty(q.size, dtype=np.uint8)
    _load().orc_encode8(_p(q), q.size, _p(out))
    return out


def act_packed_bytes(prec, M: int, K: int, G: int = 128) -> int:
    prec = _c(prec, np.uint8)
    return int(_load().orc_act_packed_bytes(_p(prec), M, K, G))


def pack_act(qa, prec, G: int = 128) -> np.ndarray:
    qa = _c(qa, np.int8)
    prec = _c(prec, np.uint8)
    M, K = qa.shape
    out = np.empty(act_packed_bytes(prec, M, K, G), dtype=np.uint8)
    if _load().orc_pack_act(_p(qa), _p(prec), M, K, G, _p(out)):
        raise ValueError("bad arguments to pack_act")
    return out


def pack_weight(qw, G: int = 128) -> np.ndarray:
    """N*K/2 bytes in 16-row panels (see oracle.h), returned with shape (N, K/2)."""
    qw = _c(qw, np.int8)
    N, K = qw.shape
    out = np.empty((N, K // 2), dtype=np.uint8)
    if _load().orc_pack_weight(_p(qw), N, K, G, _p(out)):
        raise ValueError("bad arguments to pack_weight")
    return out


# --- contraction ----------------------------------------------------------------

def group_acc(qa, qw, G: int = 128) -> np.ndarray:
    """int32 [M][N][K/G] per-block integer products."""
    qa = _c(qa, np.int8)
    qw = _c(qw, np.int8)
    M, K = qa.shape
    N = qw.shape[0]
    acc = np.empty((M, N, K // G), dtype=np.int32)
    _load().orc_group_acc(_p(qa), _p(qw), M, N, K, G, _p(acc))
    return acc


def dequant_gemm(qa, sa16, qw, sw16, G: int = 128, rows=None, nthreads: int = 0) -> np.ndarray:
    """fp64 [len(rows) or M][N]: sum over blocks of acc * sa * sw."""
    qa = _c(qa, np.int8)
    qw = _c(qw, np.int8)
    sa16 = _c(sa16, np.uint16)
    sw16 = _c(sw16, np.uint16)
    M, K = qa.shape
    N = qw.shape[0]
    if rows is None:
        r = None
        nrows = M
    else:
        r = _c(rows, np.int32)
        nrows = r.size
    ref = np.empty((nrows, N), dtype=np.float64)
    _load().orc_dequant_gemm(_p(qa), _p(sa16), _p(qw), _p(sw16), M, N, K, G,
                             None if r is None else _p(r), nrows, _p(ref), nthreads)
    return ref


def exact_gemm(X16, W16, nthreads: int = 0) -> np.ndarray:
    X16 = _c(X16, np.uint16)
    W16 = _c(W16, np.uint16)
    M, K = X16.shape
    N = W16.shape[0]
    out = np.empty((M, N), dtype=np.float64)
    _load().orc_exact_gemm(_p(X16), _p(W16), M, N, K, _p(out), nthreads)
    return out


# --- channel permutation and calibration map (Sec. 3.2) ---------------------------

def permute_columns(X16, perm) -> np.ndarray:
    """out[r][c] = X16[r][perm[c]] (uint16 fp16 bits)."""
    X16 = _c(X16, np.uint16)
    perm = _c(perm, np.int32)
    R, K = X16.shape
    out = np.empty((R, K), dtype=np.uint16)
    if _load().orc_permute_columns(_p(X16), _p(perm), R, K, _p(out)):
        raise ValueError("permutation index out of range")
    return out


def channel_absmax(X16, absmax=None) -> np.ndarray:
    """fp32 [K] running maximum of |X| per channel over the rows of X16."""
    X16 = _c(X16, np.uint16)
    M, K = X16.shape
    out = np.zeros(K, np.float32) if absmax is None else _c(absmax, np.float32).copy()
    _load().orc_channel_absmax(_p(X16), M, K, _p(out))
    return out


def plan_channel_perm(absmax, G: int, outlier_ratio: float, max_frac8: float):
    """Returns (perm int32 [K], prec uint8 [K/G], n_outliers)."""
    a = _c(absmax, np.float32).reshape(-1)
    K = a.size
    perm = np.empty(K, np.int32)
    prec = np.empty(K // G if G > 0 else 0, np.uint8)
    nout = np.zeros(1, np.int32)
    rc = _load().orc_plan_channel_perm(_p(a), K, G, outlier_ratio, max_frac8, _p(perm), _p(prec),
                                       _p(nout))
    if rc:
        raise ValueError("oracle rejected the calibration arguments")
    return perm, prec, int(nout[0])


# --- KV4 ------------------------------------------------------------------------------

def kv4_quantize(X16, G: int = 128):
    """X16 uint16 [T][C] -> (codes uint8 [T][C/2], params uint16 [T][C/G][2])."""
    X16 = _c(X16, np.uint16)
    T, C = X16.shape
    codes = np.empty((T, C // 2), np.uint8)
    params = np.empty((T, C // G, 2), np.uint16)
    if _load().orc_kv4_quantize(_p(X16), T, C, G, _p(codes), _p(params)):
        raise ValueError("oracle rejected the KV rows")
    return codes, params


def kv4_dequantize(codes, params, G: int = 128) -> np.ndarray:
    codes = _c(codes, np.uint8)
    params = _c(params, np.uint16)
    T = codes.shape[0]
    C = codes.shape[1] * 2
    out = np.empty((T, C), np.uint16)
    if _load().orc_kv4_dequantize(_p(codes), _p(params), T, C, G, _p(out)):
        raise ValueError("bad arguments to kv4_dequantize")
    return out


# --- SwiGLU and next-layer quantization ----------------------------------------------

def exp_f32(x) -> np.ndarray:
    x = np.asarray(x, np.float32).reshape(-1)
    f = _load().orc_exp_f32
    return np.array([f(float(v)) for v in x], np.float32)


def silu_f32(x) -> np.ndarray:
    x = np.asarray(x, np.float32).reshape(-1)
    f = _load().orc_silu_f32
    return np.array([f(float(v)) for v in x], np.float32)


def swiglu_f16(g16, u16) -> np.ndarray:
    g16 = np.asarray(g16, np.uint16).reshape(-1)
    u16 = np.asarray(u16, np.uint16).reshape(-1)
    f = _load().orc_swiglu_f16
    return np.array([f(int(a), int(b)) for a, b in zip(g16, u16)], np.uint16)


def swiglu_quantize(gu16, prec, G: int = 128, nthreads: int = 0):
    """gu16 uint16 [M][2I] (2G-wide gate/up column groups) -> (A_packed, sa16 [I/G][M])."""
    gu16 = _c(gu16, np.uint16)
    prec = _c(prec, np.uint8)
    M, N = gu16.shape
    I = N // 2
    A = np.empty(act_packed_bytes(prec, M, I, G), np.uint8)
    sa = np.empty((I // G, M), np.uint16)
    if _load().orc_swiglu_quantize(_p(gu16), M, I, G, _p(prec), _p(A), _p(sa), nthreads):
        raise ValueError("oracle rejected the swiglu inputs")
    return A, sa

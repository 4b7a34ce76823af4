"""Python binding of libcomet (include/comet.h): COMET's W4Ax hot path on MI355X.

The functions named like the C entry points pass tensor data pointers, sizes
and the current HIP stream straight through ctypes; every step of the path
runs in libcomet's gfx950 kernels.  PyTorch only provides device memory and
streams.  There is no CPU fallback: if libcomet.so is missing and cannot be
built, importing a function raises.

Convenience wrappers (``quantize_act``, ``pack_w4``, ``w4ax_gemm``,
``channel_absmax``, ``plan_channel_perm``, ``kv4_quantize``, ``kv4_dequantize``)
allocate the outputs with ``torch.empty`` and call the same entry points.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcomet.so")
G = 128

_lib = None


class CometError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status


def _status_name(s: int) -> str:
    return {0: "COMET_OK", 1: "COMET_ERR_INVALID_ARG", 2: "COMET_ERR_UNSUPPORTED",
            3: "COMET_ERR_HIP", 4: "COMET_ERR_OOM"}.get(s, f"status {s}")


def lib():
    """The loaded libcomet.so.  A library file whose source stamp differs from
    the sources in this tree (or a missing one) is rebuilt in-tree with hipcc
    before loading, or, with COMET_NO_REBUILD=1 in the environment, refused;
    a stale build is never loaded."""
    global _lib
    if _lib is not None:
        return _lib
    from . import build as _build

    want = _build.source_stamp()
    have = _build.library_stamp(LIB_PATH)
    if have != want:
        if os.environ.get("COMET_NO_REBUILD"):
            raise RuntimeError(f"{LIB_PATH} was built from other sources (stamp {have}, sources "
                               f"{want}) and COMET_NO_REBUILD is set; rebuild it")
        _build.build()
        have = _build.library_stamp(LIB_PATH)
        if have != want:
            raise RuntimeError(f"{LIB_PATH}: stamp {have} after rebuilding, sources {want}")
    L = ctypes.CDLL(LIB_PATH)
    P, I, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    sigs = {
        "comet_act_packed_bytes": (S, [P, I, I, I]),
        "comet_fmpq_quantize_act": (I, [P, P, P, P, I, I, I, P]),
        "comet_pack_w4": (I, [P, P, P, I, I, I, P]),
        "comet_w4ax_gemm": (I, [P, P, P, P, P, P, I, I, I, I, P]),
        "comet_w4ax_gemm_acc": (I, [P, P, P, P, P, P, I, I, I, I, I, I, I, I, P]),
        "comet_schedule_query": (I, [I, I, I, I, P, I, P, I, P, P, I, P, P, P, P]),
        "comet_fmpq_quantize_act_perm": (I, [P, P, P, P, P, I, I, I, P]),
        "comet_pack_w4_perm": (I, [P, P, P, P, I, I, I, P]),
        "comet_channel_absmax": (I, [P, P, I, I, P]),
        "comet_plan_channel_perm": (I, [P, I, I, ctypes.c_float, ctypes.c_float, P, P, P]),
        "comet_kv4_quantize": (I, [P, P, P, I, I, I, P]),
        "comet_kv4_dequantize": (I, [P, P, P, I, I, I, P]),
        "comet_w4ax_gemm_swiglu_quant": (I, [P, P, P, P, P, I, I, I, I, P, P, P, P]),
        "comet_swiglu_quantize": (I, [P, P, P, P, I, I, I, P]),
        "comet_gemm_kernel": (I, [I, I, I, I, I]),
        "comet_w4ax_gemm_noalloc": (I, [P, P, P, P, P, P, I, I, I, I, P]),
        "comet_build_stamp": (ctypes.c_char_p, []),
        "comet_status_str": (ctypes.c_char_p, [I]),
        "comet_last_error": (ctypes.c_char_p, []),
        "comet_release_caches": (None, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    if L.comet_build_stamp().decode() != want:
        raise RuntimeError(f"{LIB_PATH} reports stamp {L.comet_build_stamp().decode()}, "
                           f"sources {want}")
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise CometError(status, lib().comet_last_error().decode())


def _ptr(t) -> ctypes.c_void_p:
    if t is None:
        return ctypes.c_void_p(0)
    if isinstance(t, int):
        return ctypes.c_void_p(t)
    if isinstance(t, np.ndarray):
        return ctypes.c_void_p(t.ctypes.data)
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        import torch

        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _tensor(t, dtype: str, name: str):
    """A convenience wrapper's tensor argument.  The kernels read plain
    row-major device memory, so a view with strides, another dtype or a host
    tensor would be misread; they are rejected here instead."""
    import torch

    want = getattr(torch, dtype)
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != want or not t.is_contiguous():
        got = (f"{t.dtype} on {t.device}{'' if t.is_contiguous() else ', strided'}"
               if isinstance(t, torch.Tensor) else type(t).__name__)
        raise ValueError(f"{name}: need a contiguous {dtype} CUDA tensor, got {got}")
    return t


def _map(prec, K: Optional[int] = None, G: int = G, name: str = "group_prec_map") -> np.ndarray:
    """The host block-precision map as uint8.  With K given, it must hold
    exactly K / G entries: the library reads that many from the pointer."""
    m = np.ascontiguousarray(np.asarray(prec, dtype=np.uint8).reshape(-1))
    if K is not None and G > 0 and K % G == 0 and m.size != K // G:
        raise ValueError(f"{name}: {m.size} entries, need K/G = {K // G}")
    return m


def _nbytes(t) -> Optional[int]:
    """Size in bytes of a tensor or array argument (None for raw pointers)."""
    if t is None or isinstance(t, int):
        return None
    if isinstance(t, np.ndarray):
        return t.nbytes
    return t.numel() * t.element_size()


def _room(t, need: int, name: str) -> None:
    """A buffer passed as a tensor or array must hold at least `need` bytes
    (the kernels read or write that many); raw integer pointers are the
    caller's responsibility."""
    have = _nbytes(t)
    if have is not None and need > 0 and have < need:
        raise ValueError(f"{name}: {have} bytes, the call needs {need}")


def _gemm_room(A_packed, m, a_scales, W_packed, w_scales, M, N, K, G_):
    if M > 0 and N > 0 and K > 0 and G_ > 0 and K % G_ == 0:
        NG = K // G_
        _room(A_packed, comet_act_packed_bytes(m, M, K, G_), "A_packed")
        _room(a_scales, 2 * NG * M, "a_scales")
        _room(W_packed, N * K // 2, "W_packed")
        _room(w_scales, 2 * NG * N, "w_scales")


# --- the C entry points ----------------------------------------------------------

def comet_act_packed_bytes(group_prec_map, M: int, K: int, G: int = G) -> int:
    m = _map(group_prec_map, K, G)
    return int(lib().comet_act_packed_bytes(_ptr(m), M, K, G))


def comet_fmpq_quantize_act(X, group_prec_map, A_packed, a_scales, M: int, K: int, G: int = G,
                            stream=None) -> None:
    m = _map(group_prec_map, K, G)
    _quant_room(X, m, A_packed, a_scales, M, K, G)
    _check(lib().comet_fmpq_quantize_act(_ptr(X), _ptr(m), _ptr(A_packed), _ptr(a_scales), M, K,
                                         G, _stream(stream)))


def _quant_room(X, m, A_packed, a_scales, M, K, G_):
    if M > 0 and K > 0 and G_ > 0 and K % G_ == 0:
        _room(X, 2 * M * K, "X")
        _room(A_packed, comet_act_packed_bytes(m, M, K, G_), "A_packed")
        _room(a_scales, 2 * (K // G_) * M, "a_scales")


def _pack_room(W, W_packed, w_scales, N, K, G_):
    if N > 0 and K > 0 and G_ > 0 and K % G_ == 0:
        _room(W, 2 * N * K, "W")
        _room(W_packed, N * K // 2, "W_packed")
        _room(w_scales, 2 * (K // G_) * N, "w_scales")


def comet_pack_w4(W, W_packed, w_scales, N: int, K: int, G: int = G, stream=None) -> None:
    _pack_room(W, W_packed, w_scales, N, K, G)
    _check(lib().comet_pack_w4(_ptr(W), _ptr(W_packed), _ptr(w_scales), N, K, G,
                               _stream(stream)))


def comet_fmpq_quantize_act_perm(X, perm, group_prec_map, A_packed, a_scales, M: int, K: int,
                                 G: int = G, stream=None) -> None:
    m = _map(group_prec_map, K, G)
    _quant_room(X, m, A_packed, a_scales, M, K, G)
    _room(perm, 4 * K, "perm")
    _check(lib().comet_fmpq_quantize_act_perm(_ptr(X), _ptr(perm), _ptr(m), _ptr(A_packed),
                                              _ptr(a_scales), M, K, G, _stream(stream)))


def comet_pack_w4_perm(W, perm, W_packed, w_scales, N: int, K: int, G: int = G,
                       stream=None) -> None:
    _pack_room(W, W_packed, w_scales, N, K, G)
    _room(perm, 4 * K, "perm")
    _check(lib().comet_pack_w4_perm(_ptr(W), _ptr(perm), _ptr(W_packed), _ptr(w_scales), N, K, G,
                                    _stream(stream)))


def comet_channel_absmax(X, absmax, M: int, K: int, stream=None) -> None:
    if M > 0 and K > 0:
        _room(X, 2 * M * K, "X")
        _room(absmax, 4 * K, "absmax")
    _check(lib().comet_channel_absmax(_ptr(X), _ptr(absmax), M, K, _stream(stream)))


def comet_plan_channel_perm(absmax, K: int, G: int, outlier_ratio: float, max_frac_8bit: float,
                            perm, group_prec_map, n_outliers=None) -> None:
    """Host-only: absmax, perm, group_prec_map (and n_outliers) are host numpy arrays."""
    if K > 0 and G > 0 and K % G == 0:
        _room(absmax, 4 * K, "absmax")
        _room(perm, 4 * K, "perm")
        _room(group_prec_map, K // G, "group_prec_map")
        _room(n_outliers, 4, "n_outliers")
    _check(lib().comet_plan_channel_perm(_ptr(absmax), K, G, outlier_ratio, max_frac_8bit,
                                         _ptr(perm), _ptr(group_prec_map), _ptr(n_outliers)))


def _kv4_room(X, codes, params, T, C, G_, xname):
    if T > 0 and C > 0 and G_ > 0 and C % G_ == 0:
        _room(X, 2 * T * C, xname)
        _room(codes, T * C // 2, "codes")
        _room(params, 4 * T * (C // G_), "params")


def comet_kv4_quantize(X, codes, params, T: int, C: int, G: int = 128, stream=None) -> None:
    _kv4_room(X, codes, params, T, C, G, "X")
    _check(lib().comet_kv4_quantize(_ptr(X), _ptr(codes), _ptr(params), T, C, G,
                                    _stream(stream)))


def comet_kv4_dequantize(codes, params, out, T: int, C: int, G: int = 128, stream=None) -> None:
    _kv4_room(out, codes, params, T, C, G, "out")
    _check(lib().comet_kv4_dequantize(_ptr(codes), _ptr(params), _ptr(out), T, C, G,
                                      _stream(stream)))


def comet_w4ax_gemm_swiglu_quant(A_packed, group_prec_map, a_scales, W_packed, w_scales, M: int,
                                 N: int, K: int, G: int, out_prec_map, out_A_packed, out_a_scales,
                                 stream=None) -> None:
    m = _map(group_prec_map, K, G)
    om = _map(out_prec_map, N // 2, G, "out_prec_map")
    _gemm_room(A_packed, m, a_scales, W_packed, w_scales, M, N, K, G)
    if M > 0 and N > 0 and (N // 2) % G == 0:
        _room(out_A_packed, comet_act_packed_bytes(om, M, N // 2, G), "out_A_packed")
        _room(out_a_scales, 2 * (N // 2 // G) * M, "out_a_scales")
    _check(lib().comet_w4ax_gemm_swiglu_quant(_ptr(A_packed), _ptr(m), _ptr(a_scales),
                                              _ptr(W_packed), _ptr(w_scales), M, N, K, G,
                                              _ptr(om), _ptr(out_A_packed), _ptr(out_a_scales),
                                              _stream(stream)))


def comet_swiglu_quantize(gu, out_prec_map, out_A_packed, out_a_scales, M: int, I: int,
                          G: int = G, stream=None) -> None:
    om = _map(out_prec_map, I, G, "out_prec_map")
    if M > 0 and I > 0 and I % G == 0:
        _room(gu, 4 * M * I, "gu")
        _room(out_A_packed, comet_act_packed_bytes(om, M, I, G), "out_A_packed")
        _room(out_a_scales, 2 * (I // G) * M, "out_a_scales")
    _check(lib().comet_swiglu_quantize(_ptr(gu), _ptr(om), _ptr(out_A_packed),
                                       _ptr(out_a_scales), M, I, G, _stream(stream)))


def comet_w4ax_gemm(A_packed, group_prec_map, a_scales, W_packed, w_scales, out, M: int, N: int,
                    K: int, G: int = G, stream=None) -> None:
    m = _map(group_prec_map, K, G)
    _gemm_room(A_packed, m, a_scales, W_packed, w_scales, M, N, K, G)
    _room(out, 2 * M * N, "out")
    _check(lib().comet_w4ax_gemm(_ptr(A_packed), _ptr(m), _ptr(a_scales), _ptr(W_packed),
                                 _ptr(w_scales), _ptr(out), M, N, K, G, _stream(stream)))


def comet_w4ax_gemm_noalloc(A_packed, group_prec_map, a_scales, W_packed, w_scales, out, M: int,
                            N: int, K: int, G: int = G, stream=None) -> None:
    m = _map(group_prec_map, K, G)
    _gemm_room(A_packed, m, a_scales, W_packed, w_scales, M, N, K, G)
    _room(out, 2 * M * N, "out")
    _check(lib().comet_w4ax_gemm_noalloc(_ptr(A_packed), _ptr(m), _ptr(a_scales), _ptr(W_packed),
                                         _ptr(w_scales), _ptr(out), M, N, K, G, _stream(stream)))


def comet_w4ax_gemm_acc(A_packed, group_prec_map, a_scales, W_packed, w_scales, acc, M: int,
                        N: int, K: int, G: int, m0: int, m1: int, n0: int, n1: int,
                        stream=None) -> None:
    m = _map(group_prec_map, K, G)
    _gemm_room(A_packed, m, a_scales, W_packed, w_scales, M, N, K, G)
    if G > 0 and K % G == 0 and m1 > m0 and n1 > n0:
        _room(acc, 4 * (m1 - m0) * (n1 - n0) * (K // G), "acc")
    _check(lib().comet_w4ax_gemm_acc(_ptr(A_packed), _ptr(m), _ptr(a_scales), _ptr(W_packed),
                                     _ptr(w_scales), _ptr(acc), M, N, K, G, m0, m1, n0, n1,
                                     _stream(stream)))


def comet_schedule_query(M: int, N: int, K: int, group_prec_map, num_cus: int = 256,
                         G: int = G) -> dict:
    """Host-only view of the GEMM's tile schedule (no device needed)."""
    m = _map(group_prec_map, K, G)
    L = lib()
    nu, nw, tm, tn = ctypes.c_int(), ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(L.comet_schedule_query(M, N, K, G, _ptr(m), num_cus, None, 0, ctypes.byref(nu), None,
                                  0, ctypes.byref(nw), None, ctypes.byref(tm), ctypes.byref(tn)))
    units = np.zeros((nu.value, 5), np.int32)
    wgb = np.zeros(nw.value + 1, np.int32)
    order = np.zeros(K // G, np.int32)
    _check(L.comet_schedule_query(M, N, K, G, _ptr(m), num_cus, _ptr(units), nu.value,
                                  ctypes.byref(nu), _ptr(wgb), nw.value + 1, ctypes.byref(nw),
                                  _ptr(order), ctypes.byref(tm), ctypes.byref(tn)))
    return {"units": units, "wg_begin": wgb, "order": order, "tile_m": tm.value,
            "tile_n": tn.value, "num_wgs": nw.value}


def comet_gemm_kernel(M: int, N: int, K: int, num_cus: int, G: int = G) -> int:
    """Host-only: the comet_kernel_t that comet_w4ax_gemm runs for this shape."""
    k = lib().comet_gemm_kernel(M, N, K, G, num_cus)
    if k < 0:
        raise CometError(1, lib().comet_last_error().decode())
    return k


KERNEL_NAMES = {0: "skinny", 1: "skinny_shared", 2: "mid", 3: "tile", 4: "stream"}


def comet_build_stamp() -> str:
    return lib().comet_build_stamp().decode()


def comet_last_error() -> str:
    return lib().comet_last_error().decode()


def comet_status_str(status: int) -> str:
    return lib().comet_status_str(status).decode()


def comet_release_caches() -> None:
    lib().comet_release_caches()


# --- allocating conveniences (torch tensors on the current device) ----------------

def quantize_act(X, group_prec_map, perm=None, stream=None):
    """X: float16 [M][K] CUDA tensor -> (A_packed uint8, a_scales float16 [K/G][M]).
    perm: optional int32 [K] CUDA tensor (channel permutation)."""
    import torch

    _tensor(X, "float16", "X")
    M, K = X.shape
    if perm is not None:
        _tensor(perm, "int32", "perm")
        _exact(perm, K, "perm")
    nbytes = comet_act_packed_bytes(group_prec_map, M, K)
    if nbytes == 0:
        raise CometError(1, "invalid map or shape")
    A = torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    sa = torch.empty((K // G, M), dtype=torch.float16, device=X.device)
    comet_fmpq_quantize_act_perm(X, perm, group_prec_map, A, sa, M, K, G, stream)
    return A, sa


def pack_w4(W, perm=None, stream=None):
    """W: float16 [N][K] CUDA tensor -> (W_packed uint8 [N][K/2], w_scales float16 [K/G][N]).
    perm: optional int32 [K] CUDA tensor (the activations' channel permutation)."""
    import torch

    _tensor(W, "float16", "W")
    N, K = W.shape
    if perm is not None:
        _tensor(perm, "int32", "perm")
        _exact(perm, K, "perm")
    Wp = torch.empty((N, K // 2), dtype=torch.uint8, device=W.device)
    sw = torch.empty((K // G, N), dtype=torch.float16, device=W.device)
    comet_pack_w4_perm(W, perm, Wp, sw, N, K, G, stream)
    return Wp, sw


def channel_absmax(X, absmax=None, stream=None):
    """Running per-channel max |X| (float32 [K] CUDA tensor), accumulated into absmax."""
    import torch

    _tensor(X, "float16", "X")
    M, K = X.shape
    if absmax is None:
        absmax = torch.zeros(K, dtype=torch.float32, device=X.device)
    _tensor(absmax, "float32", "absmax")
    _exact(absmax, K, "absmax")
    comet_channel_absmax(X, absmax, M, K, stream)
    return absmax


def plan_channel_perm(absmax, G: int = G, outlier_ratio: float = 8.0, max_frac_8bit: float = 0.2):
    """Host: per-channel maxima (numpy or tensor) -> (perm int32 [K], map uint8 [K/G], n_outliers)."""
    a = np.ascontiguousarray(np.asarray(absmax.cpu() if hasattr(absmax, "cpu") else absmax,
                                        dtype=np.float32).reshape(-1))
    K = a.size
    perm = np.empty(K, np.int32)
    prec = np.empty(max(K // G, 1), np.uint8)
    nout = np.zeros(1, np.int32)
    comet_plan_channel_perm(a, K, G, outlier_ratio, max_frac_8bit, perm, prec, nout)
    return perm, prec[: K // G], int(nout[0])


def kv4_quantize(X, G: int = 128, stream=None):
    """X: float16 [T][C] CUDA tensor -> (codes uint8 [T][C/2], params float16 [T][C/G][2])."""
    import torch

    _tensor(X, "float16", "X")
    T, C = X.shape
    codes = torch.empty((T, C // 2), dtype=torch.uint8, device=X.device)
    params = torch.empty((T, C // G, 2), dtype=torch.float16, device=X.device)
    comet_kv4_quantize(X, codes, params, T, C, G, stream)
    return codes, params


def kv4_dequantize(codes, params, G: int = 128, stream=None):
    import torch

    _tensor(codes, "uint8", "codes")
    _tensor(params, "float16", "params")
    if codes.dim() != 2:
        raise ValueError(f"codes: need [T][C/2], got shape {tuple(codes.shape)}")
    T, C = codes.shape[0], codes.shape[1] * 2
    if C % G:
        raise ValueError(f"C={C} is not a multiple of G={G}")
    _exact(params, T * (C // G) * 2, "params")
    out = torch.empty((T, C), dtype=torch.float16, device=codes.device)
    comet_kv4_dequantize(codes, params, out, T, C, G, stream)
    return out


def _exact(t, numel: int, name: str) -> None:
    if t.numel() != numel:
        raise ValueError(f"{name}: {t.numel()} elements, expected {numel}")


def _gemm_operands(A_packed, a_scales, W_packed, w_scales, group_prec_map=None, M=None, N=None,
                   K=None):
    """Dtype, device and layout of the GEMM operands, and, given the shape,
    their exact sizes (the kernels read M, N and K from the arguments, not
    from the tensors)."""
    _tensor(A_packed, "uint8", "A_packed")
    _tensor(a_scales, "float16", "a_scales")
    _tensor(W_packed, "uint8", "W_packed")
    _tensor(w_scales, "float16", "w_scales")
    if M is None:
        return
    if M < 1 or N < 1 or K < G or K % G:
        raise ValueError(f"M={M}, N={N}, K={K}: need M, N >= 1 and K a positive multiple of {G}")
    m = _map(group_prec_map, K)
    nbytes = comet_act_packed_bytes(m, M, K)
    if nbytes == 0:
        raise ValueError("group_prec_map: entries must be 4 or 8")
    _exact(A_packed, nbytes, "A_packed")
    _exact(a_scales, (K // G) * M, "a_scales")
    _exact(W_packed, N * K // 2, "W_packed")
    _exact(w_scales, (K // G) * N, "w_scales")


def w4ax_gemm(A_packed, group_prec_map, a_scales, W_packed, w_scales, M: int, N: int, K: int,
              out=None, stream=None):
    import torch

    _gemm_operands(A_packed, a_scales, W_packed, w_scales, group_prec_map, M, N, K)
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=A_packed.device)
    _tensor(out, "float16", "out")
    if tuple(out.shape) != (M, N):
        raise ValueError(f"out: shape {tuple(out.shape)}, expected {(M, N)}")
    comet_w4ax_gemm(A_packed, group_prec_map, a_scales, W_packed, w_scales, out, M, N, K, G,
                    stream)
    return out


def w4ax_gemm_swiglu_quant(A_packed, group_prec_map, a_scales, W_packed, w_scales, M: int, N: int,
                           K: int, out_prec_map, stream=None):
    """Fused gate/up GEMM + SwiGLU + quantization for the next layer.
    Returns (out_A_packed uint8, out_a_scales float16 [I/G][M]), I = N / 2."""
    import torch

    _gemm_operands(A_packed, a_scales, W_packed, w_scales, group_prec_map, M, N, K)
    I = N // 2
    nbytes = comet_act_packed_bytes(out_prec_map, M, I)
    if nbytes == 0:
        raise CometError(1, "invalid output map or shape")
    A2 = torch.empty(nbytes, dtype=torch.uint8, device=A_packed.device)
    sa2 = torch.empty((I // G, M), dtype=torch.float16, device=A_packed.device)
    comet_w4ax_gemm_swiglu_quant(A_packed, group_prec_map, a_scales, W_packed, w_scales, M, N, K,
                                 G, out_prec_map, A2, sa2, stream)
    return A2, sa2


def swiglu_quantize(gu, out_prec_map, stream=None):
    """gu: float16 [M][2I] CUDA tensor (256-wide gate/up groups) -> (A_packed, a_scales)."""
    import torch

    _tensor(gu, "float16", "gu")
    M, N = gu.shape
    I = N // 2
    nbytes = comet_act_packed_bytes(out_prec_map, M, I)
    if nbytes == 0:
        raise CometError(1, "invalid output map or shape")
    A2 = torch.empty(nbytes, dtype=torch.uint8, device=gu.device)
    sa2 = torch.empty((I // G, M), dtype=torch.float16, device=gu.device)
    comet_swiglu_quantize(gu, out_prec_map, A2, sa2, M, I, G, stream)
    return A2, sa2


def w4ax_gemm_acc(A_packed, group_prec_map, a_scales, W_packed, w_scales, M: int, N: int, K: int,
                  m0: int, m1: int, n0: int, n1: int, stream=None):
    import torch

    _gemm_operands(A_packed, a_scales, W_packed, w_scales, group_prec_map, M, N, K)
    if not (0 <= m0 < m1 <= M and 0 <= n0 < n1 <= N):
        raise ValueError(f"window [{m0},{m1})x[{n0},{n1}) is empty or outside {M}x{N}")
    acc = torch.empty((m1 - m0, n1 - n0, K // G), dtype=torch.int32, device=A_packed.device)
    comet_w4ax_gemm_acc(A_packed, group_prec_map, a_scales, W_packed, w_scales, acc, M, N, K, G,
                        m0, m1, n0, n1, stream)
    return acc

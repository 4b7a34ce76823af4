"""Seeded synthetic inputs for the W4Ax path (shared by the tests, the smoke
check and the benchmark; holds none of the method's arithmetic).

Generator: counter-based.  For tensor ``tid`` of seed ``seed`` the key is
``mix64(seed * 2**32 + tid)``; element ``i`` draws two 64-bit words
``mix64(key + (2i+1) * GOLDEN)`` and ``mix64(key + (2i+2) * GOLDEN)``, where
``mix64`` is the SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014).  The
top 53 bits of each word give uniforms u1, u2 in [0, 1); the Box-Muller
transform z = sqrt(-2 ln(1 - u1)) cos(2 pi u2) in fp64 gives a standard normal,
which is scaled and rounded to fp16 (round to nearest even).  The result
depends only on (seed, tid, i), not on chunking or thread count.

Workload recipe (synthetic LLaMA-shaped layers):
  * activations X [M][K] ~ N(0, 1); the channels of every 8-bit block are
    multiplied by 50 before rounding (outlier channels);
  * weights W [N][K] ~ N(0, 0.02^2);
  * block precision map: a contiguous run of 8-bit blocks starting at block
    floor(3 * NG / 8), or a seeded random subset of blocks;
  * calibration workloads (channel permutation): ``n_out`` outlier channels
    scattered over all K channels (a seeded subset), multiplied by 50; with
    n_out = 0.5% of K this matches "a small cluster, usually under 1% of the
    features" for LLaMA-scale models;
  * KV rows [T][C] (C = KV heads x head_dim) ~ N(0, 1) with per-channel
    multipliers drawn from 2^U(0, 3), so channels differ in range.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

TID_X = 1
TID_W = 2
TID_MAP = 3
TID_OUTLIER = 4
TID_CAL = 5
TID_KV = 6
TID_KV_SCALE = 7

_CHUNK = 1 << 22


def mix64(z: np.ndarray) -> np.ndarray:
    z = z.copy()
    z ^= z >> np.uint64(30)
    z *= _M1
    z ^= z >> np.uint64(27)
    z *= _M2
    z ^= z >> np.uint64(31)
    return z


def _key(seed: int, tid: int) -> np.uint64:
    return mix64(np.array([(seed << 32) + tid], dtype=np.uint64))[0]


def _normal_chunk(key: np.uint64, start: int, count: int) -> np.ndarray:
    i = np.arange(start, start + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        w1 = mix64(key + (np.uint64(2) * i + np.uint64(1)) * GOLDEN)
        w2 = mix64(key + (np.uint64(2) * i + np.uint64(2)) * GOLDEN)
    u1 = (w1 >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)
    u2 = (w2 >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)
    return np.sqrt(-2.0 * np.log1p(-u1)) * np.cos(2.0 * np.pi * u2)


def _threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal_fp16(seed: int, tid: int, shape, std: float = 1.0, col_scale=None) -> np.ndarray:
    """fp16 bit patterns (uint16) of N(0, std^2) draws; ``col_scale`` (fp64 vector
    over the last axis) multiplies columns before rounding."""
    shape = tuple(int(s) for s in shape)
    total = int(np.prod(shape)) if shape else 1
    out = np.empty(total, dtype=np.float16)
    key = _key(seed, tid)
    ncol = shape[-1] if shape else 1
    cs = None if col_scale is None else np.asarray(col_scale, dtype=np.float64)

    def work(start):
        cnt = min(_CHUNK, total - start)
        z = _normal_chunk(key, start, cnt) * std
        if cs is not None:
            z *= cs[(np.arange(start, start + cnt) % ncol)]
        out[start:start + cnt] = z.astype(np.float16)

    starts = list(range(0, total, _CHUNK))
    if len(starts) == 1:
        work(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, starts))
    return out.view(np.uint16).reshape(shape)


def prec_map(NG: int, n8: int, placement: str = "contiguous", seed: int = 0,
             start: int | None = None) -> np.ndarray:
    """uint8 [NG] of 4/8 with ``n8`` 8-bit blocks.

    contiguous: a run starting at ``start`` (default floor(3 NG / 8)), wrapped at NG;
    random: a seeded subset drawn by a Fisher-Yates shuffle on counter-based words.
    """
    m = np.full(NG, 4, dtype=np.uint8)
    n8 = int(n8)
    if n8 <= 0:
        return m
    if n8 > NG:
        raise ValueError("more 8-bit blocks than blocks")
    if placement == "contiguous":
        s = (3 * NG) // 8 if start is None else int(start)
        for j in range(n8):
            m[(s + j) % NG] = 8
    elif placement == "random":
        words = _words(seed, TID_MAP, NG)
        idx = list(range(NG))
        for i in range(NG - 1, 0, -1):
            j = int(words[i] % np.uint64(i + 1))
            idx[i], idx[j] = idx[j], idx[i]
        m[np.array(idx[:n8])] = 8
    else:
        raise ValueError(placement)
    return m


def _words(seed: int, tid: int, n: int) -> np.ndarray:
    key = _key(seed, tid)
    with np.errstate(over="ignore"):
        return mix64(key + (np.arange(n, dtype=np.uint64) + np.uint64(1)) * GOLDEN)


def outlier_channels(K: int, n_out: int, seed: int = 0) -> np.ndarray:
    """Sorted int64 array of ``n_out`` distinct channels, a seeded Fisher-Yates subset."""
    words = _words(seed, TID_OUTLIER, K)
    idx = list(range(K))
    for i in range(K - 1, 0, -1):
        j = int(words[i] % np.uint64(i + 1))
        idx[i], idx[j] = idx[j], idx[i]
    return np.sort(np.array(idx[:n_out], dtype=np.int64))


def channel_scale(K: int, channels, factor: float = 50.0) -> np.ndarray:
    """Per-channel multiplier: ``factor`` on ``channels``, else 1."""
    cs = np.ones(K, dtype=np.float64)
    cs[np.asarray(channels, dtype=np.int64)] = factor
    return cs


def calibration_activations(seed: int, M: int, K: int, channels, tid: int = TID_CAL,
                            factor: float = 50.0) -> np.ndarray:
    """Activations with outliers on the given (scattered) channels."""
    return normal_fp16(seed, tid, (M, K), 1.0, channel_scale(K, channels, factor))


def kv_rows(seed: int, T: int, C: int) -> np.ndarray:
    """K or V rows [T][C] with per-channel ranges 2^U(0, 3)."""
    w = _words(seed, TID_KV_SCALE, C)
    u = (w >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)
    return normal_fp16(seed, TID_KV, (T, C), 1.0, np.exp2(3.0 * u))


def outlier_scale(prec: np.ndarray, G: int = 128, factor: float = 50.0) -> np.ndarray:
    """Per-channel multiplier: ``factor`` on the channels of 8-bit blocks, else 1."""
    return np.repeat(np.where(np.asarray(prec) == 8, factor, 1.0), G)


def activations(seed: int, M: int, K: int, prec: np.ndarray, G: int = 128) -> np.ndarray:
    return normal_fp16(seed, TID_X, (M, K), 1.0, outlier_scale(prec, G))


def weights(seed: int, N: int, K: int) -> np.ndarray:
    return normal_fp16(seed, TID_W, (N, K), 0.02)


# Layer shapes of the synthetic workloads (tokens M; K -> N).
LLAMA3_8B = {"qkv": (4096, 6144), "o": (4096, 4096), "gate_up": (4096, 28672),
             "down": (14336, 4096)}
LLAMA3_70B = {"qkv": (8192, 10240), "o": (8192, 8192), "gate_up": (8192, 57344),
              "down": (28672, 8192)}

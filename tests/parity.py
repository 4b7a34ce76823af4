"""Shared helpers of the GPU parity tests and the benchmark's parity checks.

The comparison rule for the fp16 GEMM output against the fp64 oracle is
elementwise: |y - ref| <= 2e-3 * max(|ref|, 0.01 * rms(ref)).  The floor of 1%
of the output RMS keeps outputs that cancel to nearly zero from failing on
rounding noise; the normwise error is reported next to it.
"""
from __future__ import annotations

import numpy as np

REL_TOL = 2e-3
FLOOR = 0.01


def block_offsets(prec, M: int, G: int = 128):
    """Byte offset of every block of a block-major A_packed, and its row pitch."""
    pitch = np.where(np.asarray(prec) == 8, G, G // 2).astype(np.int64)
    base = np.concatenate([[0], np.cumsum(pitch * M)[:-1]])
    return base, pitch


def act_rows(A_packed: np.ndarray, prec, M: int, rows, G: int = 128) -> np.ndarray:
    """Concatenated packed bytes of the given rows, block by block (the bytes
    an A_packed built from those rows alone would hold)."""
    base, pitch = block_offsets(prec, M, G)
    parts = []
    for g in range(len(prec)):
        for_rows = [A_packed[base[g] + r * pitch[g]: base[g] + (r + 1) * pitch[g]] for r in rows]
        parts.append(np.concatenate(for_rows))
    return np.concatenate(parts)


def out_errors(y16: np.ndarray, ref: np.ndarray):
    y = y16.astype(np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    denom = np.maximum(np.abs(ref), FLOOR * rms)
    denom[denom == 0] = 1.0
    rel = np.abs(y - ref) / denom
    norm = float(np.linalg.norm(y - ref) / max(np.linalg.norm(ref), 1e-300))
    return float(rel.max()) if rel.size else 0.0, norm


def assert_out_close(y16: np.ndarray, ref: np.ndarray, what: str = ""):
    assert np.all(np.isfinite(y16.astype(np.float32))), f"{what}: non-finite output"
    mx, norm = out_errors(y16, ref)
    assert mx <= REL_TOL, f"{what}: max elementwise rel err {mx:.3e} > {REL_TOL} (normwise {norm:.2e})"
    return mx, norm

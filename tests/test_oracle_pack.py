"""Pins for the oracle's byte encodings.

The storage contract is chosen so that two masks and one 4-bit rotation turn a
packed dword into OCP FP8-E4M3 bytes whose values are the codes times 2^-9
(sign-magnitude subnormals).  That property is what the GPU kernels rely on, so
it is the pin: the packed bytes are decoded here with PyTorch's own
float8_e4m3fn conversion (an independent library routine), not by re-typing
the oracle's bit layout.
"""
import numpy as np
import pytest
import torch

import oracle

MASK = np.uint32(0x87878787)


def e4m3(words_u32: np.ndarray) -> np.ndarray:
    """Values of the four E4M3 bytes of each little-endian dword, times 2^9."""
    b = torch.from_numpy(np.ascontiguousarray(words_u32).view(np.uint8).copy())
    return (b.view(torch.float8_e4m3fn).float() * 512.0).numpy().reshape(-1, 4)


def decode4(chunk: np.ndarray) -> np.ndarray:
    w = chunk.view("<u4")
    lo = e4m3(w & MASK)                                      # codes 8j+0 .. 8j+3
    rot = ((w >> np.uint32(4)) | (w << np.uint32(28))).astype(np.uint32)
    hi = e4m3(rot & MASK)                                    # codes 8j+4 .. 8j+7
    return np.concatenate([lo, hi], axis=1).reshape(-1)


def decode8(chunk: np.ndarray) -> np.ndarray:
    w = chunk.view("<u4")
    low3 = e4m3(w & MASK)                                    # sign * (m mod 8)
    high4 = e4m3(((w >> np.uint32(3)) & np.uint32(0x0F0F0F0F)) | (w & np.uint32(0x80808080)))
    return (8 * high4 + low3).reshape(-1)                   # sign * m


def test_encode4_decodes_to_codes_via_e4m3():
    rng = np.random.default_rng(1)
    for _ in range(200):
        q = rng.integers(-7, 8, 128).astype(np.int8)
        out = oracle.encode4(q)
        assert out.size == 64
        assert np.array_equal(decode4(out), q.astype(np.float32))


def test_encode4_extremes_and_zero():
    for q in (np.full(128, 7), np.full(128, -7), np.zeros(128),
              np.tile([7, -7, 0, 1, -1, 3, -3, 6], 16)):
        q = q.astype(np.int8)
        assert np.array_equal(decode4(oracle.encode4(q)), q.astype(np.float32))
    # zero codes encode as zero bytes (no negative zero)
    assert not oracle.encode4(np.zeros(128, np.int8)).any()


def test_encode8_decodes_to_codes_via_e4m3():
    rng = np.random.default_rng(2)
    for _ in range(200):
        q = rng.integers(-127, 128, 128).astype(np.int8)
        assert np.array_equal(decode8(oracle.encode8(q)), q.astype(np.float32))
    q = np.arange(-127, 128, dtype=np.int64)
    q = np.concatenate([q, q[:1]]).astype(np.int8)
    assert np.array_equal(decode8(oracle.encode8(q)), q.astype(np.float32))


def test_pack_act_block_major_layout():
    M, K, G = 3, 512, 128
    prec = np.array([4, 8, 8, 4], np.uint8)
    rng = np.random.default_rng(4)
    qa = np.where(np.repeat(prec, G)[None, :] == 8,
                  rng.integers(-127, 128, (M, K)), rng.integers(-7, 8, (M, K))).astype(np.int8)
    buf = oracle.pack_act(qa, prec, G)
    assert buf.size == M * (64 + 128 + 128 + 64) == oracle.act_packed_bytes(prec, M, K, G)
    off = 0
    for g in range(4):
        B = 64 if prec[g] == 4 else 128
        for m in range(M):
            chunk = buf[off + m * B: off + (m + 1) * B]
            dec = decode4(chunk) if prec[g] == 4 else decode8(chunk)
            assert np.array_equal(dec, qa[m, g * G:(g + 1) * G].astype(np.float32)), (g, m)
        off += M * B


def test_pack_weight_panel_layout():
    # 16-row panels: row n, block g at ((n // 16 * NG + g) * 16 + n % 16) * 64
    N, K, G = 48, 384, 128
    NG = K // G
    rng = np.random.default_rng(6)
    qw = rng.integers(-7, 8, (N, K)).astype(np.int8)
    flat = oracle.pack_weight(qw, G).reshape(-1)
    assert flat.size == N * K // 2
    seen = np.zeros(flat.size, bool)
    for n in range(N):
        for g in range(NG):
            off = ((n // 16 * NG + g) * 16 + n % 16) * 64
            dec = decode4(flat[off:off + 64].copy())
            assert np.array_equal(dec, qw[n, g * G:(g + 1) * G].astype(np.float32))
            seen[off:off + 64] = True
    assert seen.all()  # every byte belongs to exactly one (row, block)
    # one panel's block is one contiguous run of 16 rows
    run = flat[(1 * NG + 2) * 1024:(1 * NG + 2) * 1024 + 1024].reshape(16, 64)
    for r in range(16):
        assert np.array_equal(decode4(run[r].copy()), qw[16 + r, 2 * G:3 * G].astype(np.float32))


def test_pack_weight_rejects_partial_panel():
    with pytest.raises(ValueError):
        oracle.pack_weight(np.zeros((24, 256), np.int8), 128)

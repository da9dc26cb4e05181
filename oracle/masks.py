"""Packed mask layouts, written out bit by bit (test infrastructure only).

The paper keeps the mask as a dense boolean tensor (``weight != 0``, Appendix A
listing; the mask M of Section 2.1).  The library stores it packed instead;
the layouts are this repository's own definition:

BITMAP  row i uses ceil(C/32) uint32 words; element (i, j) is bit j % 32
        (least significant first) of word i*ceil(C/32) + j // 32.  Padding
        bits past C are 0.
2:4     needs C % 4 == 0.  Group g of row i is columns 4g .. 4g+3 and must keep
        exactly two positions p0 < p1; its code p0 | p1 << 2 is the nibble at
        bits 4*(g % 8) of word i*ceil(C/32) + g // 8.  Unused nibbles are 0.
"""
from __future__ import annotations

import numpy as np

BITMAP = "bitmap"
TWO_FOUR = "2:4"


def words_per_row(C: int) -> int:
    return (C + 31) // 32


def pack_bitmap(M: np.ndarray) -> np.ndarray:
    M = np.asarray(M).astype(bool)
    R, C = M.shape
    wpr = words_per_row(C)
    out = np.zeros((R, wpr), dtype=np.uint32)
    for j in range(C):  # one column (= one bit position) at a time
        w, b = divmod(j, 32)
        out[:, w] |= M[:, j].astype(np.uint32) << np.uint32(b)
    return out.reshape(-1)


def unpack_bitmap(words: np.ndarray, R: int, C: int) -> np.ndarray:
    wpr = words_per_row(C)
    words = np.asarray(words, dtype=np.uint32).reshape(R, wpr)
    M = np.zeros((R, C), dtype=np.uint8)
    for j in range(C):
        w, b = divmod(j, 32)
        M[:, j] = (words[:, w] >> np.uint32(b)) & np.uint32(1)
    return M


def first_bad_group_2_4(M: np.ndarray) -> int:
    """Linear index i*(C/4)+g of the first group not keeping exactly 2, or -1."""
    M = np.asarray(M).astype(np.uint8)
    R, C = M.shape
    counts = M.reshape(R, C // 4, 4).sum(axis=2).reshape(-1)
    bad = np.nonzero(counts != 2)[0]
    return int(bad[0]) if bad.size else -1


def pack_2_4(M: np.ndarray) -> np.ndarray:
    M = np.asarray(M).astype(np.uint8)
    R, C = M.shape
    if C % 4:
        raise ValueError("2:4 layout needs C % 4 == 0")
    bad = first_bad_group_2_4(M)
    if bad >= 0:
        raise ValueError(f"group {bad} (row {bad // (C // 4)}) does not keep exactly 2 of 4")
    wpr = words_per_row(C)
    out = np.zeros((R, wpr), dtype=np.uint32)
    g4 = M.reshape(R, C // 4, 4)
    # p0 = first kept position, p1 = second kept position, found by scanning
    # the four positions in order.
    p0 = np.full((R, C // 4), -1, dtype=np.int64)
    p1 = np.full((R, C // 4), -1, dtype=np.int64)
    for p in range(4):
        kept = g4[:, :, p] == 1
        take0 = kept & (p0 < 0)
        take1 = kept & (p0 >= 0) & ~take0
        p0 = np.where(take0, p, p0)
        p1 = np.where(take1, p, p1)
    code = (p0 | (p1 << 2)).astype(np.uint32)
    for g in range(C // 4):
        w, n = divmod(g, 8)
        out[:, w] |= code[:, g] << np.uint32(4 * n)
    return out.reshape(-1)


def unpack_2_4(words: np.ndarray, R: int, C: int) -> np.ndarray:
    wpr = words_per_row(C)
    words = np.asarray(words, dtype=np.uint32).reshape(R, wpr)
    M = np.zeros((R, C), dtype=np.uint8)
    for g in range(C // 4):
        w, n = divmod(g, 8)
        code = (words[:, w] >> np.uint32(4 * n)) & np.uint32(0xF)
        p0 = (code & 3).astype(np.int64)
        p1 = ((code >> 2) & 3).astype(np.int64)
        rows = np.arange(R)
        M[rows, 4 * g + p0] = 1
        M[rows, 4 * g + p1] = 1
    return M


def pack(M: np.ndarray, fmt: str) -> np.ndarray:
    return pack_bitmap(M) if fmt == BITMAP else pack_2_4(M)


def unpack(words: np.ndarray, R: int, C: int, fmt: str) -> np.ndarray:
    return unpack_bitmap(words, R, C) if fmt == BITMAP else unpack_2_4(words, R, C)

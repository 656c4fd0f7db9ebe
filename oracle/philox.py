"""Counter-based random numbers for dropout: Philox4x32-10, in plain NumPy.

Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
easy as 1, 2, 3", SC 2011) maps a 128-bit counter (c0, c1, c2, c3) and a
64-bit key (k0, k1) to four 32-bit words by ten rounds of

    (c0, c1, c2, c3) <- (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0))

with M0 = 0xD2511F53, M1 = 0xCD9E8D57, the key advanced by the Weyl
constants (0x9E3779B9, 0xBB67AE85) after every round.  hi/lo are the upper
and lower 32 bits of the 64-bit product.

Dropout (the paper drops each layer's input after the boundary receive, with
one mask for the forward and the backward; its appendix on implementation
details): element (r, c) of a layer input with `cols` columns, r in the
partition's local row numbering (inner rows, then boundary rows), has index
q = r * cols + c.  Word q mod 4 of Philox(counter = (q div 4 low 32 bits,
q div 4 high 32 bits, layer, iteration), key = (seed, partition)) decides it:
the element is dropped if the word is below floor(p * 2^32), else kept and
scaled by 1 / (1 - p).

Test infrastructure only (see the package header).  Pinned by the published
known-answer vectors of Philox4x32-10 (tests).
"""
from __future__ import annotations

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10(counter: np.ndarray, key) -> np.ndarray:
    """counter: uint64 array [..., 4] of 32-bit values; key: (k0, k1).  Returns [..., 4] uint64."""
    c = [np.asarray(counter[..., i], dtype=np.uint64) & MASK32 for i in range(4)]
    k0, k1 = int(key[0]) & MASK32, int(key[1]) & MASK32
    for _ in range(10):
        p0 = np.uint64(M0) * c[0]               # < 2^64: both factors are below 2^32
        p1 = np.uint64(M1) * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & np.uint64(MASK32)
        hi1, lo1 = p1 >> np.uint64(32), p1 & np.uint64(MASK32)
        c = [hi1 ^ c[1] ^ np.uint64(k0), lo1, hi0 ^ c[3] ^ np.uint64(k1), lo0]
        k0 = (k0 + W0) & MASK32
        k1 = (k1 + W1) & MASK32
    return np.stack(c, axis=-1)


def drop_threshold(p: float) -> int:
    """Words below this value drop their element: floor(p * 2^32), at most 2^32 - 1."""
    return min(int(np.floor(p * 4294967296.0)), MASK32)


def dropout_mask(rows: int, cols: int, p: float, seed: int, part: int, layer: int, iteration: int) -> np.ndarray:
    """float64 [rows, cols]: 0 for dropped elements, 1 / (1 - p) for kept ones (all ones when p = 0)."""
    return dropout_mask_rows(np.arange(rows), cols, p, seed, part, layer, iteration)


def dropout_mask_rows(row_ids, cols: int, p: float, seed: int, part: int, layer: int, iteration: int) -> np.ndarray:
    """The rows `row_ids` (local row numbers) of the mask above."""
    row_ids = np.asarray(row_ids, dtype=np.uint64)
    if p <= 0.0 or len(row_ids) * cols == 0:
        return np.ones((len(row_ids), cols))
    q = (row_ids[:, None] * np.uint64(cols) + np.arange(cols, dtype=np.uint64)[None, :]).reshape(-1)
    g = q >> np.uint64(2)
    ctr = np.stack([g & np.uint64(MASK32), g >> np.uint64(32),
                    np.full_like(g, layer), np.full_like(g, iteration)], axis=-1)
    words = philox4x32_10(ctr, (seed, part))
    u = words[np.arange(len(q)), (q & np.uint64(3)).astype(np.int64)]
    keep = u >= np.uint64(drop_threshold(p))
    return np.where(keep, 1.0 / (1.0 - p), 0.0).reshape(len(row_ids), cols)

"""Counter-based Gaussian noise for the SDE step (Sec. 3.1: eps ~ N(0, I)), float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The noise is drawn from Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011), written here from that
definition: a 4 x 32-bit counter and a 2 x 32-bit key; each of the ten rounds
multiplies counter words 0 and 2 by the constants 0xD2511F53 and 0xCD9E8D57
into 64-bit products and recombines high and low halves with the other two
words and the round key, and the key advances by the Weyl constants
(0x9E3779B9, 0xBB67AE85) between rounds.

Layout (a reading: the paper only says eps is standard normal): element d of
sample b in SDE step `step` takes word d % 4 of the Philox block with counter
(n mod 2^32, n div 2^32, b, step), n = d div 4, key (seed mod 2^32, seed div
2^32).  Words (w0, w1) and (w2, w3) each give two normals by the Box-Muller
transform with u = (w + 1/2) 2^-32: r = sqrt(-2 ln u0), z0 = r cos(2 pi u1),
z1 = r sin(2 pi u1).
"""
from __future__ import annotations

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK = 0xFFFFFFFF


def philox4x32_10(ctr: np.ndarray, key) -> np.ndarray:
    """ctr: uint array [..., 4]; key: (k0, k1).  Returns uint32 [..., 4]."""
    c = [np.asarray(ctr[..., i], dtype=np.uint64) for i in range(4)]
    k0, k1 = np.uint64(int(key[0]) & MASK), np.uint64(int(key[1]) & MASK)
    m0, m1, mask = np.uint64(M0), np.uint64(M1), np.uint64(MASK)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + np.uint64(W0)) & mask
            k1 = (k1 + np.uint64(W1)) & mask
        p0 = m0 * c[0]            # < 2^64: exact in uint64
        p1 = m1 * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return np.stack([x.astype(np.uint32) for x in c], axis=-1)


def box_muller(w: np.ndarray) -> np.ndarray:
    """uint32 words [..., 4] -> four standard normals [..., 4] (float64)."""
    u = (w.astype(np.float64) + 0.5) * 2.0 ** -32
    r0 = np.sqrt(-2.0 * np.log(u[..., 0]))
    r1 = np.sqrt(-2.0 * np.log(u[..., 2]))
    a0, a1 = 2.0 * np.pi * u[..., 1], 2.0 * np.pi * u[..., 3]
    return np.stack([r0 * np.cos(a0), r0 * np.sin(a0), r1 * np.cos(a1), r1 * np.sin(a1)], axis=-1)


def sde_noise(B: int, D: int, seed: int, step: int) -> np.ndarray:
    """eps [B, D] of one SDE step under the layout in the module docstring."""
    nb = (D + 3) // 4
    n = np.arange(nb, dtype=np.uint64)
    out = np.empty((B, nb * 4), dtype=np.float64)
    key = (seed & MASK, (seed >> 32) & MASK)
    for b in range(B):
        ctr = np.stack([n & np.uint64(MASK), n >> np.uint64(32), np.full(nb, b, dtype=np.uint64),
                        np.full(nb, step, dtype=np.uint64)], axis=-1)
        out[b] = box_muller(philox4x32_10(ctr, key)).reshape(-1)
    return out[:, :D]

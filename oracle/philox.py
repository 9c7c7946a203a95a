"""Philox4x32-10 random streams (Salmon, Moraes, Dror, Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC'11), written from the published round function.

The paper only says the updater samples uniform batches from the shared replay
pool (Section 3.3.2); the generator is this implementation's choice. Every draw is
a pure function of (seed, counter), so the GPU and this oracle reach the same
integers.

Counter convention for element i of a stream:
    counter = (i >> 2, step, purpose, tensor_id), key = (seed lo32, seed hi32),
    output word i & 3.
Purposes: INIT 0 (step 0), IDX 1, NOISE_TGT 2, NOISE_POL 3.
"""
from __future__ import annotations

import numpy as np

MASK = np.uint64(0xFFFFFFFF)
MUL0 = np.uint64(0xD2511F53)
MUL1 = np.uint64(0xCD9E8D57)
WEYL0 = np.uint64(0x9E3779B9)
WEYL1 = np.uint64(0xBB67AE85)

PURPOSE_INIT = 0
PURPOSE_IDX = 1
PURPOSE_NOISE_TGT = 2
PURPOSE_NOISE_POL = 3
PURPOSE_ACT = 4          # sampler actions: step word = the caller's counter


def block(c0, c1, c2, c3, k0, k1, rounds: int = 10):
    """Philox4x32 with `rounds` rounds on uint32 values held in uint64 arrays.

    One round: the two 32x32->64 products M0*c0 and M1*c2 are split into hi/lo
    halves and the output is (hi1^c1^k0, lo1, hi0^c3^k1, lo0); the key is advanced
    by the two Weyl constants between rounds.
    """
    c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) & MASK for x in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=np.uint64) & MASK
    k1 = np.asarray(k1, dtype=np.uint64) & MASK
    for r in range(rounds):
        if r:
            k0 = (k0 + WEYL0) & MASK
            k1 = (k1 + WEYL1) & MASK
        p0 = MUL0 * c0
        p1 = MUL1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def words(seed: int, n: int, step: int, purpose: int, tensor_id: int = 0) -> np.ndarray:
    """The first n 32-bit words of stream (seed, step, purpose, tensor_id), as uint64."""
    nb = (n + 3) // 4
    i = np.arange(nb, dtype=np.uint64)
    k0 = np.uint64(seed & 0xFFFFFFFF)
    k1 = np.uint64((seed >> 32) & 0xFFFFFFFF)
    w = block(i, np.uint64(step), np.uint64(purpose), np.uint64(tensor_id), k0, k1)
    return np.stack(w, axis=1).reshape(-1)[:n]


def indices(seed: int, step: int, batch: int, size: int) -> np.ndarray:
    """Replay rows for one step: idx[b] = floor(w_b * size / 2^32) (multiply-high).

    Sampling is uniform with replacement over the `size` valid rows.
    """
    w = words(seed, batch, step, PURPOSE_IDX)
    return ((w * np.uint64(size)) >> np.uint64(32)).astype(np.int64)


def normals(seed: int, step: int, purpose: int, n: int) -> np.ndarray:
    """n standard normal deviates by the Box-Muller transform (float64).

    Words (0,1) of a block give lanes 0 and 1, words (2,3) give lanes 2 and 3:
    u1 = ((w_a >> 8) + 1) / 2^24 in (0, 1], u2 = (w_b >> 8) / 2^24 in [0, 1),
    R = sqrt(-2 ln u1), even lane R cos(2 pi u2), odd lane R sin(2 pi u2).
    """
    nb = (n + 3) // 4
    w = words(seed, 4 * nb, step, purpose).reshape(nb, 4)
    out = np.empty((nb, 4), dtype=np.float64)
    for pair in (0, 1):
        wa, wb = w[:, 2 * pair], w[:, 2 * pair + 1]
        u1 = ((wa >> np.uint64(8)).astype(np.float64) + 1.0) * 2.0 ** -24
        u2 = (wb >> np.uint64(8)).astype(np.float64) * 2.0 ** -24
        rad = np.sqrt(-2.0 * np.log(u1))
        out[:, 2 * pair] = rad * np.cos(2.0 * np.pi * u2)
        out[:, 2 * pair + 1] = rad * np.sin(2.0 * np.pi * u2)
    return out.reshape(-1)[:n]


def init_uniform(seed: int, tensor_id: int, n: int, fan_in: int) -> np.ndarray:
    """PyTorch-default fan-in init U(-k, k), k = 1/sqrt(fan_in), as float32 values.

    k is rounded to float32 first; u = (w >> 8) / 2^24; value = fl32((2u - 1) * k)
    with the product formed in double.
    """
    k = np.float64(np.float32(1.0 / np.sqrt(np.float64(fan_in))))
    w = words(seed, n, 0, PURPOSE_INIT, tensor_id)
    u = (w >> np.uint64(8)).astype(np.float64) * 2.0 ** -24
    return ((2.0 * u - 1.0) * k).astype(np.float32)

"""Philox4x32-10 and the dropout masks drawn from it (test infrastructure only).

Philox4x32-10 is the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC 2011): ten rounds over a
128-bit counter (c0, c1, c2, c3) under a 64-bit key (k0, k1).  One round maps

    (c0, c1, c2, c3) -> (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0))

with M0 = 0xD2511F53, M1 = 0xCD9E8D57 (hi/lo: upper/lower 32 bits of the 64-bit
product), and the key advances by the Weyl constants (0x9E3779B9, 0xBB67AE85)
between rounds.  Written here from that definition, in plain NumPy uint32/uint64
arithmetic, element-wise over arrays.

Dropout (Section 2.1: a rate per convolution input and for the softmax layer's
input; the reading for sparse layers is in ``dropout_keep``).
"""

import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint32(0x9E3779B9)
W1 = np.uint32(0xBB67AE85)
MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """The four output words for counters (c0..c3) and key (k0, k1), broadcast element-wise."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64).astype(np.uint32) for c in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=np.uint64).astype(np.uint32)
    k1 = np.asarray(k1, dtype=np.uint64).astype(np.uint32)
    with np.errstate(over="ignore"):
        for _ in range(10):
            p0 = M0 * c0.astype(np.uint64)
            p1 = M1 * c2.astype(np.uint64)
            hi0, lo0 = (p0 >> np.uint64(32)).astype(np.uint32), (p0 & MASK32).astype(np.uint32)
            hi1, lo1 = (p1 >> np.uint64(32)).astype(np.uint32), (p1 & MASK32).astype(np.uint32)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
            k0 = k0 + W0
            k1 = k1 + W1
    return c0, c1, c2, c3


def drop_threshold(p: float) -> int:
    """A 32-bit word u keeps its element when u >= floor(p * 2**32) (probability 1 - p)."""
    if not 0.0 <= p < 1.0:
        raise ValueError("dropout rate must be in [0, 1)")
    return int(np.floor(p * 2.0 ** 32))


def drop_scale(p: float) -> float:
    """Inverted dropout: kept values are multiplied by 1/(1 - p), as a float32 value."""
    return float(np.float32(1.0 / (1.0 - p)))


def dropout_keep(keys, channels: int, layer: int, p: float, seed: int) -> np.ndarray:
    """Keep mask [len(keys), channels] for the rows with the given 32-bit keys.

    Element (key q, channel c) of dropout layer ``layer`` is kept when word
    ``c % 4`` of Philox4x32-10 at counter (q, c // 4, layer, 0) under key
    (seed mod 2**32, seed // 2**32) is at least ``drop_threshold(p)``.  Keys
    are the layer's packed site keys (b*S + y)*S + x (one per active site), or
    the sample index for the softmax layer's input.
    """
    keys = np.asarray(keys, dtype=np.int64).reshape(-1, 1)
    c = np.arange(channels, dtype=np.int64).reshape(1, -1)
    words = philox4x32_10(keys & 0xFFFFFFFF, c // 4, np.full_like(c, layer), np.zeros_like(c),
                          seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    w = np.stack(words, axis=-1)  # [n, C, 4]
    pick = np.take_along_axis(w, (c % 4)[..., None].repeat(w.shape[0], axis=0), axis=-1)[..., 0]
    return pick >= np.uint32(drop_threshold(p)) if drop_threshold(p) > 0 else np.ones(pick.shape, bool)

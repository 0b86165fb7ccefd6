"""Philox4x32-10 counter-based generator and the Gaussian draws built on it.

Test infrastructure only (see ``oracle/__init__.py``).

Philox4x32-10 follows its published definition (Salmon, Moraes, Dror, Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC'11): a 4-word counter and a
2-word key; each of ten rounds multiplies words 0 and 2 by fixed 32-bit
constants, keeps the high and low halves of both 64-bit products, permutes the
words and xors the high halves with the other two counter words and the key;
the key is bumped by two Weyl constants between rounds.

How the training step keys it (the paper only says Gaussian noise with
standard deviation sigma is added to the published embedding, Appendix
"Differential Privacy Protocol" and Assumption 5; the keying below is this
build's reading):

* key     = (seed mod 2**32, seed >> 32)
* counter = (step, global row id, column >> 2, tag), tag 0 for the published
  embedding, 1 for the returned gradient; ``step`` is the batch-group id of
  the message.
* the four output words feed two Box-Muller pairs: (w0, w1) gives columns
  4q and 4q+1, (w2, w3) gives columns 4q+2 and 4q+3.
* a word w maps to the uniform ((w >> 8) + 1) * 2**-24 in (0, 1], exact in
  both single and double precision.
* Box-Muller: r = sqrt(-2 ln u_a); n0 = r cos(2 pi u_b), n1 = r sin(2 pi u_b).
"""
from __future__ import annotations

import numpy as np

MUL0 = 0xD2511F53
MUL1 = 0xCD9E8D57
WEYL0 = 0x9E3779B9
WEYL1 = 0xBB67AE85
MASK = 0xFFFFFFFF

TAG_EMB = 0
TAG_GRAD = 1


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10.  Inputs are integer arrays (broadcastable)
    holding unsigned 32-bit values; returns four uint32 arrays."""
    c0, c1, c2, c3, k0, k1 = (np.asarray(v, dtype=np.uint64) & MASK
                              for v in (c0, c1, c2, c3, k0, k1))
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(c0, c1, c2, c3, k0, k1)
    for r in range(10):
        if r:
            k0 = (k0 + WEYL0) & MASK
            k1 = (k1 + WEYL1) & MASK
        p0 = np.uint64(MUL0) * c0          # < 2**64: exact in uint64
        p1 = np.uint64(MUL1) * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
    return tuple(v.astype(np.uint32) for v in (c0, c1, c2, c3))


def word_to_uniform(w) -> np.ndarray:
    """uint32 word -> uniform in (0, 1] as float64: ((w >> 8) + 1) / 2**24."""
    w = np.asarray(w, dtype=np.uint64)
    return ((w >> np.uint64(8)) + np.uint64(1)).astype(np.float64) * (2.0 ** -24)


def box_muller(ua, ub):
    """Two independent standard normals from two uniforms in (0, 1]."""
    r = np.sqrt(-2.0 * np.log(ua))
    ang = 2.0 * np.pi * ub
    return r * np.cos(ang), r * np.sin(ang)


def gaussian(seed: int, step: int, rows, n_cols: int, tag: int) -> np.ndarray:
    """Standard normals xi[i, j] for global row ids ``rows`` and columns
    0..n_cols-1 of message ``(step, tag)``; float64 [len(rows), n_cols]."""
    rows = np.asarray(rows, dtype=np.uint64)[:, None]
    cols = np.arange(n_cols, dtype=np.uint64)[None, :]
    k0, k1 = seed & MASK, (seed >> 32) & MASK
    w0, w1, w2, w3 = philox4x32_10(step & MASK, rows, cols >> np.uint64(2), tag, k0, k1)
    sel = (cols & np.uint64(3)).astype(np.int64)
    first_pair = sel < 2
    ua = word_to_uniform(np.where(first_pair, w0, w2))
    ub = word_to_uniform(np.where(first_pair, w1, w3))
    n0, n1 = box_muller(ua, ub)
    return np.where((sel & 1) == 0, n0, n1)

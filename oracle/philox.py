"""Philox4x64-10 and the integer range map (oracle side).

The paper states only that the training buffer is seeded for reproducibility
(Sec. 3.1, framework description) and that the buffer selects indices at
random (Algorithm 1).  The reading taken here: every draw is one output word of
the counter-based generator Philox4x64 with 10 rounds (Salmon, Moraes, Dror,
Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11), with

    key     = (seed, 0)
    counter = (j, ticket, kind, 0)     kind: SAMPLE=1, EVICT=2, INIT=3

and a word w is mapped onto [0, n) by floor(w * n / 2^64) (the multiply-high map
of Lemire, "Fast random integer generation in an interval", 2019, without its
rejection step; the bias is at most n / 2^64).

Pins: the raw block function is checked bit-exactly against
numpy.random.Philox (an independent implementation of the same published
generator); the range map is checked by exhaustive counting on a reduced word
width.  Python integers are used so that no step can overflow silently.
"""
from __future__ import annotations

MASK64 = (1 << 64) - 1

# Round multipliers and Weyl key increments of Philox4x64 (Salmon et al., SC'11).
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B

KIND_SAMPLE = 1
KIND_EVICT = 2
KIND_INIT = 3


def philox4x64(counter, key, rounds: int = 10):
    """One Philox4x64 block: 4 counter words and 2 key words -> 4 output words.

    Each round multiplies counter words 0 and 2 by the round multipliers,
    splits the 128-bit products into high and low halves, and forms the new
    counter (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key is bumped by the
    Weyl increments between rounds.
    """
    c0, c1, c2, c3 = (int(v) & MASK64 for v in counter)
    k0, k1 = (int(v) & MASK64 for v in key)
    for _ in range(rounds):
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> 64, p0 & MASK64
        hi1, lo1 = p1 >> 64, p1 & MASK64
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0 = (k0 + PHILOX_W0) & MASK64
        k1 = (k1 + PHILOX_W1) & MASK64
    return c0, c1, c2, c3


def draw_word(seed: int, j: int, ticket: int, kind: int) -> int:
    """Output word 0 of Philox4x64-10 at counter (j, ticket, kind, 0), key (seed, 0)."""
    return philox4x64((j, ticket, kind, 0), (seed, 0))[0]


def uniform_int(w: int, n: int) -> int:
    """Map a 64-bit word onto [0, n): floor(w * n / 2^64)."""
    if n <= 0:
        raise ValueError("uniform_int needs n >= 1")
    return (int(w) * int(n)) >> 64


def draw_index(seed: int, j: int, ticket: int, kind: int, n: int) -> int:
    """Uniform index in [0, n) for draw j of the operation holding `ticket`."""
    return uniform_int(draw_word(seed, j, ticket, kind), n)


def init_uniform(seed: int, e: int, layer: int) -> float:
    """Uniform value in [-1, 1) for parameter element e of `layer` (kind INIT).

    The top 24 bits of the word give u = m / 2^24; the value is 2u - 1, exact
    in both fp32 and fp64.
    """
    w = philox4x64((e, layer, KIND_INIT, 0), (seed, 0))[0]
    m = w >> 40
    return 2.0 * (m / float(1 << 24)) - 1.0


def _mulhilo64_vec(a, b):
    """Vectorised 64x64 -> (hi, lo) product of uint64 numpy arrays via 32-bit halves."""
    import numpy as np
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a = a.astype(np.uint64)
    b = np.uint64(b) if np.isscalar(b) else b.astype(np.uint64)
    a_lo, a_hi = a & m32, a >> s32
    b_lo, b_hi = b & m32, b >> s32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    lo = a * b
    return hi, lo


def philox4x64_vec(c0, c1, c2, c3, k0: int, k1: int, rounds: int = 10):
    """Philox4x64 over numpy uint64 counter arrays (same rounds as philox4x64)."""
    import numpy as np
    c0, c1, c2, c3 = (np.asarray(v, dtype=np.uint64).copy() for v in (c0, c1, c2, c3))
    k0, k1 = int(k0) & MASK64, int(k1) & MASK64
    for _ in range(rounds):
        hi0, lo0 = _mulhilo64_vec(c0, PHILOX_M0)
        hi1, lo1 = _mulhilo64_vec(c2, PHILOX_M1)
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
        k0 = (k0 + PHILOX_W0) & MASK64
        k1 = (k1 + PHILOX_W1) & MASK64
    return c0, c1, c2, c3


def init_uniform_vec(seed: int, e, layer: int):
    """init_uniform for an array of element indices e (fp64 result)."""
    import numpy as np
    e = np.asarray(e, dtype=np.uint64)
    z = np.zeros_like(e)
    w = philox4x64_vec(e, z + np.uint64(layer), z + np.uint64(KIND_INIT), z, seed, 0)[0]
    m = (w >> np.uint64(40)).astype(np.float64)
    return 2.0 * (m / float(1 << 24)) - 1.0

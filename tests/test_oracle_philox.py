"""Pins of the oracle's Philox4x64-10 and range map.

The block function is compared with numpy.random.Philox, an independent
implementation of the same published generator (Salmon et al., SC'11).  Numpy
increments its 256-bit counter *before* producing each block (established
below), so its block for counter c is obtained by seeding it with c - 1.
"""
import numpy as np
import pytest

from oracle import philox as ph

M64 = (1 << 64) - 1


def _numpy_block(counter, key):
    c = list(counter)
    # numpy's first block uses counter + 1: seed it with counter - 1 (with borrow).
    v = (c[0] | (c[1] << 64) | (c[2] << 128) | (c[3] << 192)) - 1
    v &= (1 << 256) - 1
    cc = np.array([(v >> (64 * i)) & M64 for i in range(4)], dtype=np.uint64)
    g = np.random.Philox(counter=cc, key=np.array(key, dtype=np.uint64))
    return tuple(int(x) for x in g.random_raw(4))


def test_numpy_increments_before_output():
    g = np.random.Philox(counter=np.zeros(4, dtype=np.uint64), key=np.array([5, 0], dtype=np.uint64))
    first = tuple(int(x) for x in g.random_raw(4))
    assert first == ph.philox4x64((1, 0, 0, 0), (5, 0))
    assert first != ph.philox4x64((0, 0, 0, 0), (5, 0))


@pytest.mark.parametrize("counter,key", [
    ((0, 0, 0, 0), (0, 0)),
    ((1, 2, 3, 4), (5, 6)),
    ((M64, 0, 1, 0), (123456789, 0)),          # carry out of word 0 on numpy's side
    ((0, M64, 7, 0), (M64, M64)),
    ((M64, M64, M64, M64 - 1), (1, 2)),
    ((12345, 678, 2, 0), (2, 0)),
])
def test_block_matches_numpy(counter, key):
    assert ph.philox4x64(counter, key) == _numpy_block(counter, key)


def test_stream_of_1e5_blocks_matches_numpy():
    """10^5 consecutive blocks, starting just below a carry of counter word 0."""
    n = 100_000
    start = M64 - 50_000
    key = (0xDEADBEEF, 0x12345)
    g = np.random.Philox(counter=np.array([start - 1, 7, 0, 0], dtype=np.uint64),
                         key=np.array(key, dtype=np.uint64))
    ref = g.random_raw(4 * n).reshape(n, 4)
    idx = np.arange(n, dtype=object) + start
    c0 = np.array([int(v) & M64 for v in idx], dtype=np.uint64)
    c1 = np.array([7 + (int(v) >> 64) for v in idx], dtype=np.uint64)
    z = np.zeros(n, dtype=np.uint64)
    out = ph.philox4x64_vec(c0, c1, z, z, key[0], key[1])
    for w in range(4):
        assert np.array_equal(out[w], ref[:, w]), w


def test_vectorised_equals_scalar():
    rng = np.random.default_rng(3)
    c = rng.integers(0, 2**63, size=(200, 4), dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    out = ph.philox4x64_vec(c[:, 0], c[:, 1], c[:, 2], c[:, 3], 99, 1 << 63)
    for i in range(200):
        ref = ph.philox4x64(tuple(int(v) for v in c[i]), (99, 1 << 63))
        assert tuple(int(out[w][i]) for w in range(4)) == ref


def test_draw_word_counter_layout():
    # draw_word(seed, j, ticket, kind) is word 0 at counter (j, ticket, kind, 0), key (seed, 0).
    assert ph.draw_word(9, 3, 11, ph.KIND_SAMPLE) == _numpy_block((3, 11, 1, 0), (9, 0))[0]
    assert ph.draw_word(9, 3, 11, ph.KIND_EVICT) == _numpy_block((3, 11, 2, 0), (9, 0))[0]


@pytest.mark.parametrize("n", [1, 2, 3, 5, 7, 10, 1000, 65535, 65536, 65537])
def test_uniform_int_balanced_on_16bit_analogue(n):
    """Words k << 48 (k < 2^16) map to floor(k n / 2^16): every value is hit
    floor(2^16/n) or ceil(2^16/n) times when n <= 2^16 (the multiply-high map's
    defining property), and exactly once per k otherwise."""
    k = np.arange(1 << 16, dtype=object)
    vals = np.array([ph.uniform_int(int(v) << 48, n) for v in k], dtype=np.int64)
    assert vals.min() >= 0 and vals.max() <= n - 1
    assert np.all(np.diff(vals) >= 0)                 # monotone in the word
    if n <= (1 << 16):
        counts = np.bincount(vals, minlength=n)
        assert counts.min() >= (1 << 16) // n
        assert counts.max() <= -(-(1 << 16) // n)


def test_uniform_int_edges():
    for n in (1, 2, 3, 100_000, 2**31 - 1, 2**40 + 3):
        assert ph.uniform_int(0, n) == 0
        assert ph.uniform_int(M64, n) == n - 1
    with pytest.raises(ValueError):
        ph.uniform_int(5, 0)


def test_init_uniform_range_and_grid():
    e = np.arange(20_000, dtype=np.uint64)
    v = ph.init_uniform_vec(42, e, 1)
    assert v.min() >= -1.0 and v.max() < 1.0
    # every value is a multiple of 2^-23 and therefore exact in fp32
    assert np.all(v.astype(np.float32).astype(np.float64) == v)
    assert np.all((v * (1 << 23)) == np.round(v * (1 << 23)))
    assert abs(v.mean()) < 0.03
    assert abs(np.mean(v * v) - 1.0 / 3.0) < 0.02
    assert ph.init_uniform(42, 17, 1) == v[17]

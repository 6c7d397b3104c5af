"""Pins of the oracle's FIFO and FIRO buffers (Sec. 3.2.3).

1. FIFO against a literal queue written from the paper's description (append
   on receipt, batches from the front, each sample used once, production
   suspended while full): identical statuses and batches, deterministically.
2. FIRO against a literal list model (new samples appended at the end, each
   read pops one uniformly chosen position): the exact distribution of every
   observable (accepted counts, batch contents in draw order, resident set),
   enumerated with exact fractions over all draw outcomes, is identical --
   the oracle's partial Fisher-Yates is a different mechanism for the same
   law.  A planted bias (never drawing the last position) is detected.
3. Closed form: a FIFO fills its slots as a ring (the i-th stored sample
   sits in slot i mod C).
4. Invariants after every operation of long seeded runs, and uniformity (chi^2)
   of FIRO's picks.
"""
from collections import deque

import numpy as np
import pytest
from scipy import stats

from oracle import buffers as bf
from oracle import reservoir as rv
from tests.test_oracle_reservoir import enumerate_outcomes


class LiteralFIFO:
    """A queue as the paper describes FIFO."""

    def __init__(self, capacity):
        self.capacity, self.q, self.next_item, self.over = capacity, deque(), 0, False

    def put(self, k):
        acc = 0
        while acc < k and len(self.q) < self.capacity:   # production suspended while full
            self.q.append(self.next_item)
            self.next_item += 1
            acc += 1
        return acc

    def batch(self, b):
        if len(self.q) == 0 and self.over:
            return "empty"
        if len(self.q) < b and not self.over:
            return "not-ready"
        return tuple(self.q.popleft() for _ in range(min(b, len(self.q))))


class LiteralFIRO:
    """A list as the paper describes FIRO: append at the end, read (and remove)
    uniformly chosen positions, only above the threshold until production ends."""

    def __init__(self, capacity, threshold, draw):
        self.capacity, self.threshold, self.draw = capacity, threshold, draw
        self.items, self.next_item, self.over = [], 0, False

    def put(self, k):
        acc = 0
        while acc < k and len(self.items) < self.capacity:
            self.items.append(self.next_item)
            self.next_item += 1
            acc += 1
        return acc

    def batch(self, b):
        n = len(self.items)
        if self.over:
            if n == 0:
                return "empty"
        elif n <= self.threshold or n < b:
            return "not-ready"
        return tuple(self.items.pop(self.draw(len(self.items))) for _ in range(min(b, n)))

    def end(self):
        self.over = True
        self.threshold = 0


def oracle_run(cls, C, T, ops, draw=None):
    kw = {} if draw is None else {"draw": lambda kind, j, t, n: draw(n)}
    r = cls(C, T, 1, 1, seed=3, store_rows=False, **kw)
    res = []
    for op in ops:
        if op[0] == "put":
            res.append(("put", r.put(None, None, k=op[1])[1]))
        elif op[0] == "batch":
            ids = r.sample_id.copy()
            st, slots, _, _, _ = r.sample_batch(op[1])
            if st == rv.OK:
                res.append(("batch", tuple(int(ids[s]) for s in slots)))
            else:
                res.append(("batch", {rv.NOT_READY: "not-ready", rv.EMPTY: "empty"}[st]))
        else:
            r.end_reception()
            res.append(("end",))
        r.check_invariants()
    return tuple(res), tuple(sorted(int(r.sample_id[s]) for s in r.occ))


def literal_run(model, ops):
    res = []
    for op in ops:
        if op[0] == "put":
            res.append(("put", model.put(op[1])))
        elif op[0] == "batch":
            res.append(("batch", model.batch(op[1])))
        else:
            if hasattr(model, "end"):
                model.end()
            else:
                model.over = True
            res.append(("end",))
    items = model.q if hasattr(model, "q") else model.items
    return tuple(res), tuple(sorted(items))


FIFO_SEQS = [
    (4, [("batch", 1), ("put", 3), ("batch", 4), ("batch", 2), ("put", 5), ("batch", 3), ("put", 2),
         ("batch", 4), ("end",), ("batch", 3), ("batch", 3)]),
    (1, [("put", 2), ("batch", 1), ("batch", 1), ("put", 1), ("end",), ("batch", 5), ("batch", 1)]),
    (7, [("put", 6), ("batch", 2), ("put", 9), ("batch", 7), ("batch", 1), ("put", 3), ("end",), ("batch", 2)]),
]


@pytest.mark.parametrize("C,ops", FIFO_SEQS)
def test_fifo_equals_literal_queue(C, ops):
    assert oracle_run(bf.FIFOBuffer, C, 0, ops) == literal_run(LiteralFIFO(C), ops)


FIRO_SEQS = [
    (3, 1, [("put", 3), ("batch", 2), ("put", 2), ("batch", 2), ("put", 1)]),
    (4, 0, [("put", 2), ("batch", 1), ("put", 3), ("batch", 3), ("put", 4), ("batch", 2)]),
    (3, 1, [("put", 3), ("batch", 1), ("put", 3), ("end",), ("batch", 2), ("batch", 2), ("batch", 1)]),
    (4, 2, [("put", 4), ("batch", 2), ("batch", 2), ("put", 2), ("batch", 3), ("end",), ("batch", 3)]),
]


@pytest.mark.parametrize("C,T,ops", FIRO_SEQS)
def test_firo_distribution_equals_literal_list(C, T, ops):
    d_oracle = enumerate_outcomes(lambda draw: oracle_run(bf.FIROBuffer, C, T, ops, draw))
    d_lit = enumerate_outcomes(lambda draw: literal_run(LiteralFIRO(C, T, draw), ops))
    assert d_oracle == d_lit


def test_firo_enumeration_detects_planted_bias():
    C, T, ops = FIRO_SEQS[0]

    def biased(draw):
        # never picks the last position while more than one remains
        return oracle_run(bf.FIROBuffer, C, T, ops, lambda n: draw(n - 1) if n > 1 else draw(n))

    d_bad = enumerate_outcomes(biased)
    d_lit = enumerate_outcomes(lambda draw: literal_run(LiteralFIRO(C, T, draw), ops))
    assert d_bad != d_lit


def test_fifo_slots_form_a_ring():
    C = 13
    r = bf.FIFOBuffer(C, 0, 1, 1, seed=0, store_rows=False)
    rng = np.random.default_rng(4)
    stored = 0
    for _ in range(300):
        if rng.random() < 0.55:
            st, a, _, slots = r.put(None, None, k=int(rng.integers(0, 9)))
            assert slots == [(stored + i) % C for i in range(a)]
            stored += a
        else:
            r.sample_batch(int(rng.integers(1, 8)))
        r.check_invariants()
    assert stored > 3 * C


@pytest.mark.parametrize("cls", [bf.FIFOBuffer, bf.FIROBuffer])
def test_invariants_long_runs(cls):
    for seed in range(4):
        rng = np.random.default_rng(seed)
        C = int(rng.integers(5, 60))
        T = int(rng.integers(0, C))
        r = cls(C, T, 3, 5, seed=seed)
        key = 0
        out_ids = []
        for step in range(400):
            if step == 350:
                r.end_reception()
            if rng.random() < 0.5 and not r.reception_over:
                k = int(rng.integers(0, 12))
                u = np.arange(key, key + k, dtype=np.float32)[:, None] * np.ones((1, 5), np.float32)
                _, a, _, _ = r.put(u[:, :3], u, k=k)
                key += a
            else:
                ids = r.sample_id.copy()
                st, slots, xb, ub, _ = r.sample_batch(int(rng.integers(1, 10)))
                if st == rv.OK:
                    got = [int(ids[s]) for s in slots]
                    assert np.array_equal(ub[:, 0], np.array(got, dtype=np.float32))   # rows travel with ids
                    out_ids += got
            r.check_invariants()
        assert len(set(out_ids)) == len(out_ids)                       # each sample read at most once
        if cls is bf.FIFOBuffer:
            assert out_ids == list(range(len(out_ids)))                # in arrival order


def test_firo_picks_are_uniform():
    """Position of the first pick of each batch over many tickets: uniform."""
    n, C = 20, 40
    r = bf.FIROBuffer(C, 5, 1, 1, seed=11, store_rows=False)
    counts = np.zeros(n, np.int64)
    for _ in range(4000):
        r.put(None, None, k=n - r.N)
        pos_of = {s: i for i, s in enumerate(r.occ)}
        st, slots, _, _, _ = r.sample_batch(3)
        assert st == rv.OK
        counts[pos_of[slots[0]]] += 1
    assert stats.chisquare(counts).pvalue > 1e-3


def test_statuses():
    f = bf.FIFOBuffer(4, 0, 1, 1, seed=0)
    assert f.sample_batch(1)[0] == rv.NOT_READY
    assert f.put(None, np.zeros((6, 1), np.float32))[:2] == (rv.OK, 4)
    assert f.put(None, np.zeros((1, 1), np.float32))[:2] == (rv.FULL, 0)
    g = bf.FIROBuffer(8, 3, 1, 1, seed=0)
    g.put(None, np.zeros((3, 1), np.float32))
    assert g.sample_batch(1)[0] == rv.NOT_READY        # N <= T
    g.put(None, np.zeros((1, 1), np.float32))
    assert g.sample_batch(5)[0] == rv.NOT_READY        # N < B
    assert g.sample_batch(4)[0] == rv.OK
    g.end_reception()
    assert g.put(None, np.zeros((1, 1), np.float32))[0] == rv.E_CLOSED
    assert g.sample_batch(1)[0] == rv.EMPTY

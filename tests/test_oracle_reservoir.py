"""Pins of the oracle's reservoir (slot encoding of Algorithm 1).

1. Exact distributions: for short operation sequences on tiny buffers, every
   draw outcome is enumerated with exact fractions, for the oracle and for a
   model of the buffer built from the behaviour Sec. 3.2.3 states
   (tests/reservoir_model.py); the distributions of everything
   observable (accepted counts, batch contents in draw order, resident items
   with their draw counts) must be identical.
2. Deterministic invariants after every operation on longer seeded runs.
3. Statistics: uniform draws, expected number of newly seen items per batch,
   and the residency time of Appendix A.
"""
from collections import Counter, defaultdict
from fractions import Fraction

import numpy as np
import pytest

from oracle import reservoir as rv
from oracle.philox import KIND_EVICT, KIND_SAMPLE, draw_index
from tests.reservoir_model import BehaviourReservoir


# --------------------------------------------------------------------------- enumeration
def enumerate_outcomes(run_fn):
    """Exact outcome distribution of run_fn(draw) over all draw sequences."""
    dist = defaultdict(Fraction)
    prefix = []
    while True:
        made = []

        def draw(n):
            pos = len(made)
            c = prefix[pos] if pos < len(prefix) else 0
            made.append((c, n))
            return c

        out = run_fn(draw)
        p = Fraction(1)
        for _, n in made:
            p /= n
        dist[out] += p
        k = len(made) - 1
        while k >= 0 and made[k][0] + 1 >= made[k][1]:
            k -= 1
        if k < 0:
            break
        prefix = [c for c, _ in made[:k]] + [made[k][0] + 1]
    assert sum(dist.values()) == 1
    return dict(dist)


def run_slots_ids(C, T, ops, draw):
    """Oracle run over ops; batch item ids are read at draw time (valid in the drain too)."""
    r = rv.Reservoir(C, T, 1, 1, seed=0, draw=lambda kind, j, t, n: draw(n), store_rows=False)
    res = []
    for op in ops:
        if op[0] == "put":
            _, acc, _, _ = r.put(None, None, k=op[1])
            res.append(("put", acc))
        elif op[0] == "batch":
            ids_before = r.sample_id.copy()
            st, slots, _, _, _ = r.sample_batch(op[1])
            if st == rv.OK:
                res.append(("batch", tuple(int(ids_before[s]) for s in slots)))
            else:
                res.append(("batch", {rv.NOT_READY: "not-ready", rv.EMPTY: "empty"}[st]))
        else:
            r.end_reception()
            res.append(("end",))
        r.check_invariants()
    resident = tuple(sorted((int(r.sample_id[s]), int(r.seen_count[s])) for s in r.occ))
    return tuple(res), resident


def run_model(C, T, ops, draw):
    m = BehaviourReservoir(C, T, draw)
    res = []
    for op in ops:
        if op[0] == "put":
            acc = 0
            while acc < op[1] and m.store():
                acc += 1
            res.append(("put", acc))
        elif op[0] == "batch":
            items = []
            status = None
            for _ in range(op[1]):
                it = m.draw_one()
                if it in (m.NOT_READY, m.EMPTY):
                    if not items:
                        status = it
                    break
                items.append(it)
            res.append(("batch", status if status is not None else tuple(items)))
        else:
            m.close()
            res.append(("end",))
    return tuple(res), m.resident()


SEQUENCES = [
    # (capacity, threshold, ops)
    (3, 1, [("put", 2), ("batch", 2), ("put", 2), ("batch", 2), ("put", 2)]),
    (3, 0, [("put", 3), ("batch", 2), ("put", 3), ("batch", 1), ("put", 1), ("batch", 2)]),
    (4, 2, [("put", 2), ("batch", 1), ("put", 3), ("batch", 3), ("put", 4)]),
    (2, 0, [("put", 1), ("batch", 2), ("put", 2), ("batch", 2), ("put", 2), ("batch", 1)]),
    (3, 1, [("put", 3), ("batch", 2), ("put", 2), ("end",), ("batch", 2), ("batch", 2), ("batch", 1)]),
    (4, 1, [("put", 3), ("batch", 3), ("put", 2), ("end",), ("batch", 3), ("batch", 3)]),
]


@pytest.mark.parametrize("C,T,ops", SEQUENCES)
def test_distribution_equals_behavioural_model(C, T, ops):
    d_slots = enumerate_outcomes(lambda draw: run_slots_ids(C, T, ops, draw))
    d_model = enumerate_outcomes(lambda draw: run_model(C, T, ops, draw))
    assert d_slots == d_model


def test_enumeration_detects_a_biased_eviction():
    """A planted mistake (evicting the first seen slot instead of a random one)
    must change the distribution, so the comparison above has teeth."""
    C, T, ops = 3, 0, [("put", 3), ("batch", 2), ("put", 1), ("batch", 2)]

    def biased(draw):
        def d(kind, j, t, n):
            return 0 if kind == KIND_EVICT else draw(n)
        r = rv.Reservoir(C, T, 1, 1, seed=0, draw=d, store_rows=False)
        out = []
        for op in ops:
            if op[0] == "put":
                out.append(("put", r.put(None, None, k=op[1])[1]))
            else:
                ids = r.sample_id.copy()
                st, slots, *_ = r.sample_batch(op[1])
                out.append(("batch", tuple(int(ids[s]) for s in slots)))
        return tuple(out), tuple(sorted((int(r.sample_id[s]), int(r.seen_count[s])) for s in r.occ))

    assert enumerate_outcomes(biased) != enumerate_outcomes(lambda draw: run_model(C, T, ops, draw))


# --------------------------------------------------------------------------- deterministic rules
def test_threshold_and_tickets():
    r = rv.Reservoir(10, 4, 2, 3, seed=1)
    x = np.zeros((4, 2), np.float32)
    u = np.arange(12, dtype=np.float32).reshape(4, 3)
    assert r.put(x, u)[:3] == (rv.OK, 4, 0)
    st, *_ = r.sample_batch(3)
    assert st == rv.NOT_READY and r.next_ticket == 1        # refused calls take no ticket
    assert r.put(x[:1], u[:1])[:3] == (rv.OK, 1, 1)
    st, slots, xb, ub, ticket = r.sample_batch(3)
    assert st == rv.OK and ticket == 2
    assert np.array_equal(ub, r.us[slots])
    r.check_invariants()


def test_prefix_accept_and_full():
    r = rv.Reservoir(4, 0, 1, 1, seed=2)
    rows = np.ones((6, 1), np.float32)
    st, acc, _, slots = r.put(rows, rows)
    assert acc == 4 and slots == [0, 1, 2, 3]
    st, acc, _, _ = r.put(rows, rows)
    assert st == rv.FULL and acc == 0                     # U == C: nothing accepted
    r.sample_batch(1)
    seen = int(np.sum(r.seen_count >= 1))
    st, acc, _, slots = r.put(rows, rows)
    assert acc == seen and all(r.seen_count[s] == 0 for s in slots)
    r.check_invariants()


def test_drain_and_closed():
    r = rv.Reservoir(8, 3, 1, 1, seed=3)
    rows = np.arange(8, dtype=np.float32)[:, None]
    r.put(rows, rows)
    r.sample_batch(5)
    r.end_reception()
    assert r.put(rows, rows)[0] == rv.E_CLOSED
    got = []
    while True:
        st, slots, xb, ub, _ = r.sample_batch(3)
        if st == rv.EMPTY:
            break
        assert st == rv.OK
        got += ub[:, 0].tolist()
        r.check_invariants()
    assert sorted(got) == list(range(8))                  # each item once, last batch short
    assert r.N == 0 and r.U == 0 and r.S == 0


def test_invariants_long_seeded_run():
    rng = np.random.default_rng(11)
    r = rv.Reservoir(50, 20, 2, 4, seed=5)
    key = 0
    for step in range(400):
        if rng.random() < 0.6:
            k = int(rng.integers(1, 12))
            keys = np.arange(key, key + k)
            u = np.repeat(keys[:, None].astype(np.float32), 4, axis=1)
            st, acc, ticket, slots = r.put(u[:, :2], u)
            ids = [int(r.sample_id[s]) for s in slots]
            assert ids == list(range(r.next_sample_id - acc, r.next_sample_id))   # consecutive
            key += acc
        else:
            st, slots, xb, ub, _ = r.sample_batch(int(rng.integers(1, 16)))
            if st == rv.OK:
                assert np.array_equal(ub[:, 0], r.sample_id[slots].astype(np.float32))
        r.check_invariants()
    assert r.total_evicted > 0
    r.end_reception()
    while r.sample_batch(7)[0] == rv.OK:
        r.check_invariants()
    assert r.N == 0


def test_philox_draws_are_the_index_path():
    """The default draw is uniform_int(Philox(seed; j, ticket, SAMPLE), N) over occupied slots."""
    r = rv.Reservoir(30, 5, 1, 1, seed=77)
    rows = np.zeros((30, 1), np.float32)
    r.put(rows, rows)
    st, slots, _, _, ticket = r.sample_batch(16)
    assert slots == [draw_index(77, j, ticket, KIND_SAMPLE, 30) for j in range(16)]


# --------------------------------------------------------------------------- statistics
def test_draws_uniform_chi_square():
    from scipy.stats import chisquare
    n = 97
    r = rv.Reservoir(n, 0, 1, 1, seed=8, store_rows=False)
    r.put(None, None, k=n)
    counts = np.zeros(n)
    for _ in range(200):
        st, slots, *_ = r.sample_batch(64)
        np.add.at(counts, slots, 1)
    assert chisquare(counts).pvalue > 1e-4


def test_victims_uniform_chi_square():
    from scipy.stats import chisquare
    C = 40
    counts = np.zeros(C)
    for seed in range(300):
        r = rv.Reservoir(C, 0, 1, 1, seed=seed, store_rows=False)
        r.put(None, None, k=C)
        for s in range(C):
            r.seen_count[s] = 1
        r.U, r.S = 0, C
        _, _, _, slots = r.put(None, None, k=5)
        np.add.at(counts, slots, 1)
    assert chisquare(counts).pvalue > 1e-4


def test_expected_newly_seen_per_batch():
    """E[# distinct unseen items drawn] = U (1 - (1 - 1/N)^B) for B draws with replacement."""
    N, B, trials = 200, 64, 400
    total = 0
    for t in range(trials):
        r = rv.Reservoir(N, 0, 1, 1, seed=1000 + t, store_rows=False)
        r.put(None, None, k=N)
        u0 = r.U
        r.sample_batch(B)
        total += u0 - r.U
    expect = N * (1 - (1 - 1 / N) ** B)
    sd = np.sqrt(N * (1 - 1 / N) ** B * (1 - (1 - 1 / N) ** B)) / np.sqrt(trials)  # loose bound
    assert abs(total / trials - expect) < 6 * sd + 0.5


def test_appendix_a_residency():
    """Appendix A: with random-location replacement in a full buffer of n slots,
    an item stays on average n - 1 further insertions.  With single-item puts
    and every resident item seen between puts, eviction is uniform over all n
    slots, which is that regime."""
    n = 25
    r = rv.Reservoir(n, 0, 1, 1, seed=4, store_rows=False)
    r.put(None, None, k=n)
    for s in range(n):
        r.seen_count[s] = 1
    r.U, r.S = 0, n
    r.total_draws = n
    born = {int(r.sample_id[s]): 0 for s in range(n)}
    lifetimes = []
    for ins in range(1, 20000):
        _, acc, _, slots = r.put(None, None, k=1)
        s = slots[0]
        # the evicted item is the one that was in slot s
        # (its id was overwritten: recover from the born map)
        new_id = int(r.sample_id[s])
        gone = [i for i in born if i not in set(r.sample_id.tolist())]
        for g in gone:
            lifetimes.append(ins - 1 - born.pop(g))
        born[new_id] = ins
        r.seen_count[s] = 1
        r.U -= 1
        r.S += 1
        r.total_draws += 1
    mean = float(np.mean(lifetimes))
    sd = np.sqrt(n * (n - 1)) / np.sqrt(len(lifetimes))
    assert abs(mean - (n - 1)) < 5 * sd

"""Reservoir training buffer, slot encoding of Algorithm 1 (oracle side).

What the paper fixes (Algorithm 1 "Reservoir" and Sec. 3.2.3):
  * fixed capacity C, items are either not-seen (never drawn into a batch)
    or seen;
  * get(): wait while the population is <= threshold; draw one index uniformly
    over seen + not-seen; a not-seen pick moves to seen; selection is with
    replacement; after reception is over, every pick is deleted (drain);
  * put(): wait while not-seen fills the capacity; if the buffer is full,
    evict one uniformly chosen *seen* item; append the new item as not-seen.

Readings taken where the paper is silent or loose:
  * the index space of the draw is the list of occupied slots in slot order
    (one uniform draw over the union, which is what the algorithm's
    seen.size + not_seen.size range means);
  * draws come from Philox4x64-10 (see philox.py), counter (j, ticket, kind);
  * a put of K rows accepts the in-order prefix a = min(K, C - U) instead of
    blocking (U = not-seen count), fills free slots first in ascending order,
    then replaces victims chosen by a partial Fisher-Yates shuffle over the
    ascending list of seen slots; row F + j goes to victim j;
  * a batch of B draws is atomic with respect to puts;
  * a batch is refused (NOT_READY) while N <= T, as the algorithm's wait
    condition reads; after end_reception the threshold is 0 and a batch of
    min(B, N) distinct items is drawn by partial Fisher-Yates and deleted.

Every call that changes state takes the next ticket; refused calls do not.

Pins: exact outcome distributions against a model of the buffer built from the
behaviour Sec. 3.2.3 states
(enumeration with exact fractions), deterministic invariants after every op,
and statistical checks (uniformity, expected number of newly seen items,
Appendix A residency).  The exact index path is this reading's own; it has no
printed worked example in the paper ("parity unpinned" for the path itself,
pinned for its distribution).
"""
from __future__ import annotations

from collections import Counter
from typing import Callable, List, Optional

import numpy as np

from .philox import KIND_EVICT, KIND_SAMPLE, draw_index

OK = 0
NOT_READY = 1
FULL = 2
EMPTY = 3
E_INVAL = -1
E_CLOSED = -4

DrawFn = Callable[[int, int, int, int], int]   # (kind, j, ticket, n) -> index in [0, n)


class Reservoir:
    """Fixed-capacity buffer of (x, u) rows with per-slot seen counts."""

    def __init__(self, capacity: int, threshold: int, x_dim: int, u_dim: int, seed: int,
                 draw: Optional[DrawFn] = None, store_rows: bool = True):
        if capacity <= 0 or threshold < 0 or x_dim <= 0 or u_dim <= 0:
            raise ValueError("bad reservoir shape")
        self.C = int(capacity)
        self.T = int(threshold)
        self.seed = int(seed)
        self.x_dim, self.u_dim = int(x_dim), int(u_dim)
        self.store_rows = store_rows
        if store_rows:
            self.xs = np.zeros((self.C, self.x_dim), dtype=np.float32)
            self.us = np.zeros((self.C, self.u_dim), dtype=np.float32)
        self.seen_count = np.zeros(self.C, dtype=np.int64)
        self.sample_id = np.full(self.C, -1, dtype=np.int64)
        self.occupied = np.zeros(self.C, dtype=bool)
        self.occ: List[int] = []          # occupied slots, index order of the draws
        self.U = 0                        # not-seen population
        self.S = 0                        # seen population
        self.total_put = 0
        self.total_evicted = 0
        self.total_deleted = 0
        self.total_draws = 0
        self.next_ticket = 0
        self.next_sample_id = 0
        self.reception_over = False
        self.evict_hist: Counter = Counter()   # seen count at eviction / deletion
        self._draw = draw if draw is not None else self._philox_draw

    # -- random draws ---------------------------------------------------------------
    def _philox_draw(self, kind: int, j: int, ticket: int, n: int) -> int:
        return draw_index(self.seed, j, ticket, kind, n)

    @property
    def N(self) -> int:
        return len(self.occ)

    # -- put ----------------------------------------------------------------------------
    def put(self, xs: Optional[np.ndarray], us: Optional[np.ndarray], k: Optional[int] = None):
        """Store up to K rows.  Returns (status, accepted, ticket, slots)."""
        if k is None:
            k = len(us)
        if self.reception_over:
            return E_CLOSED, 0, None, []
        if k < 0:
            return E_INVAL, 0, None, []
        ticket = self.next_ticket
        self.next_ticket += 1
        n_before = self.N
        a = min(k, self.C - self.U)                 # not-seen may not exceed the capacity
        f = min(a, self.C - n_before)               # rows that find a free slot
        e = a - f                                   # rows that replace a seen item
        free = np.flatnonzero(~self.occupied)[:f].tolist()
        # Victims: uniform without replacement among seen slots, by partial
        # Fisher-Yates over the ascending list of seen slots.
        seen_slots = np.flatnonzero(self.occupied & (self.seen_count >= 1)).tolist()
        assert e <= len(seen_slots)
        for j in range(e):
            r = j + self._draw(KIND_EVICT, j, ticket, len(seen_slots) - j)
            seen_slots[j], seen_slots[r] = seen_slots[r], seen_slots[j]
        victims = seen_slots[:e]
        slots = free + victims
        for v in victims:
            self.evict_hist[int(self.seen_count[v])] += 1
            self.total_evicted += 1
            self.S -= 1
        for row, s in enumerate(slots):
            if self.store_rows:
                if xs is not None:
                    self.xs[s] = xs[row]
                self.us[s] = us[row]
            self.sample_id[s] = self.next_sample_id
            self.next_sample_id += 1
            self.seen_count[s] = 0
            if not self.occupied[s]:
                self.occupied[s] = True
                self.occ.append(s)
        self.U += a
        self.total_put += a
        return (OK if a > 0 else FULL), a, ticket, slots

    # -- sample ------------------------------------------------------------------------
    def sample_batch(self, b: int):
        """Draw a batch.  Returns (status, slots, x rows, u rows, ticket)."""
        if b <= 0:
            return E_INVAL, [], None, None, None
        n = self.N
        if self.reception_over:
            if n == 0:
                return EMPTY, [], None, None, None
        elif n <= self.T:
            return NOT_READY, [], None, None, None
        ticket = self.next_ticket
        self.next_ticket += 1
        if not self.reception_over:
            idx = [self._draw(KIND_SAMPLE, j, ticket, n) for j in range(b)]
            slots = [self.occ[i] for i in idx]
            for s in slots:
                if self.seen_count[s] == 0:
                    self.U -= 1
                    self.S += 1
                self.seen_count[s] += 1
            self.total_draws += b
        else:
            bb = min(b, n)
            order = list(self.occ)
            for j in range(bb):
                r = j + self._draw(KIND_SAMPLE, j, ticket, n - j)
                order[j], order[r] = order[r], order[j]
            slots = order[:bb]
            for s in slots:
                if self.seen_count[s] == 0:
                    self.U -= 1
                else:
                    self.S -= 1
                self.seen_count[s] += 1
                self.evict_hist[int(self.seen_count[s])] += 1
                self.total_deleted += 1
                self.occupied[s] = False
            self.total_draws += bb
            self.occ = order[bb:]
        if self.store_rows:
            xb = self.xs[slots].copy()
            ub = self.us[slots].copy()
        else:
            xb = ub = None
        return OK, slots, xb, ub, ticket

    def end_reception(self) -> int:
        """No more puts; the threshold is lifted and later batches drain the buffer."""
        self.reception_over = True
        self.T = 0
        return OK

    # -- invariants --------------------------------------------------------------------
    def check_invariants(self) -> None:
        """Deterministic invariants that hold after every operation."""
        C, N, U, S = self.C, self.N, self.U, self.S
        assert 0 <= U <= C and S >= 0 and N == U + S <= C
        occ = np.zeros(C, dtype=bool)
        occ[self.occ] = True
        assert np.array_equal(occ, self.occupied)
        assert len(set(self.occ)) == N
        resident_unseen = int(np.sum(self.occupied & (self.seen_count == 0)))
        resident_seen = int(np.sum(self.occupied & (self.seen_count >= 1)))
        assert resident_unseen == U and resident_seen == S
        if not self.reception_over:
            assert self.occ == list(range(N))
            assert N == min(C, self.total_put)
            assert self.total_put == N + self.total_evicted
        assert self.evict_hist.get(0, 0) == 0
        # Every draw is counted once: on a resident slot's seen count, or in the
        # histogram of items that left the buffer (evicted by a put, or deleted
        # by a drain batch).
        drawn = int(np.sum(self.seen_count[self.occupied]))
        drawn += sum(k * c for k, c in self.evict_hist.items())
        assert drawn == self.total_draws
        assert sum(self.evict_hist.values()) == self.total_evicted + self.total_deleted
        ids = self.sample_id[self.occupied]
        assert len(set(ids.tolist())) == N

    def stats(self) -> dict:
        return dict(capacity=self.C, threshold=self.T, n=self.N, unseen=self.U, seen=self.S,
                    total_put=self.total_put, total_evicted=self.total_evicted,
                    total_deleted=self.total_deleted, total_draws=self.total_draws,
                    next_ticket=self.next_ticket, next_sample_id=self.next_sample_id,
                    reception_over=self.reception_over)

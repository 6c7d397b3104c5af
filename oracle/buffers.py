"""FIFO and FIRO training buffers (oracle side): the two comparison buffers of
Sec. 3.2.3, which evict a sample when it is read, unlike the Reservoir.

What the paper fixes:
  * FIFO (first in, first out): batches are formed in the order samples were
    received; every sample is used exactly once; a batch can be extracted as
    soon as the buffer holds one; production is suspended while the buffer is
    full.
  * FIRO (first in, random out): like FIFO, samples leave the buffer when they
    are read, but they are taken from random positions; batches are extracted
    only while the buffer holds more than a threshold of samples; the
    threshold becomes 0 once production is over.  The buffer is a list and
    new samples are appended at its end.

Readings taken where the paper is silent or loose:
  * a put of K rows accepts the in-order prefix a = min(K, C - N) instead of
    blocking (a = 0 when the buffer is full);
  * a batch in the normal phase needs B samples (FIFO: N >= B; FIRO: N > T and
    N >= B); after end_reception the last batch may be short, min(B, N), and
    an empty buffer answers EMPTY;
  * FIRO draws its B distinct positions by a partial Fisher-Yates shuffle of
    the list, step j taking position j after swapping it with position
    j + uniform_int(Philox(seed; j, ticket, SAMPLE), N - j); the list that
    remains is the shuffled list without its first B entries;
  * slot storage: a freed slot joins the end of a queue of free slots, and a
    stored row takes the slot at the head of that queue (initially 0..C-1 in
    order), so FIFO fills the slab as a ring.

Every call that changes state takes the next ticket; refused calls do not.
"""
from __future__ import annotations

from collections import Counter, deque
from typing import List, Optional

import numpy as np

from .philox import KIND_SAMPLE, draw_index
from .reservoir import E_CLOSED, E_INVAL, EMPTY, FULL, NOT_READY, OK, DrawFn


class _ListBuffer:
    """Buffer whose samples leave when read; `random_out` selects FIRO."""

    random_out = False

    def __init__(self, capacity: int, threshold: int, x_dim: int, u_dim: int, seed: int,
                 draw: Optional[DrawFn] = None, store_rows: bool = True):
        if capacity <= 0 or threshold < 0 or x_dim <= 0 or u_dim <= 0:
            raise ValueError("bad buffer shape")
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
        self.occ: List[int] = []                  # the list of stored samples (their slots)
        self.free = deque(range(self.C))          # free slots, head first
        self.total_put = 0
        self.total_evicted = 0                    # never: nothing is replaced by a put
        self.total_deleted = 0
        self.total_draws = 0
        self.next_ticket = 0
        self.next_sample_id = 0
        self.reception_over = False
        self.evict_hist: Counter = Counter()      # seen count of samples that left the buffer
        self._draw = draw if draw is not None else (
            lambda kind, j, ticket, n: draw_index(self.seed, j, ticket, kind, n))

    @property
    def N(self) -> int:
        return len(self.occ)

    @property
    def U(self) -> int:                           # every stored sample is unseen
        return len(self.occ)

    @property
    def S(self) -> int:
        return 0

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
        a = min(k, self.C - self.N)
        slots = [self.free.popleft() for _ in range(a)]
        for row, s in enumerate(slots):
            if self.store_rows:
                if xs is not None:
                    self.xs[s] = xs[row]
                self.us[s] = us[row]
            self.sample_id[s] = self.next_sample_id
            self.next_sample_id += 1
            self.seen_count[s] = 0
            self.occupied[s] = True
        self.occ.extend(slots)
        self.total_put += a
        return (OK if a > 0 else FULL), a, ticket, slots

    def ready(self, b: int) -> bool:
        if self.random_out:
            return self.N > self.T and self.N >= b
        return self.N >= b

    def sample_batch(self, b: int):
        """Take a batch out of the buffer.  Returns (status, slots, x rows, u rows, ticket)."""
        if b <= 0:
            return E_INVAL, [], None, None, None
        n = self.N
        if self.reception_over:
            if n == 0:
                return EMPTY, [], None, None, None
            bb = min(b, n)
        elif not self.ready(b):
            return NOT_READY, [], None, None, None
        else:
            bb = b
        ticket = self.next_ticket
        self.next_ticket += 1
        order = list(self.occ)
        if self.random_out:
            for j in range(bb):
                r = j + self._draw(KIND_SAMPLE, j, ticket, n - j)
                order[j], order[r] = order[r], order[j]
        slots = order[:bb]
        self.occ = order[bb:]
        for s in slots:
            self.seen_count[s] += 1
            self.evict_hist[int(self.seen_count[s])] += 1
            self.occupied[s] = False
            self.free.append(s)
        self.total_deleted += bb
        self.total_draws += bb
        if self.store_rows:
            xb = self.xs[slots].copy()
            ub = self.us[slots].copy()
        else:
            xb = ub = None
        return OK, slots, xb, ub, ticket

    def end_reception(self) -> int:
        self.reception_over = True
        self.T = 0
        return OK

    def check_invariants(self) -> None:
        C, N = self.C, self.N
        assert 0 <= N <= C
        occ = np.zeros(C, dtype=bool)
        occ[self.occ] = True
        assert np.array_equal(occ, self.occupied) and len(set(self.occ)) == N
        assert sorted(list(self.free) + self.occ) == list(range(C))   # free queue and list partition the slots
        assert np.all(self.seen_count[self.occupied] == 0)          # a sample is read at most once
        assert self.total_put == N + self.total_deleted
        assert self.total_draws == self.total_deleted
        assert dict(self.evict_hist) in ({}, {1: self.total_deleted})
        assert len(set(self.sample_id[self.occupied].tolist())) == N

    def stats(self) -> dict:
        return dict(capacity=self.C, threshold=self.T, n=self.N, unseen=self.U, seen=self.S,
                    total_put=self.total_put, total_evicted=self.total_evicted,
                    total_deleted=self.total_deleted, total_draws=self.total_draws,
                    next_ticket=self.next_ticket, next_sample_id=self.next_sample_id,
                    reception_over=self.reception_over)


class FIFOBuffer(_ListBuffer):
    """Samples in arrival order, each read once (Sec. 3.2.3, FIFO)."""
    random_out = False


class FIROBuffer(_ListBuffer):
    """Samples read once from random positions, above a threshold (Sec. 3.2.3, FIRO)."""
    random_out = True

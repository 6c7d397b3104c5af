"""A list-based model of the paper's Reservoir buffer (Algorithm 1), for tests.

It keeps the two Python lists of the algorithm, `not_seen` and `seen`, and
performs one item per get() / put() exactly as the algorithm describes, with
the waits turned into refusals.  The draw over seen + not_seen indexes the
concatenation not_seen ++ seen (the algorithm's single index over both lists).
Its only purpose is to serve as the independent reference against which the
oracle's slot encoding is checked in distribution.
"""
from __future__ import annotations

from collections import Counter


class ListReservoir:
    NOT_READY = "not-ready"
    EMPTY = "empty"

    def __init__(self, capacity, threshold, draw):
        self.capacity = capacity
        self.threshold = threshold
        self.seen = []
        self.not_seen = []
        self.reception_over = False
        self.draw = draw                 # draw(n) -> index in [0, n)
        self.draw_count = Counter()      # bookkeeping for tests, not part of the algorithm
        self.next_item = 0

    def size(self):
        return len(self.seen) + len(self.not_seen)

    def get(self):
        if self.reception_over:
            if self.size() == 0:
                return self.EMPTY
        elif self.size() <= self.threshold:
            return self.NOT_READY
        index = self.draw(self.size())
        if index < len(self.not_seen):
            item = self.not_seen.pop(index)
            if not self.reception_over:
                self.seen.append(item)
        else:
            pos = index - len(self.not_seen)
            item = self.seen[pos]
            if self.reception_over:
                del self.seen[pos]
        self.draw_count[item] += 1
        return item

    def put(self):
        """Offer one new item; False means the algorithm would block."""
        if len(self.not_seen) >= self.capacity:
            return False
        if self.size() >= self.capacity:
            del self.seen[self.draw(len(self.seen))]
        self.not_seen.append(self.next_item)
        self.next_item += 1
        return True

    def end_reception(self):
        self.reception_over = True
        self.threshold = 0

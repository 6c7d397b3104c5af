"""A model of the paper's Reservoir buffer built from the behaviour Sec. 3.2.3
states, for tests: it is the independent reference against which the
oracle's slot encoding is compared in distribution.

What the section fixes, and all this model does:
* the buffer stores items, each unseen until it is first drawn into a batch;
* a draw picks uniformly among every stored item, seen or unseen, and leaves
  it in the buffer (with replacement), while more items than the threshold
  are stored; otherwise it is refused;
* storing a new item is refused while unseen items fill the buffer; when the
  buffer is full, a uniformly chosen seen item makes room (no unseen item is
  ever discarded);
* after reception ends the threshold is lifted and every draw removes the
  item it picks, until the buffer is empty.

Items live in one list in arrival order together with the number of times
each was drawn; draw(n) supplies a uniform index in [0, n).
"""
from __future__ import annotations


class BehaviourReservoir:
    NOT_READY = "not-ready"
    EMPTY = "empty"

    def __init__(self, capacity, threshold, draw):
        self.capacity = capacity
        self.threshold = threshold
        self.draw = draw
        self.stored = []                 # [item, times drawn] in arrival order
        self.closed = False              # reception over
        self.next_item = 0

    def store(self) -> bool:
        """Offer one new item; False when unseen items fill the buffer."""
        if sum(1 for _, drawn in self.stored if drawn == 0) >= self.capacity:
            return False
        if len(self.stored) == self.capacity:
            seen = [entry for entry in self.stored if entry[1] > 0]
            self.stored.remove(seen[self.draw(len(seen))])
        self.stored.append([self.next_item, 0])
        self.next_item += 1
        return True

    def draw_one(self):
        """One draw: an item id, NOT_READY or EMPTY."""
        if self.closed and not self.stored:
            return self.EMPTY
        if not self.closed and len(self.stored) <= self.threshold:
            return self.NOT_READY
        entry = self.stored[self.draw(len(self.stored))]
        entry[1] += 1
        if self.closed:
            self.stored.remove(entry)
        return entry[0]

    def close(self):
        self.closed = True
        self.threshold = 0

    def resident(self):
        """Sorted (item, times drawn) of the stored items."""
        return tuple(sorted((item, drawn) for item, drawn in self.stored))

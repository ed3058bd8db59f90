"""Integer model of the rolling KV cache as a ring of chunk slots (oracle; test infrastructure only).

Paper Sec. 3.5, "Structured Rolling KV Cache": committed chunks enter a
fixed-capacity FIFO; once it is over capacity the oldest committed chunks are
discarded.  Committed chunks are never modified afterwards.

Model: chunks are numbered by commit order c = 0, 1, 2, ...  ``head`` counts
commits, ``tail`` counts evictions; the live chunks are [tail, head).  The
ring has S slots and chunk c lives in slot c mod S.  A commit into a full ring
(head - tail == S) and an eviction of more chunks than are live are errors.
The attention window of w chunks is the newest w live chunks, oldest first.
"""
from __future__ import annotations


class RingError(Exception):
    pass


class RingModel:
    def __init__(self, slots: int):
        if slots < 1:
            raise RingError("slots must be >= 1")
        self.S = int(slots)
        self.head = 0
        self.tail = 0

    @property
    def live(self) -> int:
        return self.head - self.tail

    def append(self) -> int:
        """Commit the next chunk; returns the slot it is written to."""
        if self.live == self.S:
            raise RingError("ring full")
        slot = self.head % self.S
        self.head += 1
        return slot

    def evict(self, n: int) -> None:
        """Discard the n oldest live chunks."""
        if n < 0 or n > self.live:
            raise RingError("evict beyond live chunks")
        self.tail += n

    def slot_of(self, chunk: int) -> int:
        return chunk % self.S if self.tail <= chunk < self.head else -1

    def window(self, w=None) -> list:
        """Logical chunk ids of the newest w live chunks (all live if None), oldest first."""
        if w is None:
            w = self.live
        if w < 0 or w > self.live:
            raise RingError("window larger than live chunks")
        return list(range(self.head - w, self.head))

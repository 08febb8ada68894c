"""Eviction order restated as an LRU over recorded history -- TEST INFRASTRUCTURE.

An independent, pure-Python statement of the retention rule of page-based
RaaS (Sections 3.2 and 3.3 of arXiv 2502.11147), used to pin the C oracle.
It keeps no timestamps. Instead it records, for every decode page, the step
that created it and every step at which it was "used" (its score was among
the top-r of the evictable pages), and when the cache is full it evicts the
page whose most recent use is oldest -- the definition of least recently
used -- breaking ties by the older page (smaller logical id).

Driven with the same page scores as the oracle, the two must make the same
decisions at every step.
"""
from __future__ import annotations

import math


class HistoryLRU:
    def __init__(self, page_size: int, slots: int, r: float, prefill_len: int,
                 pin_head: bool = True, rank_pinned: bool = False):
        self.ps, self.S, self.r = page_size, slots, r
        self.rank_pinned = rank_pinned           # pinned pages take part in the ranking
        pages = -(-prefill_len // page_size)
        keep = min(pages, slots - 1) if pin_head else pages
        if keep > slots - 1:
            raise ValueError("prefill does not fit")
        self.pinned = list(range(keep))          # logical ids, never evicted
        self.resident = []                       # decode pages, logical ids
        self.fill = {}                           # lid -> tokens
        self.created = {}                        # lid -> step
        self.used = {}                           # lid -> list of steps
        self.next_lid = pages
        self.tail = None
        self.step = prefill_len                  # absolute position of the next token
        self.evictions = []                      # (step, lid)

    def capacity_left(self) -> bool:
        return len(self.pinned) + len(self.resident) < self.S

    def decode(self, score_of):
        """score_of(lid) -> score of page lid at this step (decode pages, and
        pinned pages too when they are ranked)."""
        t = self.step
        if self.tail is None or self.fill[self.tail] == self.ps:
            assert self.capacity_left()
            lid = self.next_lid
            self.next_lid += 1
            self.resident.append(lid)
            self.fill[lid] = 0
            self.created[lid] = t
            self.used[lid] = []
            self.tail = lid
        self.fill[self.tail] += 1
        ranked = self.resident + (self.pinned if self.rank_pinned else [])
        n = len(ranked)
        k = math.floor(self.r * n)
        scores = {lid: score_of(lid) for lid in ranked}
        # "used" = among the k highest scores, counting ties at the cut as
        # not used: a page is used when at least n-k pages score strictly less
        # (only decode pages have a use to record)
        for lid in self.resident:
            below = sum(1 for o in ranked if scores[o] < scores[lid])
            if k > 0 and below >= n - k:
                self.used[lid].append(t)
        evicted = None
        if self.fill[self.tail] == self.ps and not self.capacity_left():
            def last_use(lid):
                return max([self.created[lid]] + self.used[lid])
            evicted = min(self.resident, key=lambda lid: (last_use(lid), lid))
            self.resident.remove(evicted)
            if evicted == self.tail:
                self.tail = None
            self.evictions.append((t, evicted))
        self.step = t + 1
        return evicted

    def resident_lids(self):
        return sorted(self.pinned + self.resident)

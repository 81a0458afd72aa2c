"""Simulation of the paged KV cache's page assignment.

The paper describes no cache layout; the verify step keeps each model's keys
and values in fixed-size pages (16 tokens) so that accepting or rejecting
drafts only moves a length.  Page indices are made a deterministic function of
the history of lengths by two rules:

* allocation always takes the lowest-numbered free page;
* a page is freed as soon as it holds no position below the sequence's length
  (after a commit or a rollback).

Within one call, sequences are served in the order they are listed and each
sequence's missing pages in increasing logical order.
"""

from __future__ import annotations

import heapq
from typing import Dict, List


class PageOOM(Exception):
    pass


class PagePool:
    def __init__(self, num_pages: int, page_size: int = 16):
        self.num_pages = num_pages
        self.page_size = page_size
        self.free = list(range(num_pages))
        heapq.heapify(self.free)
        self.tables: Dict[int, List[int]] = {}

    def pages_for(self, length: int) -> int:
        return (length + self.page_size - 1) // self.page_size

    def ensure(self, seq: int, length: int):
        """Make the page table of ``seq`` cover positions 0..length-1."""
        need = self.need(seq, length)
        if need > len(self.free):
            raise PageOOM(f"seq {seq} needs {need} pages, {len(self.free)} free")
        t = self.tables.setdefault(seq, [])
        for _ in range(need):
            t.append(heapq.heappop(self.free))

    def need(self, seq: int, length: int) -> int:
        return max(0, self.pages_for(length) - len(self.tables.get(seq, [])))

    def truncate(self, seq: int, length: int):
        """Free the pages of ``seq`` that hold no position below ``length``."""
        t = self.tables.get(seq, [])
        keep = self.pages_for(length)
        for pg in t[keep:]:
            heapq.heappush(self.free, pg)
        del t[keep:]

    def release(self, seq: int):
        self.truncate(seq, 0)
        self.tables.pop(seq, None)

    def slot(self, seq: int, pos: int) -> int:
        """Flat slot index page * page_size + offset of position ``pos``."""
        return self.tables[seq][pos // self.page_size] * self.page_size + pos % self.page_size

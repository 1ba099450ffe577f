"""Paged KV-cache bookkeeping (oracle).

Oracle (test infrastructure).  The paper serves requests from a vLLM-style
engine whose active-request set supplies L(t) (Section 4.2); it states no
paging policy.  Reading used here (listed in the design doc): fixed 16-token pages
drawn from one pool; a page is taken when a token lands at a length that is a
multiple of the page size; every allocation takes the lowest free page id; a
request added with a pre-filled length takes its pages in ascending id order;
cutting a request back (after a probe) returns the pages beyond the kept
length to the pool.  Allocation is all-or-nothing.  A probe may run on a fork
of a request: the fork shares the request's full pages (a page returns to the
pool when no table holds it any more) and gets a fresh lowest-id page for a
copy of the partial last page; no length may end inside a shared page.

Pinned by brute force in tests (lowest-free-id after arbitrary interleavings,
probe restore, exhaustion leaves the state unchanged).
"""
from __future__ import annotations

import heapq
from typing import Dict, List


class OutOfPages(Exception):
    pass


class PagePool:
    def __init__(self, num_pages: int, page_size: int = 16):
        self.page_size = page_size
        self.free: List[int] = list(range(num_pages))
        heapq.heapify(self.free)
        self.tables: Dict[int, List[int]] = {}
        self.lens: Dict[int, int] = {}
        self.refs: Dict[int, int] = {}

    def pages_for(self, n: int) -> int:
        return -(-n // self.page_size)

    def _take(self, count: int) -> List[int]:
        if count > len(self.free):
            raise OutOfPages(count)
        got = [heapq.heappop(self.free) for _ in range(count)]
        for pid in got:
            self.refs[pid] = 1
        return got

    def _release(self, pid: int) -> None:
        self.refs[pid] -= 1
        if self.refs[pid] == 0:
            heapq.heappush(self.free, pid)

    def add_seq(self, seq: int, length: int) -> None:
        if seq in self.tables:
            raise KeyError(seq)
        self.tables[seq] = self._take(self.pages_for(length))
        self.lens[seq] = length

    def append(self, seq: int, n: int = 1) -> None:
        """Grow a request by n tokens, taking one lowest-id page each time a page boundary is crossed."""
        need = self.pages_for(self.lens[seq] + n) - len(self.tables[seq])
        if need > len(self.free):
            raise OutOfPages(need)
        for _ in range(n):
            if self.lens[seq] % self.page_size == 0 and self.pages_for(self.lens[seq] + 1) > len(self.tables[seq]):
                self.tables[seq].extend(self._take(1))
            self.lens[seq] += 1

    def truncate(self, seq: int, length: int) -> None:
        keep = self.pages_for(length)
        if length % self.page_size and self.refs[self.tables[seq][keep - 1]] > 1:
            raise ValueError("length ends inside a shared page")
        for pid in self.tables[seq][keep:]:
            self._release(pid)
        del self.tables[seq][keep:]
        self.lens[seq] = length

    def fork(self, src: int, dst: int):
        """dst sees src's positions: full pages shared, the partial last page copied.

        Returns (src_page, dst_page) of the copy, or None when src ends on a page boundary."""
        if dst in self.tables:
            raise KeyError(dst)
        full, partial = divmod(self.lens[src], self.page_size)
        copy_to = self._take(1)[0] if partial else None
        shared = self.tables[src][:full]
        for pid in shared:
            self.refs[pid] += 1
        self.tables[dst] = list(shared) + ([copy_to] if partial else [])
        self.lens[dst] = self.lens[src]
        return (self.tables[src][full], copy_to) if partial else None

    def free_seq(self, seq: int) -> None:
        self.truncate(seq, 0)
        del self.tables[seq]
        del self.lens[seq]

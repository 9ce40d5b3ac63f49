"""Integer metadata of the batched path: varlen offsets, positions, pooling
indices and the paged draft-KV allocator (oracle; test infrastructure only).

Definitions (Section 3.1: a request is a prompt x = (x_1..x_n); Section 3.2:
static prediction after the prompt, dynamic prediction after each generated
token):

* cu_seqlens: exclusive prefix sum of the prompt lengths, cu[0] = 0, so
  request i owns packed rows [cu[i], cu[i+1]).
* positions: 0..n_i-1 for the prompt of request i; a decode step adds one
  token at position (tokens already cached).
* last_idx: cu[i+1] - 1, the row of the newest token (the "last" half of the
  pooled head input); the mean half pools rows [cu[i], cu[i+1]).

Page allocation of the draft KV cache (the paper leaves it open; this is the
rule both sides implement so the tables are unique):

* the pool holds pages 0..num_pages-1 of ``page_size`` tokens;
* a free page is always the lowest free id;
* a prefill allocates ceil(n_i / page_size) pages per request, requests in
  argument order, pages of one request in increasing token order;
* a decode step allocates one page for a request exactly when its cached
  length is a multiple of page_size before the append, in argument order;
* release returns a slot's pages to the free set and clears its row.

Validation happens before any change, so a call that fails leaves the state
as it was.  Checks and error codes, in the order they are applied:

prefill: n < 0 -> INVALID_ARG; then for each request in order: slot outside
  [0, max_slots) or repeated in the call -> INVALID_ARG, length <= 0 or
  > max_seq_len -> INVALID_ARG; then any slot already active -> SLOT_BUSY;
  then pages needed > pages free -> OUT_OF_PAGES.
step: n < 0 -> INVALID_ARG; for each request: bad or repeated slot ->
  INVALID_ARG; then any slot inactive -> SLOT_EMPTY; then any cached length
  already max_seq_len -> INVALID_ARG; then pages needed > free -> OUT_OF_PAGES.
release: bad or repeated slot -> INVALID_ARG (inactive slots are a no-op).
"""
from __future__ import annotations

import heapq
from typing import List, Sequence

import numpy as np

OK = 0
ERR_INVALID_ARG = -1
ERR_SLOT_BUSY = -2
ERR_SLOT_EMPTY = -3
ERR_OUT_OF_PAGES = -4


def cu_seqlens(lens: Sequence[int]) -> np.ndarray:
    out = [0]
    for n in lens:
        out.append(out[-1] + int(n))
    return np.array(out, dtype=np.int32)


def positions(lens: Sequence[int], start: Sequence[int] = None) -> np.ndarray:
    """Packed positions; ``start[i]`` (default 0) is request i's first position."""
    out: List[int] = []
    for i, n in enumerate(lens):
        s = 0 if start is None else int(start[i])
        out.extend(range(s, s + int(n)))
    return np.array(out, dtype=np.int32)


def last_idx(lens: Sequence[int]) -> np.ndarray:
    cu = cu_seqlens(lens)
    return (cu[1:] - 1).astype(np.int32)


def pages_for(n_tokens: int, page_size: int) -> int:
    return -(-int(n_tokens) // page_size)


class PageAllocator:
    def __init__(self, num_pages: int, page_size: int, max_slots: int, max_seq_len: int):
        self.num_pages = num_pages
        self.page_size = page_size
        self.max_slots = max_slots
        self.max_seq_len = max_seq_len
        self.max_pages_per_seq = pages_for(max_seq_len, page_size)
        self.free = list(range(num_pages))        # a min-heap of free ids
        heapq.heapify(self.free)
        self.pages: List[List[int]] = [[] for _ in range(max_slots)]
        self.seq_len = [0] * max_slots
        self.active = [False] * max_slots

    def _check_slots(self, slots) -> int:
        seen = set()
        for s in slots:
            s = int(s)
            if s < 0 or s >= self.max_slots or s in seen:
                return ERR_INVALID_ARG
            seen.add(s)
        return OK

    def prefill(self, slots: Sequence[int], lens: Sequence[int]) -> int:
        if len(slots) != len(lens):
            return ERR_INVALID_ARG
        seen = set()
        for s, n in zip(slots, lens):
            s, n = int(s), int(n)
            if s < 0 or s >= self.max_slots or s in seen:
                return ERR_INVALID_ARG
            seen.add(s)
            if n <= 0 or n > self.max_seq_len:
                return ERR_INVALID_ARG
        if any(self.active[int(s)] for s in slots):
            return ERR_SLOT_BUSY
        need = sum(pages_for(n, self.page_size) for n in lens)
        if need > len(self.free):
            return ERR_OUT_OF_PAGES
        for s, n in zip(slots, lens):
            s = int(s)
            self.pages[s] = [heapq.heappop(self.free) for _ in range(pages_for(n, self.page_size))]
            self.seq_len[s] = int(n)
            self.active[s] = True
        return OK

    def step(self, slots: Sequence[int]) -> int:
        rc = self._check_slots(slots)
        if rc != OK:
            return rc
        if any(not self.active[int(s)] for s in slots):
            return ERR_SLOT_EMPTY
        if any(self.seq_len[int(s)] >= self.max_seq_len for s in slots):
            return ERR_INVALID_ARG
        need = sum(1 for s in slots if self.seq_len[int(s)] % self.page_size == 0)
        if need > len(self.free):
            return ERR_OUT_OF_PAGES
        for s in slots:
            s = int(s)
            if self.seq_len[s] % self.page_size == 0:
                self.pages[s].append(heapq.heappop(self.free))
            self.seq_len[s] += 1
        return OK

    def release(self, slots: Sequence[int]) -> int:
        rc = self._check_slots(slots)
        if rc != OK:
            return rc
        for s in slots:
            s = int(s)
            for p in self.pages[s]:
                heapq.heappush(self.free, p)
            self.pages[s] = []
            self.seq_len[s] = 0
            self.active[s] = False
        return OK

    def table(self) -> np.ndarray:
        t = np.full((self.max_slots, self.max_pages_per_seq), -1, dtype=np.int32)
        for s, pg in enumerate(self.pages):
            t[s, :len(pg)] = pg
        return t

    def seq_lens(self) -> np.ndarray:
        return np.array(self.seq_len, dtype=np.int32)

    def n_free(self) -> int:
        return len(self.free)

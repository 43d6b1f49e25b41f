"""Oracle of the virtual-address chunk pool (Section 4).

Test infrastructure.  Device memory is a cache of equal physical chunks of
``m_c`` bytes.  A request of ``m_r`` bytes gets ``k = ceil(m_r / m_c)`` chunks,
taken from the cache in any order and mapped one after another into a fresh
contiguous virtual range of ``m_a = k m_c`` bytes; freeing releases the range
and returns the chunks to the cache.  Because chunks can be combined in any
order there is no external fragmentation, and the only waste is the internal
fragmentation ``m_a - m_r < m_c`` per request (eq. 1), at most ``N_max m_c``
in total for ``N_max`` live requests (eq. 2).

The cache hands out the lowest-numbered free chunks first, which makes the
chunk assignment of a schedule deterministic.
"""

from __future__ import annotations

import heapq
from collections import deque

SWAPIN, ALLOC, CANCEL, WAIT_OUT, SWAPOUT, FREE = 0, 1, 2, 3, 4, 5


class OutOfChunks(Exception):
    pass


class VAPool:
    def __init__(self, n_chunks, chunk):
        self.chunk = chunk
        self.n_chunks = n_chunks
        self.free = list(range(n_chunks))
        heapq.heapify(self.free)
        self.ranges = {}          # range id -> (requested bytes, [chunk ids])
        self.next_id = 0

    def alloc(self, m_r):
        k = -(-m_r // self.chunk)
        if k > len(self.free):
            raise OutOfChunks(f"need {k} chunks, {len(self.free)} free")
        chunks = [heapq.heappop(self.free) for _ in range(k)]
        rid = self.next_id
        self.next_id += 1
        self.ranges[rid] = (m_r, chunks)
        return rid, chunks

    def release(self, rid):
        _, chunks = self.ranges.pop(rid)
        for c in chunks:
            heapq.heappush(self.free, c)

    def mapped_bytes(self):
        return sum(len(c) for _, c in self.ranges.values()) * self.chunk

    def requested_bytes(self):
        return sum(m for m, _ in self.ranges.values())


def assign(ops, var_bytes, n_chunks, chunk):
    """Replay a schedule's ops through the pool.

    Every SWAPIN or ALLOC opens a residency interval of one device copy; FREE
    closes the variable's working copy, WAIT_OUT the oldest pending copy (the
    swap-out queue order), CANCEL turns a pending copy back into the working
    one.  Returns the intervals in opening order as dicts
    ``{"var", "open", "close", "chunks"}`` (op indices; close = None if never
    closed) and the most chunks in use at once.
    """
    pool = VAPool(n_chunks, chunk)
    intervals = []
    working = {}               # var -> interval index
    pending = deque()          # interval indices with a swap-out issued, oldest first
    max_used = 0
    for k, (_, _, kind, u) in enumerate(ops):
        if kind in (SWAPIN, ALLOC):
            rid, chunks = pool.alloc(var_bytes[u])
            intervals.append({"var": u, "open": k, "close": None, "chunks": chunks, "rid": rid})
            working[u] = len(intervals) - 1
        elif kind == SWAPOUT:
            pending.append(working.pop(u))
        elif kind == CANCEL:
            j = next(j for j in pending if intervals[j]["var"] == u)
            pending.remove(j)
            working[u] = j
        elif kind == WAIT_OUT:
            j = pending.popleft()
            assert intervals[j]["var"] == u
            intervals[j]["close"] = k
            pool.release(intervals[j]["rid"])
        elif kind == FREE:
            j = working.pop(u)
            intervals[j]["close"] = k
            pool.release(intervals[j]["rid"])
        max_used = max(max_used, n_chunks - len(pool.free))
    for iv in intervals:
        del iv["rid"]
    return intervals, max_used

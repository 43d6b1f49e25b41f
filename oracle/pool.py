"""Oracle of the virtual-address chunk pool (Section 4).

Test infrastructure.  Device memory is a cache of equal physical chunks of
``m_c`` bytes.  A request of ``m_r`` bytes gets ``k = ceil(m_r / m_c)`` chunks,
taken from the cache in any order and mapped one after another into a fresh
contiguous virtual range of ``m_a = k m_c`` bytes; freeing releases the range
and returns the chunks to the cache.  Because chunks can be combined in any
order there is no external fragmentation, and the only waste is the internal
fragmentation ``m_a - m_r < m_c`` per request (eq. 1), at most ``N_max m_c``
in total for ``N_max`` live requests (eq. 2).

The cache hands out freed chunks in the order they were freed (the least
recently freed first), and a chunk never used before (lowest id first) only
when no freed chunk is left.  This makes the chunk assignment of a schedule
deterministic.
"""

from __future__ import annotations

from collections import deque

SWAPIN, ALLOC, CANCEL, WAIT_OUT, SWAPOUT, FREE = 0, 1, 2, 3, 4, 5


class OutOfChunks(Exception):
    pass


class VAPool:
    def __init__(self, n_chunks, chunk):
        self.chunk = chunk
        self.n_chunks = n_chunks
        self.freed = deque()      # released chunks, oldest release first
        self.unused = 0           # chunks [unused, n_chunks) were never handed out
        self.ranges = {}          # range id -> (requested bytes, [chunk ids])
        self.next_id = 0

    @property
    def free(self):
        """Every chunk not in use: the freed ones in queue order, then the unused ones."""
        return list(self.freed) + list(range(self.unused, self.n_chunks))

    def alloc(self, m_r):
        k = -(-m_r // self.chunk)
        if k > len(self.freed) + self.n_chunks - self.unused:
            raise OutOfChunks(f"need {k} chunks, {len(self.freed) + self.n_chunks - self.unused} free")
        chunks = []
        for _ in range(k):
            if self.freed:
                chunks.append(self.freed.popleft())
            else:
                chunks.append(self.unused)
                self.unused += 1
        rid = self.next_id
        self.next_id += 1
        self.ranges[rid] = (m_r, chunks)
        return rid, chunks

    def release(self, rid):
        _, chunks = self.ranges.pop(rid)
        self.freed.extend(chunks)

    def mapped_bytes(self):
        return sum(len(c) for _, c in self.ranges.values()) * self.chunk

    def requested_bytes(self):
        return sum(m for m, _ in self.ranges.values())


def assign(ops, var_bytes, n_chunks, chunk):
    """Replay a schedule's ops through the pool.

    Every SWAPIN or ALLOC opens a residency interval of one device copy; FREE
    closes the variable's working copy, WAIT_OUT the variable's oldest pending
    copy, CANCEL turns a pending copy back into the working one.  Returns the intervals in opening order as dicts
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
            j = next(j for j in pending if intervals[j]["var"] == u)
            pending.remove(j)
            intervals[j]["close"] = k
            pool.release(intervals[j]["rid"])
        elif kind == FREE:
            j = working.pop(u)
            intervals[j]["close"] = k
            pool.release(intervals[j]["rid"])
        max_used = max(max_used, pool.unused - len(pool.freed))     # chunks in use
    for iv in intervals:
        del iv["rid"]
    return intervals, max_used


def best_fit(ops, var_bytes, align=256, placements=None):
    """Replay a schedule's device copies through one contiguous best-fit heap.

    The comparison point of Section 4: an allocator that hands out contiguous
    address ranges (as a caching allocator on top of one device allocation
    does) suffers external fragmentation, so the address range it needs can
    exceed the bytes live at any moment.  Each residency interval (the same
    copies as ``assign``: SWAPIN / ALLOC open one, FREE closes the working
    copy, WAIT_OUT the variable's oldest pending one, CANCEL makes a pending copy the
    working one again) asks for its size rounded up to ``align``.  A request
    takes the smallest free hole that holds it (lowest address on ties); when
    no hole does, it goes to the end of the heap, starting inside the free tail
    if there is one.  Returns ``(extent, peak_live)``: the highest address ever
    used and the most bytes live at once.  ``placements``, if a list, receives
    ``(op index, offset, size)`` per request and ``(op index, None, size)`` per
    release.
    """
    holes = []                 # [offset, size], sorted by offset, disjoint, not adjacent
    heap_end = 0
    live = peak = 0
    blocks = {}                # interval id -> (offset, size, var)
    working, pending = {}, deque()

    def alloc(size):
        nonlocal heap_end
        fit = [h for h in holes if h[1] >= size]
        if fit:
            h = min(fit, key=lambda x: (x[1], x[0]))
            off = h[0]
            h[0] += size
            h[1] -= size
            if h[1] == 0:
                holes.remove(h)
            return off
        if holes and holes[-1][0] + holes[-1][1] == heap_end:
            off = holes.pop()[0]
        else:
            off = heap_end
        heap_end = off + size
        return off

    def release(off, size):
        holes.append([off, size])
        holes.sort()
        merged = []
        for h in holes:
            if merged and merged[-1][0] + merged[-1][1] == h[0]:
                merged[-1][1] += h[1]
            else:
                merged.append(h)
        holes[:] = merged

    for k, (_, _, kind, u) in enumerate(ops):
        if kind in (SWAPIN, ALLOC):
            size = -(-var_bytes[u] // align) * align
            blocks[k] = (alloc(size), size, u)
            if placements is not None:
                placements.append((k, blocks[k][0], size))
            working[u] = k
            live += size
            peak = max(peak, live)
        elif kind == SWAPOUT:
            pending.append(working.pop(u))
        elif kind == CANCEL:
            j = next(j for j in pending if blocks[j][2] == u)
            pending.remove(j)
            working[u] = j
        elif kind in (WAIT_OUT, FREE):
            if kind == WAIT_OUT:
                j = next(j for j in pending if blocks[j][2] == u)
                pending.remove(j)
            else:
                j = working.pop(u)
            off, size, _ = blocks.pop(j)
            release(off, size)
            if placements is not None:
                placements.append((k, None, off))
            live -= size
    return heap_end, peak

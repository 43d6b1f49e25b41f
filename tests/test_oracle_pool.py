"""Pins of the oracle VA pool (Section 4): eq. 1, eq. 2, no external fragmentation; and of the
contiguous best-fit heap it is compared with."""

import random

import pytest

from oracle import pool as P
from oracle import schedule as S
from oracle.lower import lower, as_schedule_input
from paper_2010_14109_amd import synth


def test_eq1_internal_fragmentation_below_one_chunk():
    pool = P.VAPool(10 ** 6, 4096)
    for m_r in [1, 4095, 4096, 4097, 10 ** 6, 123457, 8192]:
        rid, chunks = pool.alloc(m_r)
        m_a = len(chunks) * pool.chunk
        assert 0 <= m_a - m_r < pool.chunk
        assert len(chunks) == -(-m_r // pool.chunk)


def test_eq2_and_no_external_fragmentation_adversarial():
    """After any alloc/free history, a request fits iff it needs no more chunks than are
    free (no external fragmentation), and mapped - requested < live * m_c (eq. 2)."""
    rng = random.Random(1)
    m_c = 64
    pool = P.VAPool(200, m_c)
    live = []
    for _ in range(5000):
        if live and rng.random() < 0.45:
            pool.release(live.pop(rng.randrange(len(live))))
        else:
            m_r = rng.randint(1, 40 * m_c)
            k = -(-m_r // m_c)
            if k <= len(pool.free):
                rid, chunks = pool.alloc(m_r)
                live.append(rid)
            else:
                with pytest.raises(P.OutOfChunks):
                    pool.alloc(m_r)
        waste = pool.mapped_bytes() - pool.requested_bytes()
        assert 0 <= waste < max(1, len(live)) * m_c or (not live and waste == 0)
        # chunks of live ranges are disjoint
        used = [c for _, cs in pool.ranges.values() for c in cs]
        assert len(used) == len(set(used))
        assert len(used) + len(pool.free) == pool.n_chunks


@pytest.mark.parametrize("policy", ["C", "L"])
def test_schedule_assignment_fits_budget(policy):
    spec = synth.resnet(batch=2, hw=32, classes=7, blocks=(1, 1, 1, 1), width=4)
    b, k, f = as_schedule_input(lower(spec))
    chunk = 512
    p = S.incore_peak(b, k, f, chunk)
    for frac in (1.0, 0.5, 0.25, 0.1):
        B = max(S.budget_for(frac, p, chunk), S.working_set_max(b, f, chunk))
        out = S.build(b, k, f, B, B // 2, chunk, policy)
        n_chunks = B // chunk
        ivs, max_used = P.assign(out["ops"], b, n_chunks, chunk)
        assert max_used * chunk <= B
        assert max_used * chunk == out["peak"]
        # every interval has exactly ceil(b/m_c) chunks and none is shared while both live
        events = []
        for j, iv in enumerate(ivs):
            assert len(iv["chunks"]) == -(-b[iv["var"]] // chunk)
            assert iv["close"] is not None
            events.append((iv["open"], 1, j))
            events.append((iv["close"], 0, j))
        owner = {}
        for _, kind, j in sorted(events):
            for c in ivs[j]["chunks"]:
                if kind == 1:
                    assert c not in owner
                    owner[c] = j
                else:
                    assert owner.pop(c) == j


# ---------------------------------------------------------------- best-fit comparison heap
def test_best_fit_hand_example():
    """A = B = 4, C = 8 bytes: after A is freed its 4-byte hole cannot take C, so C goes above B
    (extent 16 although at most 12 bytes are live); the next 4-byte request takes the smallest
    hole that fits."""
    ops = [(0, 0, S.ALLOC, 0), (0, 0, S.ALLOC, 1), (0, 1, S.FREE, 0), (1, 0, S.ALLOC, 2),
           (1, 1, S.FREE, 1), (2, 0, S.ALLOC, 0)]
    trace = []
    assert P.best_fit(ops, [4, 4, 8], 1, trace) == (16, 12)
    assert [t for t in trace if t[1] is not None] == [(0, 0, 4), (1, 4, 4), (3, 8, 8), (5, 0, 4)]


def _check_best_fit(ops, sizes, align):
    """Brute force: recompute the free intervals from the live blocks at every request and check
    the placement against the best-fit rule; blocks never overlap; extent >= peak live."""
    trace = []
    extent, peak = P.best_fit(ops, sizes, align, trace)
    live = {}                      # offset -> size
    end = 0
    peak_seen = 0
    for k, off, size in trace:
        if off is None:
            del live[size]         # release: the third field holds the block's offset
            continue
        spans = sorted(live.items())
        free, cur = [], 0
        for o, sz in spans:
            if o > cur:
                free.append((cur, o - cur))
            cur = max(cur, o + sz)
        if cur < end:
            free.append((cur, end - cur))      # the free tail is a hole like any other
        fits = [f for f in free if f[1] >= size]
        if fits:
            assert off == min(fits, key=lambda f: (f[1], f[0]))[0]
        else:
            tail = cur if cur < end else end
            assert off == tail
        for o, sz in spans:
            assert off + size <= o or o + sz <= off
        live[off] = size
        end = max(end, off + size)
        peak_seen = max(peak_seen, sum(live.values()))
    assert extent == end and peak == peak_seen and extent >= peak
    return extent, peak


@pytest.mark.parametrize("policy", ["C", "L"])
def test_best_fit_replays_network_schedules(policy):
    for spec in (synth.mlp(batch=4, width=16, depth=4, classes=5),
                 synth.resnet(batch=2, hw=32, classes=7, blocks=(1, 2, 1, 1), width=4)):
        b, k, f = as_schedule_input(lower(spec))
        p = S.incore_peak(b, k, f, 1)
        ws = S.working_set_max(b, f, 1)
        for frac in (0.6, 0.3):
            out = S.build(b, k, f, max(S.budget_for(frac, p, 1), ws), 0, 1, policy)
            _check_best_fit(out["ops"], b, 256)


def test_best_fit_equal_sizes_do_not_fragment():
    rng = random.Random(3)
    for _ in range(50):
        n = rng.randint(2, 12)
        kinds = [S.TEMP] * n
        fns = []
        produced = [False] * n
        for _ in range(rng.randint(3, 20)):
            vs = rng.sample(range(n), rng.randint(1, min(3, n)))
            fns.append([(v, S.RW if produced[v] else S.W) for v in vs])
            for v in vs:
                produced[v] = True
        sizes = [512] * n
        ws = S.working_set_max(sizes, fns, 1)
        out = S.build(sizes, kinds, fns, ws + rng.randint(0, 3) * 512, 0, 1, rng.choice("CL"))
        extent, peak = _check_best_fit(out["ops"], sizes, 256)
        assert extent == peak

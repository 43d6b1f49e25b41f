"""Pins of the oracle VA pool (Section 4): eq. 1, eq. 2, no external fragmentation."""

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

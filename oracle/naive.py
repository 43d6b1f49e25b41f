"""The naive out-of-core schedule (Section 1): transfer before and after every layer.

Test infrastructure.  Built directly from its description, without the
window scheduler: before ``f_i`` every variable of ``f_i`` that already has a
value is copied to the device (a variable that ``f_i`` produces first is only
allocated); after ``f_i`` every variable of ``f_i`` that a later function uses,
or whose final value belongs on the host (PARAM, STATE, OUTPUT), is copied back.
Nothing stays on the device between two functions.
"""

from __future__ import annotations

from collections import Counter

INPUT, PARAM, STATE, OUTPUT, TEMP = 0, 1, 2, 3, 4


def transfers(var_kinds, fn_vars):
    """Multiset of transfers: ``Counter({("in", i, v): 1, ("out", i, v): 1, ...})``."""
    seen = set(v for v, k in enumerate(var_kinds) if k in (INPUT, PARAM, STATE))
    used_at = {}
    for i, vs in enumerate(fn_vars):
        for v, _ in vs:
            used_at.setdefault(v, []).append(i)
    out = Counter()
    for i, vs in enumerate(fn_vars):
        names = []
        for v, _ in vs:
            if v not in names:
                names.append(v)
        for v in names:
            if v in seen:
                out[("in", i, v)] += 1
        for v in names:
            seen.add(v)
            later = any(j > i for j in used_at[v])
            if later or var_kinds[v] in (PARAM, STATE, OUTPUT):
                out[("out", i, v)] += 1
    return out


def working_set(var_bytes, fn_vars, chunk=1):
    """Largest chunk-rounded footprint of one function: the naive schedule's peak."""
    best = 0
    for vs in fn_vars:
        names = set(v for v, _ in vs)
        best = max(best, sum(-(-var_bytes[v] // chunk) * chunk for v in names))
    return best

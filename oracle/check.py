"""Independent replayer of a swap schedule (test infrastructure).

Given a function sequence and an op list, it re-derives everything from the
ops alone -- without the scheduler's window logic -- and fails on the first op
that breaks one of the rules the paper's procedure must keep (Section 3,
Fig. 2; Section 4 for the budget):

* the device never holds more than the budget (chunk-rounded bytes, eq. 1);
* before ``f_i`` runs, every variable it uses is on the device and holds the
  newest value of that variable (swap-ins read host copies that are current);
* swap-outs are completed oldest first (or, with ``wait="furthest"``, a budget
  wait completes the earliest pending swap-out whose variable is used again
  furthest ahead, positions counted in the variable-sequence);
* at the end of the step nothing is left on the device and every PARAM, STATE
  and OUTPUT variable has its final value on the host.

It tracks data versions: every write of a variable makes a new version, a
swap-out carries the device version to the host, a swap-in the host version
to the device.
"""

from __future__ import annotations

from collections import deque

R_, W_ = 1, 2
INPUT, PARAM, STATE, OUTPUT, TEMP = 0, 1, 2, 3, 4
SWAPIN, ALLOC, CANCEL, WAIT_OUT, SWAPOUT, FREE = 0, 1, 2, 3, 4, 5
PRE, POST, END = 0, 1, 2


class ScheduleError(AssertionError):
    pass


def _merge(vs):
    acc = {}
    for v, a in vs:
        acc[v] = acc.get(v, 0) | a
    order = []
    for v, _ in vs:
        if v not in order:
            order.append(v)
    return [(v, acc[v]) for v in order]


def replay(var_bytes, var_kinds, fn_vars, ops, budget, chunk=1, policy="C", held=None,
           wait="oldest"):
    """Check an op list; returns ``{"peak", "h2d", "d2h", "max_live"}`` or raises ScheduleError."""
    fns = [_merge(vs) for vs in fn_vars]
    N = len(fns)
    nv = len(var_bytes)
    size = [-(-b // chunk) * chunk for b in var_bytes]
    uses = [[i for i, vs in enumerate(fns) if any(v == u for v, _ in vs)] for u in range(nv)]
    start = [0] * (N + 1)              # position of each function's first variable
    for i, vs in enumerate(fns):
        start[i + 1] = start[i] + len(vs)

    def next_position(u, i):
        """Position of the first use of u by a function after f_i (infinity if none)."""
        for j in uses[u]:
            if j > i:
                return start[j] + [v for v, _ in fns[j]].index(u)
        return float("inf")

    version = [0] * nv                 # newest value of each variable
    host_ver = [0 if var_kinds[u] in (INPUT, PARAM, STATE) else None for u in range(nv)]
    working = [None] * nv              # version held by the working device copy, or None
    pending = deque()                  # (var, version, next use) of issued swap-outs, oldest first
    cur = 0
    h2d = d2h = 0
    peak = 0
    max_live = 0
    pos = 0                            # next function expected to run
    ran = [False] * N

    def fail(k, msg):
        raise ScheduleError(f"op {k} {ops[k] if k < len(ops) else ''}: {msg}")

    def run_until(i, k):
        """Run functions pos..i-1 (all of their ops must already have been seen)."""
        nonlocal pos
        while pos < i:
            execute(pos, k)
            pos += 1

    def execute(i, k):
        for u, a in fns[i]:
            if working[u] is None:
                fail(k, f"f{i} runs without variable {u} on the device")
            if a & R_ and working[u] != version[u]:
                fail(k, f"f{i} reads a stale copy of variable {u}")
            if a & W_:
                version[u] += 1
                working[u] = version[u]
        ran[i] = True

    phase_of = {}
    last_key = (-1, -1)
    for k, (i, phase, kind, u) in enumerate(ops):
        if not (0 <= u < nv):
            fail(k, "unknown variable")
        key = (i, phase)
        if key < last_key:
            fail(k, "ops are out of function/phase order")
        last_key = key
        if phase == END:
            if i != N:
                fail(k, "END op must carry fn = N")
            run_until(N, k)
        elif phase == PRE:
            run_until(i, k)
        elif phase == POST:
            run_until(i + 1, k)
            if not any(v == u for v, _ in fns[i]):
                fail(k, f"POST op of f{i} on a variable it does not use")
        else:
            fail(k, "bad phase")
        phase_of[k] = phase

        if kind == SWAPIN:
            if phase != PRE:
                fail(k, "swap-in outside a PRE phase")
            if working[u] is not None:
                fail(k, "swap-in of a variable already on the device")
            if policy == "C" and any(p[0] == u for p in pending):
                fail(k, "swap-in of a variable whose swap-out is pending (policy C cancels)")
            if host_ver[u] is None or host_ver[u] != version[u]:
                fail(k, "swap-in of a variable whose host copy is not current")
            working[u] = host_ver[u]
            cur += size[u]
            h2d += var_bytes[u]
        elif kind == ALLOC:
            if phase != PRE:
                fail(k, "alloc outside a PRE phase")
            if working[u] is not None or version[u] != 0 or host_ver[u] is not None:
                fail(k, "alloc of a variable that already has a value")
            working[u] = 0
            cur += size[u]
        elif kind == CANCEL:
            if policy != "C":
                fail(k, "cancel under policy L")
            idx = [j for j, p in enumerate(pending) if p[0] == u]
            if not idx or working[u] is not None:
                fail(k, "cancel of a variable without a pending swap-out")
            _, ver, _ = pending[idx[0]]
            del pending[idx[0]]
            working[u] = ver
        elif kind == WAIT_OUT:
            if phase == POST:
                fail(k, "wait in a POST phase")
            if not pending:
                fail(k, "wait with no pending swap-out")
            j = 0
            if wait == "furthest" and phase == PRE:
                far = max(p[2] for p in pending)
                j = next(q for q, p in enumerate(pending) if p[2] == far)
            w = pending[j][0]
            del pending[j]
            if w != u:
                fail(k, f"wait for {u} but the pending swap-out to complete is {w}")
            cur -= size[u]
        elif kind == SWAPOUT:
            if phase != POST:
                fail(k, "swap-out outside a POST phase")
            if working[u] is None:
                fail(k, "swap-out of a variable not on the device")
            pending.append((u, working[u], next_position(u, i)))
            host_ver[u] = working[u]
            working[u] = None
            d2h += var_bytes[u]
        elif kind == FREE:
            if phase != POST:
                fail(k, "free outside a POST phase")
            if working[u] is None:
                fail(k, "free of a variable not on the device")
            if var_kinds[u] not in (INPUT, TEMP):
                fail(k, "free of a PARAM/STATE/OUTPUT variable (it must be written back)")
            if any(j > i for j in uses[u]):
                fail(k, f"free of variable {u} that f{[j for j in uses[u] if j > i][0]} uses later")
            working[u] = None
            cur -= size[u]
        else:
            fail(k, "bad op kind")
        if cur > budget:
            fail(k, f"device holds {cur} > budget {budget}")
        if held is not None and held[k] != cur:
            fail(k, f"reported held {held[k]} != replayed {cur}")
        peak = max(peak, cur)
        live = sum(1 for u in range(nv) if working[u] is not None) + len(pending)
        max_live = max(max_live, live)
    run_until(N, len(ops))
    if pending:
        raise ScheduleError("swap-outs still pending at the end")
    for u in range(nv):
        if working[u] is not None:
            raise ScheduleError(f"variable {u} still on the device at the end")
        if var_kinds[u] in (PARAM, STATE, OUTPUT) and version[u] > 0 and host_ver[u] != version[u]:
            raise ScheduleError(f"final value of variable {u} never reached the host")
    if not all(ran):
        raise ScheduleError("some function never ran")
    return {"peak": peak, "h2d": h2d, "d2h": d2h, "max_live": max_live}


def resident_before(fn_vars, ops, i):
    """Variables on the device right before f_i runs (working copies and pending swap-outs)."""
    dev = set()
    pend = []
    for (j, phase, kind, u) in ops:
        if (j, phase) > (i, PRE):
            break
        if kind in (SWAPIN, ALLOC):
            dev.add(u)
        elif kind == CANCEL:
            pend.remove(u)
            dev.add(u)
        elif kind == SWAPOUT:
            dev.discard(u)
            pend.append(u)
        elif kind == WAIT_OUT:
            pend.remove(u)
        elif kind == FREE:
            dev.discard(u)
    return dev, set(pend)

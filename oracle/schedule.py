"""Oracle of the adaptive-window swap scheduler (Section 3, Fig. 2).

Test infrastructure: only ``tests/``, ``smoke()`` and the CPU-baseline leg of
``bench.py`` use it.

The paper's objects and how they appear here:

* function-sequence ``[f_1..f_N]`` and, per function, the variables it uses
  ``V_i`` (Section 2 and 3): ``fn_vars[i] = [(var, access), ...]`` in
  registered order, duplicates merged (first position kept, accesses or-ed);
* variable-sequence ``v = flatten([V_1..V_N])`` with repeats (Section 3):
  ``seq`` (one entry per position), ``first[i]`` / ``last[i]`` = positions of
  the first and last variable of ``f_i`` (``l`` and ``e`` below);
* sizes ``b_v`` in bytes; budget accounting uses the chunk-rounded
  ``a_v = ceil(b_v / m_c) * m_c`` of Section 4 (eq. 1) so that the physical
  pool never holds more than the budget;
* state ``sigma(v)`` (1 = on the CPU).  The paper's state is binary; the
  oracle splits "on the GPU" into DEV and PEND (a swap-out issued but not yet
  waited for) and "on the CPU" into HOST and UNMAT (never produced yet).

Per function ``f_i`` the procedure of Section 3 / Fig. 2 runs:

1. schedule-window: ``r`` is the largest index with
   ``sum(b_{v[p]} for p in l..r) <= W`` (positional sum, repeats counted);
   the window always covers ``f_i``'s own variables and never moves back;
2. step (a) swap-in of every variable entering the window that is on the CPU,
   step (b) completion of the oldest pending swap-outs until the new
   residents fit in the budget (the wait sits right before ``f_i``);
3. ``f_i`` runs;
4. step (c) swap-out reservation for the variables of ``f_i``, with the skips
   of step (d): no swap-out for variables never used again, nor for
   variables already inside the window.

Readings of the paper where it is silent (stated once, used throughout):

* a variable that re-enters the window while its swap-out is pending keeps
  its device copy (the swap-out is cancelled, policy "C"); policy "L" takes
  the binary state literally: the variable is already on the CPU, so it is
  swapped in again into fresh memory after its swap-out completes;
* a variable first produced inside the window is allocated (no transfer);
* at its last use an INPUT or TEMP variable is freed, a PARAM, STATE or
  OUTPUT variable is written back (swap-out) so the host holds the result;
* when the budget cannot be met even with no pending swap-out left, the
  window is cut short before the variable that does not fit; the call fails
  only if a variable of ``f_i`` itself does not fit (infeasible budget);
* swap-outs of one function are reserved in registered order; "oldest" is
  the order of reservation.
"""

from __future__ import annotations

import math
from collections import deque

# access flags
R, W, RW = 1, 2, 3
# variable kinds
INPUT, PARAM, STATE, OUTPUT, TEMP = 0, 1, 2, 3, 4
PERSISTENT = (INPUT, PARAM, STATE)       # valid on the host when a step starts
WRITE_BACK = (PARAM, STATE, OUTPUT)      # must be on the host when a step ends
# op kinds and phases
SWAPIN, ALLOC, CANCEL, WAIT_OUT, SWAPOUT, FREE = 0, 1, 2, 3, 4, 5
PRE, POST, END = 0, 1, 2
OP_NAMES = ["SWAPIN", "ALLOC", "CANCEL", "WAIT_OUT", "SWAPOUT", "FREE"]
# variable states
UNMAT, HOST, DEV, PEND = "UNMAT", "HOST", "DEV", "PEND"

INCORE = 2 ** 64 - 1   # budget / window value meaning "no limit"


class Infeasible(Exception):
    """The budget cannot hold the variables of one function."""


class Invalid(Exception):
    """The registration breaks a rule of the function sequence."""


def rounded(nbytes, chunk):
    """Chunk-rounded allocation size a = ceil(b / m_c) * m_c (Section 4, eq. 1)."""
    return -(-nbytes // chunk) * chunk


def normalize(fn_vars):
    """Merge repeated variables inside one function: first position, accesses or-ed."""
    out = []
    for vs in fn_vars:
        seen = {}
        order = []
        for v, a in vs:
            if v in seen:
                seen[v] |= a
            else:
                seen[v] = a
                order.append(v)
        out.append([(v, seen[v]) for v in order])
    return out


def validate(var_bytes, var_kinds, fn_vars):
    """Rules of a well-formed function sequence; raises ``Invalid``."""
    nv = len(var_bytes)
    if len(var_kinds) != nv:
        raise Invalid("sizes and kinds differ in length")
    for v in range(nv):
        if var_bytes[v] <= 0:
            raise Invalid(f"variable {v} has no bytes")
        if var_kinds[v] not in (INPUT, PARAM, STATE, OUTPUT, TEMP):
            raise Invalid(f"variable {v} has unknown kind {var_kinds[v]}")
    produced = [var_kinds[v] in PERSISTENT for v in range(nv)]
    for i, vs in enumerate(fn_vars):
        if not vs:
            raise Invalid(f"function {i} uses no variable")
        for v, a in vs:
            if not (0 <= v < nv):
                raise Invalid(f"function {i} names unknown variable {v}")
            if a not in (R, W, RW):
                raise Invalid(f"function {i} has bad access {a}")
            if var_kinds[v] == INPUT and a & W:
                raise Invalid(f"function {i} writes input variable {v}")
            if not produced[v] and a != W:
                raise Invalid(f"function {i} reads variable {v} before it is written")
            produced[v] = True


def sequence(fn_vars):
    """Variable-sequence v = flatten([V_1..V_N]) and each function's first/last position."""
    seq, first, last = [], [], []
    for vs in fn_vars:
        first.append(len(seq))
        for v, _ in vs:
            seq.append(v)
        last.append(len(seq) - 1)
    return seq, first, last


def next_use(seq, first, last):
    """For each function i and each of its variables: position of the next use after f_i.

    ``nxt[i][v]`` is the smallest position p > last[i] with seq[p] == v, or None.
    """
    n = len(first)
    nxt = []
    for i in range(n):
        d = {}
        for p in range(first[i], last[i] + 1):
            v = seq[p]
            q = last[i] + 1
            while q < len(seq) and seq[q] != v:
                q += 1
            d[v] = q if q < len(seq) else None
        nxt.append(d)
    return nxt


def window_end(seq, sizes, l, window):
    """Largest r >= l-1 with sum(b_{v[p]}, p = l..r) <= window (Section 3)."""
    total = 0
    r = l - 1
    for p in range(l, len(seq)):
        total += sizes[seq[p]]
        if total > window:
            break
        r = p
    return r


def build(var_bytes, var_kinds, fn_vars, budget, window, chunk=1, policy="C", ahead=None,
          threshold=None, wait="oldest"):
    """Schedule one training step.  Returns a dict:

    ``ops``      list of (fn, phase, kind, var) in emission order (fn = N at END);
    ``held``     budget bytes held after each op;
    ``windows``  r_i per function;
    ``peak``     max held; ``h2d`` / ``d2h`` bytes moved by SWAPIN / SWAPOUT.

    ``wait`` chooses which pending swap-out a budget wait in step (b) completes:
    ``"oldest"`` as in Fig. 2, or ``"furthest"``: the one whose variable's next
    use lies furthest ahead in the variable-sequence (never used again counts
    as furthest; the earliest reserved among equals).  The paper leaves the
    order of swap-outs open (Section 6).  The waits at END are oldest first.
    """
    if policy not in ("C", "L"):
        raise Invalid("policy must be 'C' or 'L'")
    if wait not in ("oldest", "furthest"):
        raise Invalid("wait must be 'oldest' or 'furthest'")
    # fixed-distance rule of LMS (Section 2): swap in `ahead` functions before a use, keep a
    # variable whose next use is at most `threshold` functions away
    fixed = ahead is not None or threshold is not None
    if fixed and (ahead is None or threshold is None or ahead < 0 or threshold < 0):
        raise Invalid("the fixed-distance rule needs ahead >= 0 and threshold >= 0")
    if chunk <= 0:
        raise Invalid("chunk must be positive")
    fn_vars = normalize(fn_vars)
    validate(var_bytes, var_kinds, fn_vars)
    N = len(fn_vars)
    b = list(var_bytes)
    a = [rounded(x, chunk) for x in var_bytes]
    seq, first, last = sequence(fn_vars)
    nxt = next_use(seq, first, last)
    fn_of = [i for i in range(N) for _ in fn_vars[i]]

    state = [HOST if k in PERSISTENT else UNMAT for k in var_kinds]
    # pending swap-outs, oldest first; under policy L an entry is one device copy.
    # fifo_next[k] is the position of the next use of fifo[k]'s variable
    # (infinity when it has none).
    fifo = deque()
    fifo_next = deque()
    held = 0
    ops, trace, windows = [], [], []
    h2d = d2h = 0
    r_prev = -1

    def emit(i, phase, kind, v):
        ops.append((i, phase, kind, v))
        trace.append(held)

    for i in range(N):
        l, e = first[i], last[i]
        # 1. schedule-window (bytes), or the functions up to f_{i + ahead}
        if fixed:
            r = max(last[min(i + ahead, N - 1)], e, r_prev)
        else:
            r = max(window_end(seq, b, l, window), e, r_prev)
        # 2. steps (a)+(b): admit positions r_prev+1 .. r
        p = r_prev + 1
        while p <= r:
            u = seq[p]
            if state[u] == DEV:
                p += 1
                continue
            if state[u] == PEND and policy == "C":
                k = fifo.index(u)
                del fifo[k]
                del fifo_next[k]
                state[u] = DEV
                emit(i, PRE, CANCEL, u)
                p += 1
                continue
            need = a[u]
            while held + need > budget and fifo:
                k = 0
                if wait == "furthest":
                    k = max(range(len(fifo)), key=lambda q: (fifo_next[q], -q))
                w = fifo[k]
                del fifo[k]
                del fifo_next[k]
                held -= a[w]
                _swapped_out(w, fifo, state)
                emit(i, PRE, WAIT_OUT, w)
            if held + need <= budget:
                if state[u] == UNMAT:
                    kind = ALLOC
                else:
                    kind = SWAPIN
                    h2d += b[u]
                state[u] = DEV
                held += need
                emit(i, PRE, kind, u)
            elif p <= e:
                raise Infeasible(f"function {i} does not fit in budget {budget}")
            else:
                r = p - 1
                break
            p += 1
        windows.append(r)
        # 3. f_i runs here: every variable of V_i is on the device
        # 4. steps (c)+(d)
        for u, _ in fn_vars[i]:
            n = nxt[i][u]
            if n is None and var_kinds[u] in (INPUT, TEMP):
                state[u] = UNMAT
                held -= a[u]
                emit(i, POST, FREE, u)
            elif n is not None and (n <= r or (fixed and fn_of[n] - i <= threshold)):
                pass  # already reserved inside the window (or close enough): keep it
            else:
                state[u] = PEND
                fifo.append(u)
                fifo_next.append(math.inf if n is None else n)
                d2h += b[u]
                emit(i, POST, SWAPOUT, u)
        r_prev = r

    while fifo:
        w = fifo.popleft()
        fifo_next.popleft()
        held -= a[w]
        _swapped_out(w, fifo, state)
        emit(N, END, WAIT_OUT, w)
    return {"ops": ops, "held": trace, "windows": windows,
            "peak": max(trace, default=0), "h2d": h2d, "d2h": d2h}


def _swapped_out(w, fifo, state):
    """A pending swap-out of w has completed: its device copy is released.

    Under policy C the variable is then on the host.  Under policy L the
    variable's state follows its newest copy: it becomes HOST only if the copy
    that just completed was the newest one, i.e. w is PEND and has no later
    swap-out still queued; a newer working copy (DEV) or a freed one (UNMAT)
    is left as it is.
    """
    if state[w] == PEND and w not in fifo:
        state[w] = HOST


# --------------------------------------------------------------------------
# in-core plan and the budget bounds derived from it
# --------------------------------------------------------------------------


def first_last_use(fn_vars, nv):
    fu = [None] * nv
    lu = [None] * nv
    for i, vs in enumerate(normalize(fn_vars)):
        for v, _ in vs:
            if fu[v] is None:
                fu[v] = i
            lu[v] = i
    return fu, lu


def incore_plan(var_bytes, var_kinds, fn_vars, chunk=1):
    """In-core allocation plan: persistent variables (INPUT/PARAM/STATE/OUTPUT) stay on
    the device for the whole step; a TEMP is allocated before its first use and freed
    after its last use.  No transfers.  Returns ``{"ops", "held", "peak"}``."""
    fn_vars = normalize(fn_vars)
    validate(var_bytes, var_kinds, fn_vars)
    nv = len(var_bytes)
    a = [rounded(x, chunk) for x in var_bytes]
    fu, lu = first_last_use(fn_vars, nv)
    held = sum(a[v] for v in range(nv) if var_kinds[v] != TEMP)
    ops, trace = [], []
    for i, vs in enumerate(fn_vars):
        for v, _ in vs:
            if var_kinds[v] == TEMP and fu[v] == i:
                held += a[v]
                ops.append((i, PRE, ALLOC, v))
                trace.append(held)
        for v, _ in vs:
            if var_kinds[v] == TEMP and lu[v] == i:
                held -= a[v]
                ops.append((i, POST, FREE, v))
                trace.append(held)
    base = sum(a[v] for v in range(nv) if var_kinds[v] != TEMP)
    return {"ops": ops, "held": trace, "peak": max(trace, default=base)}


def incore_peak(var_bytes, var_kinds, fn_vars, chunk=1):
    """P_incore: the most chunk-rounded bytes live at any function in the in-core plan."""
    return incore_plan(var_bytes, var_kinds, fn_vars, chunk)["peak"]


def working_set_max(var_bytes, fn_vars, chunk=1):
    """WS_max = max over functions of the chunk-rounded bytes of V_i; no budget below it works."""
    return max(sum(rounded(var_bytes[v], chunk) for v, _ in vs) for vs in normalize(fn_vars))


def budget_for(fraction, p_incore, chunk=1):
    """B = floor(fraction * P_incore / m_c) * m_c (integer arithmetic on a rational fraction)."""
    from fractions import Fraction
    f = Fraction(fraction).limit_denominator(10 ** 6)
    return (p_incore * f.numerator // f.denominator) // chunk * chunk

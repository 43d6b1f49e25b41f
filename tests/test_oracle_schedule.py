"""Pins of the oracle scheduler against what the paper fixes (CPU only).

* a hand-derived worked example of the procedure of Section 3 / Fig. 2;
* the window definition of Section 3, recomputed by brute force;
* an independent replayer (``oracle.check``): budget never exceeded, every
  variable resident and current when a function runs, oldest swap-outs waited
  first, final values written back;
* the naive schedule of Section 1 as the zero-window limit;
* the in-core limit (unbounded window and budget);
* the feasibility boundary (the largest per-function footprint).
"""

import os
import random
from collections import Counter

import pytest
from hypothesis import given, settings, strategies as st

from oracle import check, naive, schedule as S
from oracle.lower import lower, as_schedule_input
from paper_2010_14109_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "window_schedule_4vars.txt")
NAMES = {n: i for i, n in enumerate(S.OP_NAMES)}
PH = {"PRE": S.PRE, "POST": S.POST, "END": S.END}


def golden_case():
    kinds = [S.INPUT, S.TEMP, S.TEMP, S.TEMP]
    A, B, C, D = range(4)
    fns = [[(A, S.R), (B, S.W)], [(B, S.R), (C, S.W)], [(C, S.R), (D, S.W)],
           [(D, S.R), (C, S.R)], [(B, S.R)], [(A, S.R)]]
    return [8] * 4, kinds, fns


def parse_golden():
    out = {}
    cur = None
    with open(GOLDEN) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            t = line.split()
            if t[0] == "windows":
                (out[cur] if cur == "fixed" else out)["windows"] = [int(x) for x in t[1:]]
            elif t[0] == "policy":
                cur = t[1]
                out[cur] = {"ops": [], "held": []}
            elif t[0] == "fixed":
                cur = "fixed"
                out[cur] = {"ops": [], "held": [], "ahead": int(t[1]), "threshold": int(t[2])}
            elif t[0] == "totals":
                out[cur]["peak"], out[cur]["h2d"], out[cur]["d2h"] = int(t[2]), int(t[4]), int(t[6])
            else:
                fn, ph, op, var, held = t
                out[cur]["ops"].append((int(fn) - 1, PH[ph], NAMES[op], "ABCD".index(var)))
                out[cur]["held"].append(int(held))
    return out


@pytest.mark.parametrize("policy", ["C", "L"])
def test_golden_worked_example(policy):
    g = parse_golden()
    b, k, f = golden_case()
    out = S.build(b, k, f, budget=24, window=24, chunk=1, policy=policy)
    assert out["windows"] == g["windows"]
    assert out["ops"] == g[policy]["ops"]
    assert out["held"] == g[policy]["held"]
    assert (out["peak"], out["h2d"], out["d2h"]) == (g[policy]["peak"], g[policy]["h2d"],
                                                      g[policy]["d2h"])
    check.replay(b, k, f, out["ops"], 24, policy=policy, held=out["held"])


def test_golden_fixed_distance_example():
    """The fixed-distance rule of LMS (Section 2) on the same sequence, worked out by hand."""
    g = parse_golden()["fixed"]
    b, k, f = golden_case()
    out = S.build(b, k, f, budget=24, window=0, chunk=1, policy="C", ahead=g["ahead"],
                  threshold=g["threshold"])
    assert out["windows"] == g["windows"]
    assert out["ops"] == g["ops"]
    assert out["held"] == g["held"]
    assert (out["peak"], out["h2d"], out["d2h"]) == (g["peak"], g["h2d"], g["d2h"])
    check.replay(b, k, f, out["ops"], 24, policy="C", held=out["held"])


@pytest.mark.parametrize("policy", ["C", "L"])
def test_fixed_distance_schedules_replay(policy):
    """Random registrations, every ahead up to 4 with a random threshold: the replayer accepts
    every schedule that fits (variables kept by the threshold are not waited for, so, as with
    LMS itself, a tight budget can be infeasible); a zero-ahead, zero-threshold schedule swaps
    exactly like the zero byte window."""
    rng = random.Random(11)
    built = failed = 0
    for _ in range(120):
        b, k, f = random_registration(rng)
        bud = S.working_set_max(b, f, 1) + rng.randint(0, 120)
        for ahead in range(5):
            thr = rng.randint(0, 4)
            try:
                out = S.build(b, k, f, budget=bud, window=0, chunk=1, policy=policy, ahead=ahead,
                              threshold=thr)
            except S.Infeasible:
                failed += 1
                continue
            built += 1
            check.replay(b, k, f, out["ops"], bud, policy=policy, held=out["held"])
        z = S.build(b, k, f, budget=bud, window=0, chunk=1, policy=policy, ahead=0, threshold=0)
        w0 = S.build(b, k, f, budget=bud, window=0, chunk=1, policy=policy)
        assert z["ops"] == w0["ops"]
    assert built > 2 * failed


def test_fixed_distance_needs_both_parameters():
    b, k, f = golden_case()
    for kw in ({"ahead": 1}, {"threshold": 1}, {"ahead": -1, "threshold": 0}):
        with pytest.raises(S.Invalid):
            S.build(b, k, f, budget=24, window=0, **kw)


# ---------------------------------------------------------------- registrations
def random_registration(rng, nv=10, nf=14, maxsize=64):
    kinds = [rng.choice([S.INPUT, S.PARAM, S.STATE, S.TEMP, S.TEMP, S.TEMP, S.OUTPUT])
             for _ in range(nv)]
    sizes = [rng.randint(1, maxsize) for _ in range(nv)]
    produced = [k in (S.INPUT, S.PARAM, S.STATE) for k in kinds]
    fns = []
    for _ in range(nf):
        vs = rng.sample(range(nv), rng.randint(1, min(4, nv)))
        row = []
        for v in vs:
            if not produced[v]:
                a = S.W
            elif kinds[v] == S.INPUT:
                a = S.R
            else:
                a = rng.choice([S.R, S.R, S.RW, S.W])
            produced[v] = True
            row.append((v, a))
        fns.append(row)
    return sizes, kinds, fns


def small_networks():
    return [
        synth.mlp(batch=4, width=16, depth=4, classes=5),
        synth.plain_cnn(batch=2, channels=4, depth=3, hw=8, classes=5),
        synth.resnet(batch=2, hw=32, classes=7, blocks=(1, 2, 1, 1), width=4),
        synth.resnet(batch=1, hw=32, classes=7, blocks=(1, 1, 1, 1), width=4, momentum=0.0),
        synth.densenet(batch=2, hw=8, growth=4, blocks=(3, 3), stem=4, classes=5),
        synth.unet(batch=1, hw=16, base=4, depth=3, classes=3),
    ]


def brute_window(seq, sizes, l, W):
    best = l - 1
    for r in range(l, len(seq)):
        if sum(sizes[seq[p]] for p in range(l, r + 1)) <= W:
            best = r
    return best


def test_windows_match_definition():
    rng = random.Random(7)
    for _ in range(40):
        b, k, f = random_registration(rng)
        W = rng.choice([0, 10, 40, 100, 400])
        out = S.build(b, k, f, budget=10 ** 9, window=W)
        fn = S.normalize(f)
        seq, first, last = S.sequence(fn)
        prev = -1
        for i in range(len(fn)):
            expect = max(brute_window(seq, b, first[i], W), last[i], prev)
            assert out["windows"][i] == expect
            prev = expect


@pytest.mark.parametrize("policy", ["C", "L"])
def test_random_schedules_replay(policy):
    rng = random.Random(11 if policy == "C" else 12)
    for _ in range(150):
        b, k, f = random_registration(rng)
        ws = S.working_set_max(b, f)
        B = rng.randint(ws, ws * 3)
        W = rng.choice([0, 16, 64, 256, S.INCORE])
        out = S.build(b, k, f, budget=B, window=W, policy=policy)
        res = check.replay(b, k, f, out["ops"], B, policy=policy, held=out["held"])
        assert res["peak"] == out["peak"] <= B
        assert (res["h2d"], res["d2h"]) == (out["h2d"], out["d2h"])


def test_resident_set_is_window_plus_pending():
    """Policy C: before f_i the device holds exactly the window's variables and the
    pending swap-outs (nothing else, nothing missing)."""
    rng = random.Random(3)
    for _ in range(60):
        b, k, f = random_registration(rng)
        B = 10 ** 9  # no truncation
        W = rng.choice([0, 16, 64, 256])
        out = S.build(b, k, f, budget=B, window=W)
        fn = S.normalize(f)
        seq, first, _ = S.sequence(fn)
        for i in range(len(fn)):
            dev, pend = check.resident_before(f, out["ops"], i)
            window_vars = set(seq[first[i]:out["windows"][i] + 1])
            assert dev == window_vars
            assert not (pend & dev)


@pytest.mark.parametrize("spec", small_networks(), ids=lambda s: s["name"])
@pytest.mark.parametrize("policy", ["C", "L"])
def test_network_schedules_replay(spec, policy):
    reg = lower(spec)
    b, k, f = as_schedule_input(reg)
    for chunk in (1, 256):
        p = S.incore_peak(b, k, f, chunk)
        ws = S.working_set_max(b, f, chunk)
        for frac in (1.0, 0.75, 0.5, 0.4, 0.25, 1 / 7.5, 0.2, 0.0):
            B = max(S.budget_for(frac, p, chunk), ws)
            for W in (0, B // 8, B // 2, B, S.INCORE):
                out = S.build(b, k, f, B, W, chunk, policy)
                res = check.replay(b, k, f, out["ops"], B, chunk, policy, held=out["held"])
                assert res["peak"] <= B


def test_naive_schedule_is_zero_window_limit():
    """Policy L with a zero window moves exactly what the naive swap-every-layer schedule
    moves (Section 1), and it is feasible exactly from the largest footprint on."""
    rng = random.Random(5)
    cases = [random_registration(rng) for _ in range(60)]
    cases += [as_schedule_input(lower(s)) for s in small_networks()]
    for b, k, f in cases:
        ws = naive.working_set(b, f)
        out = S.build(b, k, f, budget=ws, window=0, policy="L")
        got = Counter()
        for (i, ph, kind, v) in out["ops"]:
            if kind == S.SWAPIN:
                got[("in", i, v)] += 1
            elif kind == S.SWAPOUT:
                got[("out", i, v)] += 1
        assert got == naive.transfers(k, f)
        with pytest.raises(S.Infeasible):
            S.build(b, k, f, budget=ws - 1, window=0, policy="L")


def test_zero_window_policy_c_swaps_after_every_use():
    rng = random.Random(6)
    for _ in range(40):
        b, k, f = random_registration(rng)
        out = S.build(b, k, f, budget=10 ** 9, window=0, policy="C")
        fn = S.normalize(f)
        seq, first, last = S.sequence(fn)
        assert out["windows"] == last
        outs = {(i, v) for (i, ph, kind, v) in out["ops"] if kind == S.SWAPOUT}
        for i, vs in enumerate(fn):
            for v, _ in vs:
                later = any(v in [u for u, _ in fn[j]] for j in range(i + 1, len(fn)))
                if later or k[v] in (S.PARAM, S.STATE, S.OUTPUT):
                    assert (i, v) in outs


def test_incore_limit():
    """Unbounded window and budget: only the first loads and the final write-backs move,
    and no swap-out is waited for before the end."""
    rng = random.Random(8)
    cases = [random_registration(rng) for _ in range(40)]
    cases += [as_schedule_input(lower(s)) for s in small_networks()]
    for b, k, f in cases:
        B = sum(b)
        out = S.build(b, k, f, budget=B, window=S.INCORE)
        fn = S.normalize(f)
        uses = {}
        for i, vs in enumerate(fn):
            for v, _ in vs:
                uses.setdefault(v, []).append(i)
        ins = [(i, v) for (i, ph, kind, v) in out["ops"] if kind == S.SWAPIN]
        outs = [(i, v) for (i, ph, kind, v) in out["ops"] if kind == S.SWAPOUT]
        assert sorted(v for _, v in ins) == sorted(v for v in uses if k[v] in S.PERSISTENT)
        assert all(i == 0 for i, _ in ins)
        assert sorted(outs) == sorted((uses[v][-1], v) for v in uses if k[v] in S.WRITE_BACK)
        assert all(ph == S.END for (_, ph, kind, _) in out["ops"] if kind == S.WAIT_OUT)
        assert not any(kind == S.CANCEL for (_, _, kind, _) in out["ops"])


def brute_incore_peak(b, k, f, chunk):
    """P_incore from its definition, one function at a time: every INPUT, PARAM, STATE and
    OUTPUT variable counts for the whole step (the in-core step keeps them resident, so that
    their values can be read back after it); a TEMP counts at the functions from its first
    to its last use; sizes are rounded up to whole chunks."""
    uses = {}
    for i, vs in enumerate(f):
        for v, _ in vs:
            uses.setdefault(v, []).append(i)
    rounded = [-(-x // chunk) * chunk for x in b]
    resident = sum(rounded[v] for v in range(len(b)) if k[v] != S.TEMP)
    best = 0
    for i in range(len(f)):
        live = [v for v, at in uses.items() if k[v] == S.TEMP and min(at) <= i <= max(at)]
        best = max(best, resident + sum(rounded[v] for v in live))
    return best


def test_incore_peak_is_the_live_set_maximum():
    """P_incore against the brute-force live-set sum per function, on random registrations and
    the networks at several chunk sizes; WS_max against the largest single function."""
    rng = random.Random(12)
    cases = [random_registration(rng, nv=rng.randint(1, 12), nf=rng.randint(1, 20))
             for _ in range(300)]
    cases += [as_schedule_input(lower(s)) for s in small_networks()]
    cases += [as_schedule_input(lower(synth.workload(n))) for n in ("cnn", "resnet50_b256")]
    for b, k, f in cases:
        for chunk in (1, 8, 4096, 2 << 20):
            assert S.incore_peak(b, k, f, chunk) == brute_incore_peak(b, k, f, chunk)
            ws = max(sum(-(-b[v] // chunk) * chunk for v in {v for v, _ in vs}) for vs in f)
            assert S.working_set_max(b, f, chunk) == ws
    # a chain x -> t1 -> t2 -> t3: two TEMPs live at once at most (24 bytes); a TEMP kept one
    # function past its last use would make three live at f2 (32)
    b, k = [8, 8, 8, 8], [S.INPUT, S.TEMP, S.TEMP, S.TEMP]
    f = [[(0, S.R), (1, S.W)], [(1, S.R), (2, S.W)], [(2, S.R), (3, S.W)], [(3, S.R)]]
    assert S.incore_peak(b, k, f) == brute_incore_peak(b, k, f, 1) == 24
    late = f[:2] + [[(2, S.R), (3, S.W), (1, S.R)]] + f[3:]
    assert S.incore_peak(b, k, late) == brute_incore_peak(b, k, late, 1) == 32
    # OUTPUT counts for the whole step, like the persistent kinds
    assert S.incore_peak(b, [S.INPUT, S.OUTPUT, S.TEMP, S.TEMP], f) == 8 + 8 + 16


@pytest.mark.parametrize("spec", small_networks(), ids=lambda s: s["name"])
def test_feasibility_boundary(spec):
    b, k, f = as_schedule_input(lower(spec))
    for chunk in (1, 64):
        ws = S.working_set_max(b, f, chunk)
        for W in (0, 1000, S.INCORE):
            for policy in ("C", "L"):
                out = S.build(b, k, f, ws, W, chunk, policy)
                check.replay(b, k, f, out["ops"], ws, chunk, policy, held=out["held"])
                with pytest.raises(S.Infeasible):
                    S.build(b, k, f, ws - 1, W, chunk, policy)


def test_invalid_registrations():
    with pytest.raises(S.Invalid):   # TEMP read before written
        S.build([4, 4], [S.INPUT, S.TEMP], [[(0, S.R), (1, S.R)]], 100, 100)
    with pytest.raises(S.Invalid):   # INPUT written
        S.build([4], [S.INPUT], [[(0, S.RW)]], 100, 100)
    with pytest.raises(S.Invalid):   # unknown variable
        S.build([4], [S.INPUT], [[(3, S.R)]], 100, 100)
    with pytest.raises(S.Invalid):   # empty function
        S.build([4], [S.INPUT], [[]], 100, 100)
    with pytest.raises(S.Invalid):   # zero-byte variable
        S.build([0], [S.INPUT], [[(0, S.R)]], 100, 100)


# ---------------------------------------------------------------- the replayer catches mistakes
def test_replayer_catches_planted_mistakes():
    """Every plausible scheduler slip must be caught by the replayer."""
    b, k, f = golden_case()
    good = S.build(b, k, f, 24, 24)["ops"]
    check.replay(b, k, f, good, 24)
    mutants = []
    # dropped swap-in
    mutants.append([o for o in good if o != (0, S.PRE, S.SWAPIN, 0)])
    # waits taken in the wrong order (newest first)
    m = list(good)
    m[good.index((2, S.PRE, S.WAIT_OUT, 0))] = (2, S.PRE, S.WAIT_OUT, 1)
    mutants.append(m)
    # a cancel replaced by a swap-in of a variable whose swap-out is still pending
    m = list(good)
    m[good.index((3, S.PRE, S.CANCEL, 2))] = (3, S.PRE, S.SWAPIN, 2)
    mutants.append(m)
    # a variable freed although used later
    m = list(good)
    m[good.index((1, S.POST, S.SWAPOUT, 1))] = (1, S.POST, S.FREE, 1)
    mutants.append(m)
    # budget too small for the same ops
    for mt in mutants:
        with pytest.raises(check.ScheduleError):
            check.replay(b, k, f, mt, 24)
    with pytest.raises(check.ScheduleError):
        check.replay(b, k, f, good, 23)
    # a PARAM whose update is never written back
    kinds = [S.PARAM]
    fns = [[(0, S.RW)]]
    with pytest.raises(check.ScheduleError):
        check.replay([4], kinds, fns, [(0, S.PRE, S.SWAPIN, 0), (0, S.POST, S.FREE, 0)], 8)


# ---------------------------------------------------------------- fuzz
@settings(max_examples=200, deadline=None)
@given(seed=st.integers(0, 10 ** 9), nv=st.integers(1, 12), nf=st.integers(1, 20),
       wsel=st.integers(0, 4), bsel=st.integers(0, 3), policy=st.sampled_from(["C", "L"]),
       chunk=st.sampled_from([1, 8, 32]))
def test_fuzz_chains_with_skips(seed, nv, nf, wsel, bsel, policy, chunk):
    rng = random.Random(seed)
    b, k, f = random_registration(rng, nv=nv, nf=nf)
    ws = S.working_set_max(b, f, chunk)
    B = [ws, ws + chunk, 2 * ws, 10 ** 9][bsel]
    W = [0, 8, 64, 512, S.INCORE][wsel]
    out = S.build(b, k, f, B, W, chunk, policy)
    check.replay(b, k, f, out["ops"], B, chunk, policy, held=out["held"])
    r = out["windows"]
    fn = S.normalize(f)
    _, first, last = S.sequence(fn)
    assert all(r[i] >= last[i] for i in range(len(r)))
    assert all(r[i] >= r[i - 1] for i in range(1, len(r)))


# ---------------------------------------------------------------- wait order of pending swap-outs
def test_wait_order_hand_example():
    """Three unit TEMPs, budget 2, W = 0, policy C: f0 writes A, f1 writes B, f2 writes C, then
    f3, f4, f5 read A, B, C.  Admitting C at f2 needs one pending swap-out completed.  Oldest
    first completes A, which f3 then swaps back in (after completing B); furthest first completes
    B (next used at f4, after A's use at f3), and A's pending swap-out is cancelled at f3.  Derived
    by hand from the procedure of Section 3."""
    A, B_, C = 0, 1, 2
    b, k = [1, 1, 1], [S.TEMP] * 3
    f = [[(A, S.W)], [(B_, S.W)], [(C, S.W)], [(A, S.R)], [(B_, S.R)], [(C, S.R)]]
    pre, post = S.PRE, S.POST
    common = [(0, pre, S.ALLOC, A), (0, post, S.SWAPOUT, A), (1, pre, S.ALLOC, B_),
              (1, post, S.SWAPOUT, B_)]
    oldest = common + [(2, pre, S.WAIT_OUT, A), (2, pre, S.ALLOC, C), (2, post, S.SWAPOUT, C),
                       (3, pre, S.WAIT_OUT, B_), (3, pre, S.SWAPIN, A), (3, post, S.FREE, A),
                       (4, pre, S.SWAPIN, B_), (4, post, S.FREE, B_),
                       (5, pre, S.CANCEL, C), (5, post, S.FREE, C)]
    furthest = common + [(2, pre, S.WAIT_OUT, B_), (2, pre, S.ALLOC, C), (2, post, S.SWAPOUT, C),
                         (3, pre, S.CANCEL, A), (3, post, S.FREE, A),
                         (4, pre, S.SWAPIN, B_), (4, post, S.FREE, B_),
                         (5, pre, S.CANCEL, C), (5, post, S.FREE, C)]
    out_o = S.build(b, k, f, 2, 0, 1, "C")
    out_f = S.build(b, k, f, 2, 0, 1, "C", wait="furthest")
    assert out_o["ops"] == oldest and out_f["ops"] == furthest
    assert (out_o["h2d"], out_f["h2d"]) == (2, 1)
    check.replay(b, k, f, out_f["ops"], 2, wait="furthest")
    with pytest.raises(check.ScheduleError):        # the replayer tells the two rules apart
        check.replay(b, k, f, out_f["ops"], 2)
    with pytest.raises(check.ScheduleError):
        check.replay(b, k, f, out_o["ops"], 2, wait="furthest")
    with pytest.raises(S.Invalid):
        S.build(b, k, f, 2, 0, 1, "C", wait="newest")


@pytest.mark.parametrize("policy", ["C", "L"])
def test_furthest_wait_schedules_replay(policy):
    """Random registrations and the small networks under the furthest-next-use wait order:
    budget, residency, data versions and the wait rule hold (independent replayer)."""
    rng = random.Random(31 if policy == "C" else 32)
    for _ in range(150):
        b, k, f = random_registration(rng)
        ws = S.working_set_max(b, f)
        B = rng.randint(ws, ws * 3)
        W = rng.choice([0, 16, 64, 256, S.INCORE])
        out = S.build(b, k, f, budget=B, window=W, policy=policy, wait="furthest")
        res = check.replay(b, k, f, out["ops"], B, policy=policy, held=out["held"], wait="furthest")
        assert res["peak"] == out["peak"] <= B
        assert (res["h2d"], res["d2h"]) == (out["h2d"], out["d2h"])
    for spec in small_networks():
        b, k, f = as_schedule_input(lower(spec))
        p = S.incore_peak(b, k, f, 256)
        ws = S.working_set_max(b, f, 256)
        for frac in (0.5, 0.25, 0.0):
            B = max(S.budget_for(frac, p, 256), ws)
            out = S.build(b, k, f, B, B // 2, 256, policy, wait="furthest")
            check.replay(b, k, f, out["ops"], B, 256, policy, held=out["held"], wait="furthest")

"""The C library on the host (no GPU): exports, call order, validation, and
bit-exact parity of its function sequence, schedule and chunk plan with the
oracle's independent ones."""

import os
import random
import re

import pytest

from oracle import pool as opool
from oracle import schedule as S
from oracle.lower import lower, as_schedule_input
from paper_2010_14109_amd import netdef, ooc, synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "ooc.h")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(ooc_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol(lib):
    names = declared_symbols()
    assert names == sorted(ooc.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def specs_small():
    return [
        synth.transformer(batch=2, seq=8, d=64, heads=4, ffn=96, layers=2, vocab=50),
        synth.mlp(batch=4, width=16, depth=4, classes=5),
        synth.mlp(batch=3, width=8, depth=2, classes=3, momentum=0.9),
        synth.plain_cnn(batch=2, channels=4, depth=3, hw=8, classes=5),
        synth.resnet(batch=2, hw=32, classes=7, blocks=(1, 2, 1, 1), width=4),
        synth.densenet(batch=2, hw=8, growth=4, blocks=(3, 2), stem=4, classes=5),
        synth.unet(batch=1, hw=16, base=4, depth=3, classes=3),
    ]


def specs_full():
    return [synth.workload(n) for n in ("mlp", "cnn", "resnet50_b256", "resnet50_b1440",
                                        "transformer", "densenet", "unet")]


@pytest.mark.parametrize("spec", specs_small() + specs_full(), ids=lambda s: s["name"])
@pytest.mark.parametrize("keep", [False, True])
def test_function_sequence_matches_oracle_lowering(spec, keep):
    mine = netdef.Net(spec, keep_grads=keep)
    ref = lower(spec, keep_grads=keep, slices=mine.slices)
    assert mine.var_bytes == [v["bytes"] for v in ref["vars"]]
    assert mine.var_kinds == [v["kind"] for v in ref["vars"]]
    assert mine.names == [v["name"] for v in ref["vars"]]
    opname = {"add_fwd": "add", "add_grad": "add", "acc_grad": "acc"}
    assert mine.fn_ops == [opname.get(f["op"], f["op"]) for f in ref["fns"]]
    assert mine.fn_vars == [f["vars"] for f in ref["fns"]]


def host_ctx(net, budget, window, chunk, policy):
    ctx = ooc.Context(-1)
    net.register(ctx)
    ctx.set_chunk(chunk)
    ctx.set_budget(budget)
    if window is not None:
        ctx.set_window(window)
    ctx.set_policy(policy)
    ctx.build_schedule()
    return ctx


@pytest.mark.parametrize("spec,full", [(s, False) for s in specs_small()] +
                         [(s, True) for s in specs_full()], ids=lambda s: s["name"]
                         if isinstance(s, dict) else ("full" if s else "small"))
def test_schedule_and_plan_match_oracle(spec, full):
    net = netdef.Net(spec)
    b, k, f = as_schedule_input(lower(spec, slices=net.slices))
    chunks = (2 << 20,) if full else (64, 4096)
    fracs = (1.0, 0.5, 0.25, 1 / 7.5, 0.0) if full else (1.0, 0.75, 0.5, 0.4, 0.25, 1 / 7.5, 0.2, 0.0)
    for chunk in chunks:
        ctx0 = host_ctx(net, ooc.UNLIMITED, None, chunk, "C")
        p = S.incore_peak(b, k, f, chunk)
        ws = S.working_set_max(b, f, chunk)
        assert ctx0.incore_peak() == p
        assert ctx0.working_set_max() == ws
        inc = S.incore_plan(b, k, f, chunk)
        ops0, held0 = ctx0.schedule()
        assert ops0 == inc["ops"] and held0 == inc["held"]
        ctx0.close()
        for frac in fracs:
            B = max(S.budget_for(frac, p, chunk), ws)
            wins = (0, B // 4, B // 2, B, S.INCORE) if not full else (0, B // 2, B)
            for W in wins:
                for policy in ("C", "L"):
                    ref = S.build(b, k, f, B, W, chunk, policy)
                    ctx = host_ctx(net, B, W, chunk, policy)
                    ops, held = ctx.schedule()
                    assert ops == ref["ops"], (frac, W, policy)
                    assert held == ref["held"]
                    assert ctx.windows() == ref["windows"]
                    st = ctx.stats()
                    assert (st["peak_accounted"], st["sched_h2d_bytes"], st["sched_d2h_bytes"]) == \
                        (ref["peak"], ref["h2d"], ref["d2h"])
                    ivs, max_used = opool.assign(ref["ops"], b, B // chunk, chunk)
                    got = ctx.plan()
                    assert [(g["var"], g["open"], g["close"], g["chunks"]) for g in got] == \
                        [(i["var"], i["open"], i["close"], i["chunks"]) for i in ivs]
                    assert st["max_chunks_used"] == max_used
                    ctx.close()


def random_registration(rng, nv=10, nf=14, maxsize=64):
    kinds = [rng.choice([S.INPUT, S.PARAM, S.STATE, S.TEMP, S.TEMP, S.TEMP, S.OUTPUT])
             for _ in range(nv)]
    sizes = [rng.randint(1, maxsize) for _ in range(nv)]
    produced = [kd in (S.INPUT, S.PARAM, S.STATE) for kd in kinds]
    fns = []
    for _ in range(nf):
        row = []
        for v in rng.sample(range(nv), rng.randint(1, min(4, nv))):
            if not produced[v]:
                a = S.W
            elif kinds[v] == S.INPUT:
                a = S.R
            else:
                a = rng.choice([S.R, S.RW, S.W])
            produced[v] = True
            row.append((v, a))
        fns.append(row)
    return sizes, kinds, fns


def test_random_sequences_match_oracle(lib):
    rng = random.Random(2024)
    for trial in range(300):
        b, k, f = random_registration(rng, nv=rng.randint(1, 12), nf=rng.randint(1, 20))
        chunk = rng.choice([1, 8, 32])
        ws = S.working_set_max(b, f, chunk)
        B = rng.choice([ws, ws + chunk, 2 * ws, 10 ** 6])
        W = rng.choice([0, 8, 64, 512, S.INCORE])
        policy = rng.choice("CL")
        ref = S.build(b, k, f, B, W, chunk, policy)
        ctx = ooc.Context(-1)
        for nb, kd in zip(b, k):
            ctx.add_var(nb, kd)
        for vs in f:
            ctx.add_fn("noop", [v for v, _ in vs], [a for _, a in vs])
        ctx.set_chunk(chunk)
        ctx.set_budget(B)
        ctx.set_window(W)
        ctx.set_policy(policy)
        ctx.build_schedule()
        ops, held = ctx.schedule()
        assert ops == ref["ops"], trial
        assert held == ref["held"], trial
        assert ctx.windows() == ref["windows"], trial
        ivs, _ = opool.assign(ref["ops"], b, B // chunk, chunk)
        assert [(g["var"], g["open"], g["close"], g["chunks"]) for g in ctx.plan()] == \
            [(i["var"], i["open"], i["close"], i["chunks"]) for i in ivs]
        with pytest.raises(ooc.OocError) as e:
            ctx.prepare()          # host-only context
        assert e.value.status == ooc.E_UNSUPPORTED
        ctx.close()


def test_fixed_distance_matches_oracle(lib):
    """The fixed-distance (LMS) rule: random registrations and the small networks, schedules
    and chunk plans op for op, infeasible budgets reported on both sides."""
    rng = random.Random(77)
    cases = []
    for _ in range(200):
        b, k, f = random_registration(rng, nv=rng.randint(1, 12), nf=rng.randint(1, 20))
        chunk = rng.choice([1, 8, 32])
        ws = S.working_set_max(b, f, chunk)
        cases.append((b, k, f, chunk, rng.choice([ws, ws + chunk, 2 * ws, 10 ** 6])))
    for spec in specs_small():
        b, k, f = as_schedule_input(lower(spec))
        p = S.incore_peak(b, k, f, 4096)
        ws = S.working_set_max(b, f, 4096)
        for frac in (0.5, 0.25):
            cases.append((b, k, f, 4096, max(S.budget_for(frac, p, 4096), ws)))
    n_inf = 0
    for trial, (b, k, f, chunk, B) in enumerate(cases):
        ahead, thr = rng.randint(0, 6), rng.randint(0, 6)
        policy = rng.choice("CL")
        ctx = ooc.Context(-1)
        for nb, kd in zip(b, k):
            ctx.add_var(nb, kd)
        for vs in f:
            ctx.add_fn("noop", [v for v, _ in vs], [a for _, a in vs])
        ctx.set_chunk(chunk)
        ctx.set_budget(B)
        ctx.set_policy(policy)
        ctx.set_fixed_distance(ahead, thr)
        try:
            ref = S.build(b, k, f, B, 0, chunk, policy, ahead=ahead, threshold=thr)
        except S.Infeasible:
            n_inf += 1
            with pytest.raises(ooc.OocError) as e:
                ctx.build_schedule()
            assert e.value.status == ooc.E_INFEASIBLE
            ctx.close()
            continue
        ctx.build_schedule()
        ops, held = ctx.schedule()
        assert ops == ref["ops"], trial
        assert held == ref["held"], trial
        assert ctx.windows() == ref["windows"], trial
        ivs, _ = opool.assign(ref["ops"], b, B // chunk, chunk)
        assert [(g["var"], g["open"], g["close"], g["chunks"]) for g in ctx.plan()] == \
            [(i["var"], i["open"], i["close"], i["chunks"]) for i in ivs]
        ctx.close()
    assert n_inf < len(cases) // 2
    ctx = ooc.Context(-1)
    for bad in ((1, -1), (-1, 2), (-2, -2)):
        with pytest.raises(ooc.OocError) as e:
            ctx.set_fixed_distance(*bad)
        assert e.value.status == ooc.E_INVALID
    ctx.set_fixed_distance(-1, -1)
    ctx.close()


def test_wait_order_matches_oracle(lib):
    """The furthest-next-use wait order: random registrations and the small networks, both
    policies, with the window or the fixed-distance rule; schedules and chunk plans op for op."""
    rng = random.Random(91)
    cases = []
    for _ in range(200):
        b, k, f = random_registration(rng, nv=rng.randint(1, 12), nf=rng.randint(1, 20))
        chunk = rng.choice([1, 8, 32])
        ws = S.working_set_max(b, f, chunk)
        cases.append((b, k, f, chunk, rng.choice([ws, ws + chunk, 2 * ws, 10 ** 6]),
                      rng.choice([0, 8, 64, 512, S.INCORE])))
    for spec in specs_small():
        b, k, f = as_schedule_input(lower(spec))
        p = S.incore_peak(b, k, f, 4096)
        ws = S.working_set_max(b, f, 4096)
        for frac in (0.5, 0.25, 0.0):
            B = max(S.budget_for(frac, p, 4096), ws)
            cases.append((b, k, f, 4096, B, B // 2))
    for trial, (b, k, f, chunk, B, W) in enumerate(cases):
        policy = rng.choice("CL")
        fixed = (rng.randint(0, 4), rng.randint(0, 4)) if rng.random() < 0.25 else None
        ctx = ooc.Context(-1)
        for nb, kd in zip(b, k):
            ctx.add_var(nb, kd)
        for vs in f:
            ctx.add_fn("noop", [v for v, _ in vs], [a for _, a in vs])
        ctx.set_chunk(chunk)
        ctx.set_budget(B)
        ctx.set_window(W)
        ctx.set_policy(policy)
        ctx.set_wait_order("furthest")
        if fixed:
            ctx.set_fixed_distance(*fixed)
        kw = {"ahead": fixed[0], "threshold": fixed[1]} if fixed else {}
        try:
            ref = S.build(b, k, f, B, W, chunk, policy, wait="furthest", **kw)
        except S.Infeasible:
            with pytest.raises(ooc.OocError) as e:
                ctx.build_schedule()
            assert e.value.status == ooc.E_INFEASIBLE
            ctx.close()
            continue
        ctx.build_schedule()
        ops, held = ctx.schedule()
        assert ops == ref["ops"], trial
        assert held == ref["held"], trial
        assert ctx.windows() == ref["windows"], trial
        ivs, _ = opool.assign(ref["ops"], b, B // chunk, chunk)
        assert [(g["var"], g["open"], g["close"], g["chunks"]) for g in ctx.plan()] == \
            [(i["var"], i["open"], i["close"], i["chunks"]) for i in ivs]
        ctx.close()
    ctx = ooc.Context(-1)
    with pytest.raises(ooc.OocError) as e:
        ctx.set_wait_order(2)
    assert e.value.status == ooc.E_INVALID
    ctx.set_wait_order("oldest")
    ctx.close()


def test_bestfit_extent_matches_oracle(lib):
    """The contiguous best-fit comparison heap: extent and peak live bytes equal the oracle's on
    random registrations and the small networks, for both policies and several alignments."""
    rng = random.Random(5)
    cases = []
    for _ in range(150):
        b, k, f = random_registration(rng, nv=rng.randint(1, 12), nf=rng.randint(1, 20))
        ws = S.working_set_max(b, f, 1)
        cases.append((b, k, f, rng.choice([ws, ws + 8, 2 * ws])))
    for spec in specs_small():
        b, k, f = as_schedule_input(lower(spec))
        p = S.incore_peak(b, k, f, 1)
        ws = S.working_set_max(b, f, 1)
        for frac in (0.5, 0.25):
            cases.append((b, k, f, max(S.budget_for(frac, p, 1), ws)))
    for trial, (b, k, f, B) in enumerate(cases):
        policy = rng.choice("CL")
        wait = rng.choice(["oldest", "furthest"])
        W = rng.choice([0, B // 2, B])
        align = rng.choice([1, 8, 256])
        ref = S.build(b, k, f, B, W, 1, policy, wait=wait)
        ctx = ooc.Context(-1)
        for nb, kd in zip(b, k):
            ctx.add_var(nb, kd)
        for vs in f:
            ctx.add_fn("noop", [v for v, _ in vs], [a for _, a in vs])
        ctx.set_chunk(1)
        ctx.set_budget(B)
        ctx.set_window(W)
        ctx.set_policy(policy)
        ctx.set_wait_order(wait)
        ctx.build_schedule()
        assert ctx.bestfit_extent(align) == opool.best_fit(ref["ops"], b, align), trial
        ctx.close()


def test_infeasible_budget_reports_error(lib):
    spec = specs_small()[0]
    net = netdef.Net(spec)
    b, k, f = as_schedule_input(lower(spec, slices=net.slices))
    ws = S.working_set_max(b, f, 1)
    ctx = ooc.Context(-1)
    net.register(ctx)
    ctx.set_chunk(1)
    ctx.set_budget(ws - 1)
    with pytest.raises(ooc.OocError) as e:
        ctx.build_schedule()
    assert e.value.status == ooc.E_INFEASIBLE
    ctx.close()


def test_call_order_and_validation(lib):
    ctx = ooc.Context(-1)
    with pytest.raises(ooc.OocError) as e:
        ctx.build_schedule()                       # nothing registered
    assert e.value.status == ooc.E_INVALID
    x = ctx.add_var(64, ooc.INPUT)
    t = ctx.add_var(64, ooc.TEMP)
    with pytest.raises(ooc.OocError) as e:         # TEMP read before written
        ctx.add_fn("relu_fwd", [t, x], [ooc.R, ooc.W], [16])
    assert e.value.status == ooc.E_INVALID
    with pytest.raises(ooc.OocError) as e:         # INPUT written
        ctx.add_fn("noop", [x], [ooc.RW])
    assert e.value.status == ooc.E_INVALID
    with pytest.raises(ooc.OocError) as e:         # sizes contradict the attributes
        ctx.add_fn("relu_fwd", [x, t], [ooc.R, ooc.W], [17])
    assert e.value.status == ooc.E_INVALID
    with pytest.raises(ooc.OocError) as e:         # wrong access pattern
        ctx.add_fn("relu_fwd", [x, t], [ooc.R, ooc.RW], [16])
    with pytest.raises(ooc.OocError) as e:         # unknown op
        ctx.add_fn(99, [x], [ooc.R])
    with pytest.raises(ooc.OocError) as e:         # unknown variable
        ctx.add_fn("noop", [7], [ooc.R])
    ctx.add_fn("relu_fwd", [x, t], [ooc.R, ooc.W], [16])
    with pytest.raises(ooc.OocError) as e:         # out of order
        ctx.prepare()
    assert e.value.status == ooc.E_STATE
    ctx.set_budget(8 << 20)
    ctx.build_schedule()
    with pytest.raises(ooc.OocError) as e:
        ctx.set_budget(5)
    assert e.value.status == ooc.E_STATE
    with pytest.raises(ooc.OocError) as e:
        ctx.add_var(4, ooc.TEMP)
    assert e.value.status == ooc.E_STATE
    with pytest.raises(ooc.OocError) as e:
        ctx.step(0.1)
    assert e.value.status == ooc.E_STATE
    ctx.close()
    with pytest.raises(ooc.OocError):
        ooc.Context(-2)


def test_conv_and_bn_signatures_are_checked(lib):
    ctx = ooc.Context(-1)
    x = ctx.add_var(2 * 8 * 8 * 4 * 4, ooc.INPUT)
    w = ctx.add_var(6 * 3 * 3 * 4 * 4, ooc.PARAM)
    y = ctx.add_var(2 * 8 * 8 * 6 * 4, ooc.TEMP)
    good = [2, 8, 8, 4, 6, 3, 3, 1, 1, 8, 8]
    bad_out = [2, 8, 8, 4, 6, 3, 3, 1, 1, 7, 8]     # P does not follow from H
    with pytest.raises(ooc.OocError):
        ctx.add_fn("conv_fwd", [x, w, y], [ooc.R, ooc.R, ooc.W], bad_out)
    with pytest.raises(ooc.OocError):
        ctx.add_fn("conv_fwd", [x, w, y], [ooc.R, ooc.R, ooc.W], good[:-1])
    ctx.add_fn("conv_fwd", [x, w, y], [ooc.R, ooc.R, ooc.W], good)
    g = ctx.add_var(6 * 4, ooc.PARAM)
    bt = ctx.add_var(6 * 4, ooc.PARAM)
    yb = ctx.add_var(2 * 8 * 8 * 6 * 4, ooc.TEMP)
    st = ctx.add_var((2 + 2 * 3) * 6 * 4, ooc.TEMP)
    with pytest.raises(ooc.OocError):                 # stats too small for 4 slices
        ctx.add_fn("bn_fwd", [y, g, bt, yb, st], [ooc.R] * 3 + [ooc.W] * 2, [128, 6, 4])
    ctx.add_fn("bn_fwd", [y, g, bt, yb, st], [ooc.R] * 3 + [ooc.W] * 2, [128, 6, 3])
    ctx.close()


def test_host_limit_validation(lib):
    """A host limit of 0 is rejected; any positive limit is accepted until prepare (the
    placement itself needs a device)."""
    ctx = ooc.Context(-1)
    try:
        with pytest.raises(ooc.OocError) as e:
            ctx.set_host_limit(0)
        assert e.value.status == ooc.E_INVALID
        ctx.set_host_limit(1)
        ctx.set_host_limit(56 << 30)
        x = ctx.add_var(64, ooc.INPUT)
        t = ctx.add_var(64, ooc.TEMP)
        ctx.add_fn("relu_fwd", [x, t], [ooc.R, ooc.W], [16])
        ctx.build_schedule()
        ctx.set_host_limit(ooc.UNLIMITED)           # still allowed after the schedule
    finally:
        ctx.close()


def test_queries_report_status_and_message(lib):
    """Each query: a NULL out-pointer (or a NULL buffer with a capacity) is OOC_E_INVALID, a
    query before the stage it needs is OOC_E_STATE, and either way ooc_last_error names the
    call.  A NULL context is OOC_E_INVALID with its message on ooc_last_error(NULL)."""
    import ctypes as C
    ctx = ooc.Context(-1)
    a = ctx.add_var(64, ooc.INPUT)
    t = ctx.add_var(64, ooc.TEMP)
    ctx.add_fn("relu_fwd", [a, t], [ooc.R, ooc.W], [16])
    ctx.set_chunk(1)
    h = ctx.h
    u64, i64 = C.c_uint64(), C.c_int64()

    def expect(status, call, name):
        assert call == status, name
        msg = lib.ooc_last_error(h).decode()
        assert msg.startswith(name), (name, msg)

    n = C.byref(u64)
    # before ooc_build_schedule
    for name, f in (("ooc_schedule_get", lambda: lib.ooc_schedule_get(h, None, 0, n)),
                    ("ooc_schedule_windows", lambda: lib.ooc_schedule_windows(h, None, 0, n)),
                    ("ooc_plan_intervals", lambda: lib.ooc_plan_intervals(h, None, 0, n)),
                    ("ooc_plan_chunks", lambda: lib.ooc_plan_chunks(h, None, 0, n)),
                    ("ooc_bestfit_extent", lambda: lib.ooc_bestfit_extent(h, 8, n, n)),
                    ("ooc_get_stats", lambda: lib.ooc_get_stats(h, C.byref(ooc.ooc_stats()))),
                    ("ooc_fn_times", lambda: lib.ooc_fn_times(h, None, 0, n))):
        expect(ooc.E_STATE, f(), name)
    # NULL out-pointers and buffers
    for name, f in (("ooc_schedule_get", lambda: lib.ooc_schedule_get(h, None, 0, None)),
                    ("ooc_schedule_get", lambda: lib.ooc_schedule_get(h, None, 4, n)),
                    ("ooc_schedule_windows", lambda: lib.ooc_schedule_windows(h, None, 0, None)),
                    ("ooc_schedule_windows", lambda: lib.ooc_schedule_windows(h, None, 2, n)),
                    ("ooc_incore_peak", lambda: lib.ooc_incore_peak(h, None)),
                    ("ooc_working_set_max", lambda: lib.ooc_working_set_max(h, None)),
                    ("ooc_plan_intervals", lambda: lib.ooc_plan_intervals(h, None, 0, None)),
                    ("ooc_plan_intervals", lambda: lib.ooc_plan_intervals(h, None, 3, n)),
                    ("ooc_plan_chunks", lambda: lib.ooc_plan_chunks(h, None, 0, None)),
                    ("ooc_plan_chunks", lambda: lib.ooc_plan_chunks(h, None, 3, n)),
                    ("ooc_bestfit_extent", lambda: lib.ooc_bestfit_extent(h, 8, None, n)),
                    ("ooc_bestfit_extent", lambda: lib.ooc_bestfit_extent(h, 8, n, None)),
                    ("ooc_get_stats", lambda: lib.ooc_get_stats(h, None)),
                    ("ooc_fn_times", lambda: lib.ooc_fn_times(h, None, 0, None)),
                    ("ooc_fn_times", lambda: lib.ooc_fn_times(h, None, 2, n)),
                    ("ooc_timeline", lambda: lib.ooc_timeline(h, None, 0, None)),
                    ("ooc_timeline", lambda: lib.ooc_timeline(h, None, 2, n))):
        expect(ooc.E_INVALID, f(), name)
    assert lib.ooc_incore_peak(h, n) == ooc.OK and u64.value == 128
    ctx.build_schedule()
    expect(ooc.E_INVALID, lib.ooc_bestfit_extent(h, 12, n, n), "ooc_bestfit_extent")
    assert lib.ooc_bestfit_extent(h, 8, n, C.byref(C.c_uint64())) == ooc.OK
    assert lib.ooc_schedule_get(h, None, 0, n) == ooc.OK and u64.value == len(ctx.schedule()[0])
    # stages past the schedule: a host-only context cannot prepare, so no slot and no step
    p = C.c_void_p()
    expect(ooc.E_STATE, lib.ooc_host_ptr(h, a, C.byref(p)), "ooc_host_ptr")
    expect(ooc.E_STATE, lib.ooc_step(h, C.c_float(0.1), C.c_float(0.0), None), "ooc_step")
    expect(ooc.E_STATE, lib.ooc_timeline(h, None, 0, n), "no step")
    assert lib.ooc_prepare(h) == ooc.E_UNSUPPORTED
    assert "host-only" in lib.ooc_last_error(h).decode()
    ctx.close()
    # a NULL context
    for name, f in (("ooc_incore_peak", lambda: lib.ooc_incore_peak(None, n)),
                    ("ooc_get_stats", lambda: lib.ooc_get_stats(None, None)),
                    ("ooc_step", lambda: lib.ooc_step(None, C.c_float(0.1), C.c_float(0.0), None))):
        assert f() == ooc.E_INVALID
        assert lib.ooc_last_error(None).decode() == name + ": NULL context"
    assert lib.ooc_create(0, None) == ooc.E_INVALID
    assert lib.ooc_last_error(None).decode() == "ooc_create: out is NULL"
    assert lib.ooc_wgrad_slices(10, None, 0, C.byref(i64)) == ooc.E_INVALID
    assert lib.ooc_last_error(None).decode().startswith("ooc_wgrad_slices")


def test_bestfit_layout_keeps_live_intervals_apart(lib):
    """OOC_LAYOUT_BESTFIT: the same schedule as the chunk pool, and every two residency
    intervals alive at the same time cover disjoint heap segments (so no two live copies share
    device bytes); the heap's extent is the one ooc_bestfit_extent reports at 256-byte
    alignment."""
    rng = random.Random(31)
    cases = []
    for _ in range(60):
        b, k, f = random_registration(rng, nv=rng.randint(1, 12), nf=rng.randint(1, 20))
        ws = S.working_set_max(b, f, 8)
        cases.append((b, k, f, rng.choice([ws, 2 * ws, 10 ** 6])))
    for spec in specs_small():
        net = netdef.Net(spec)
        b, k, f = net.var_bytes, net.var_kinds, net.fn_vars
        p = S.incore_peak(b, k, f, 4096)
        cases.append((b, k, f, max(S.budget_for(0.25, p, 4096), S.working_set_max(b, f, 4096))))
    for trial, (b, k, f, B) in enumerate(cases):
        ctxs = []
        for layout in ("pool", "bestfit"):
            ctx = ooc.Context(-1)
            for nb, kd in zip(b, k):
                ctx.add_var(nb, kd)
            for vs in f:
                ctx.add_fn("noop", [v for v, _ in vs], [a for _, a in vs])
            ctx.set_chunk(8 if B < 10 ** 6 or trial < 60 else 4096)
            ctx.set_budget(B)
            ctx.set_layout(layout)
            ctx.build_schedule()
            ctxs.append(ctx)
        pool, best = ctxs
        assert pool.schedule() == best.schedule(), trial
        ivs = best.plan()
        nops = len(best.schedule()[0])
        span = [(iv["open"] if iv["open"] >= 0 else -1,
                 iv["close"] if iv["close"] >= 0 else nops) for iv in ivs]
        for x in range(len(ivs)):
            for y in range(x + 1, len(ivs)):
                if span[x][0] < span[y][1] and span[y][0] < span[x][1]:
                    assert not set(ivs[x]["chunks"]) & set(ivs[y]["chunks"]), (trial, x, y)
        extent, _ = pool.bestfit_extent(256)
        assert best.stats()["max_chunks_used"] == pool.stats()["max_chunks_used"]
        assert best.bestfit_extent(256)[0] == extent
        for c in ctxs:
            c.close()
    ctx = ooc.Context(-1)
    with pytest.raises(ooc.OocError) as e:
        ctx.set_layout(2)
    assert e.value.status == ooc.E_INVALID
    ctx.close()

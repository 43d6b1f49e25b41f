"""Helpers of the GPU tests: run a registered network through the library."""

import numpy as np

from paper_2010_14109_amd import netdef, ooc


def run_net(spec, x, labels, params, *, budget=ooc.UNLIMITED, window=None, chunk=2 << 20,
            policy="C", keep_grads=True, momentum_state=None, steps=1, inspect=None,
            wait="oldest", host_limit=None, fixed=None, layout="pool"):
    """One (or more) training steps on device 0.  Returns (loss, outputs, stats) with
    outputs = {name: array} for every PARAM, STATE and OUTPUT variable.  ``inspect(ctx,
    net)``, when given, runs after the steps."""
    net = netdef.Net(spec, keep_grads=keep_grads)
    ctx = ooc.Context(0)
    try:
        net.register(ctx)
        ctx.set_chunk(chunk)
        ctx.set_budget(budget)
        if window is not None:
            ctx.set_window(window)
        ctx.set_policy(policy)
        ctx.set_wait_order(wait)
        if host_limit is not None:
            ctx.set_host_limit(host_limit)
        if fixed is not None:
            ctx.set_fixed_distance(*fixed)
        ctx.set_layout(layout)
        ctx.build_schedule()
        ctx.prepare()
        net.view(ctx, "x")[...] = x
        net.view(ctx, "labels")[...] = labels
        for name in net.param_names():
            net.view(ctx, name)[...] = params[name]
        for name in net.names:
            if name.startswith("m:"):
                st = (momentum_state or {}).get(name)
                net.view(ctx, name)[...] = 0 if st is None else st
        ctx.upload()
        mu = spec["optimizer"]["momentum"]
        losses = [ctx.step(spec["optimizer"]["lr"], mu) for _ in range(steps)]
        if inspect is not None:
            inspect(ctx, net)
        ctx.download()
        outs = {}
        for name in net.names:
            if net.meta[name][2] in (ooc.PARAM, ooc.STATE, ooc.OUTPUT):
                outs[name] = np.array(net.view(ctx, name))
        return losses[-1], outs, ctx.stats()
    finally:
        ctx.close()


def persistent_host_bytes(spec, keep_grads=True):
    """Bytes of the pinned slots of the persistent variables (4 KiB-aligned each)."""
    net = netdef.Net(spec, keep_grads=keep_grads)
    return sum((b + 4095) // 4096 * 4096 for b, k in zip(net.var_bytes, net.var_kinds)
               if k != ooc.TEMP)


STAGING_BYTES = 2 << 30   # the staging slots a host limit reserves


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def rel_max(a, b):
    """Largest element error relative to the largest element of b."""
    a = np.asarray(a, dtype=np.float64).reshape(-1)
    b = np.asarray(b, dtype=np.float64).reshape(-1)
    return float(np.abs(a - b).max(initial=0.0) / max(np.abs(b).max(initial=0.0), 1e-30))


def rel_err(a, b):
    """The larger of the relative L2 error and the element-wise one (rel_max): one wrong
    element among millions barely moves the norm but shows in the largest element error."""
    return max(rel_l2(a, b), rel_max(a, b))


def within_fp32_error(name, got, ref, ref32, tol, factor=1.5, element_factor=3.0):
    """Where float32 evaluation itself is ill-conditioned (ReLU masks and max-pool choices
    flipped by rounding), the device's error against float64 is bounded by the float32
    oracle's own: its relative L2 error at most max(tol, factor times the float32 oracle's),
    and its largest element error (relative to the largest element) at most max(tol,
    element_factor times the float32 oracle's).  The largest element error is an extreme value
    of whichever decisions flip, and two float32 evaluations flip different ones, so it varies
    between them more than the L2 error does; a single wrong element of typical size still
    shows wherever the float32 oracle's own largest error is below a third of the largest
    element.  Returns the two ratios error / bound."""
    got = np.asarray(got).reshape(np.shape(ref))
    r32 = np.asarray(ref32).reshape(np.shape(ref))
    l2 = rel_l2(got, ref) / max(tol, factor * rel_l2(r32, ref))
    mx = rel_max(got, ref) / max(tol, element_factor * rel_max(r32, ref))
    assert l2 <= 1.0 and mx <= 1.0, (name, l2, mx)
    return l2, mx

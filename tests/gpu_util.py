"""Helpers of the GPU tests: run a registered network through the library."""

import numpy as np

from paper_2010_14109_amd import netdef, ooc


def run_net(spec, x, labels, params, *, budget=ooc.UNLIMITED, window=None, chunk=2 << 20,
            policy="C", keep_grads=True, momentum_state=None, steps=1, inspect=None,
            wait="oldest", host_limit=None, fixed=None):
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

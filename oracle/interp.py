"""Runs a function sequence with the textbook ops: one training step (test infrastructure).

The result of an out-of-core step equals that of the ordinary in-core step,
because swaps only move bytes (Section 1, Section 3); this interpreter is that
ordinary step.  It executes the functions of ``oracle.lower`` in order, in
the given dtype (float64 for parity), and returns every variable's final
value, so tests can compare the loss, parameter gradients and updated
parameters with the device.
"""

from __future__ import annotations

import numpy as np

from . import ops


def run(reg, x, labels, params, state=None, dtype=np.float64):
    """One step.  ``params`` / ``state``: {name: array}.  Returns {var name: array}.

    ``state`` holds momentum buffers by name (``m:<param>``); missing ones start at 0.
    """
    state = state or {}
    names = [v["name"] for v in reg["vars"]]
    env = {}
    for v in reg["vars"]:
        nm = v["name"]
        if nm == "x":
            env[nm] = np.asarray(x, dtype=np.int64 if v["dtype"] == "i32" else dtype)
        elif nm == "labels":
            env[nm] = np.asarray(labels, dtype=np.int64)
        elif v["kind"] == 1:
            env[nm] = np.asarray(params[nm], dtype=dtype).copy()
        elif v["kind"] == 2:
            env[nm] = np.asarray(state.get(nm, np.zeros(v["shape"])), dtype=dtype).copy()
    bnstat = {}
    for f in reg["fns"]:
        op, a = f["op"], f["attrs"]
        vs = [names[i] for i, _ in f["vars"]]
        g = env.get
        if op == "linear_fwd":
            X, Wn, b, Y = vs
            env[Y] = ops.linear_fwd(g(X), g(Wn), g(b))
        elif op == "conv_fwd":
            X, Wn, Y = vs
            env[Y] = ops.conv_fwd(g(X), g(Wn), a["stride"], a["pad"])
        elif op == "bn_fwd":
            X, gm, bt, Y, st = vs
            env[Y], mean, invstd = ops.bn_fwd(g(X), g(gm), g(bt))
            bnstat[st] = (mean, invstd)
            env[st] = np.concatenate([mean, invstd, np.zeros(2 * a["slices"] * a["C"])])
        elif op == "relu_fwd":
            X, Y = vs
            env[Y] = ops.relu_fwd(g(X))
        elif op == "maxpool_fwd":
            X, Y, ix = vs
            env[Y], env[ix] = ops.maxpool_fwd(g(X), a["k"], a["stride"], a["pad"])
        elif op == "avgpool_fwd":
            X, Y = vs
            env[Y] = ops.avgpool_fwd(g(X))
        elif op == "add_fwd":
            A, B, Y = vs
            env[Y] = g(A) + g(B)
        elif op == "softmax_ce":
            lg, lb, loss, dl = vs
            logits = g(lg)          # per-pixel logits: one row per position of the last axis
            rows, mean, d = ops.softmax_ce(logits.reshape(-1, logits.shape[-1]), g(lb))
            env[dl] = d.reshape(logits.shape)
            env[loss] = np.concatenate([rows, [mean]])
        elif op == "linear_bwd_w":
            X, dY, dW, db = vs[:4]
            env[dW], env[db] = ops.linear_bwd_w(g(X), g(dY))
        elif op == "linear_bwd_x":
            Wn, dY, dX = vs
            env[dX] = ops.linear_bwd_x(g(Wn), g(dY))
        elif op == "conv_bwd_w":
            X, dY, dW = vs[:3]
            shape = (a["K"], a["R"], a["S"], a["C"])
            env[dW] = ops.conv_bwd_w(g(X), g(dY), shape, a["stride"], a["pad"])
        elif op == "conv_bwd_x":
            Wn, dY, dX = vs
            shape = (a["N"], a["H"], a["W"], a["C"])
            env[dX] = ops.conv_bwd_x(g(Wn), g(dY), shape, a["stride"], a["pad"])
        elif op == "bn_bwd":
            X, gm, st, dY, dX, dg, dbt = vs
            mean, invstd = bnstat[st]
            env[dX], env[dg], env[dbt] = ops.bn_bwd(g(X), g(gm), mean, invstd, g(dY))
        elif op == "relu_bwd":
            Y, dY, dX = vs
            env[dX] = ops.relu_bwd(g(Y), g(dY))
        elif op == "maxpool_bwd":
            ix, dY, dX = vs
            shape = (a["N"], a["H"], a["W"], a["C"])
            env[dX] = ops.maxpool_bwd(g(ix), g(dY), shape, a["k"], a["stride"], a["pad"])
        elif op == "avgpool_bwd":
            dY, dX = vs
            env[dX] = ops.avgpool_bwd(g(dY), (a["N"], a["H"], a["W"], a["C"]))
        elif op == "add_grad":
            A, B, Y = vs
            env[Y] = g(A) + g(B)
        elif op == "acc_grad":
            A, B = vs
            env[A] = g(A) + g(B)
        elif op == "sgd":
            lr, mu = a["lr"], a["momentum"]
            step = 3 if mu else 2
            for j in range(0, len(vs), step):
                p, dp = vs[j], vs[j + 1]
                if mu:
                    m = vs[j + 2]
                    env[p], env[m] = ops.sgd_momentum(g(p), g(dp), g(m), lr, mu)
                else:
                    env[p] = ops.sgd(g(p), g(dp), lr)
        elif op == "embed_fwd":
            ids, E, pos, Y = vs
            env[Y] = ops.embed_fwd(g(ids), g(E), g(pos))
        elif op == "embed_bwd":
            ids, dY, dE, dpos = vs
            env[dE], env[dpos] = ops.embed_bwd(g(ids), g(dY), a["V"])
        elif op == "layernorm_fwd":
            X, gm, bt, Y, st = vs
            env[Y], mean, rstd = ops.layernorm_fwd(g(X), g(gm), g(bt))
            bnstat[st] = (mean, rstd)
            env[st] = np.concatenate([mean, rstd, np.zeros(2 * a["slices"] * a["d"])])
        elif op == "layernorm_bwd":
            X, gm, st, dY, dX, dg, dbt = vs
            mean, rstd = bnstat[st]
            env[dX], env[dg], env[dbt] = ops.layernorm_bwd(g(X), g(gm), mean, rstd, g(dY))
        elif op == "gelu_fwd":
            X, Y = vs
            env[Y] = ops.gelu_fwd(g(X))
        elif op == "gelu_bwd":
            X, dY, dX = vs
            env[dX] = ops.gelu_bwd(g(X), g(dY))
        elif op == "concat_fwd":
            env[vs[-1]] = ops.concat_fwd([g(v) for v in vs[:-1]])
        elif op == "concat_bwd":
            parts = ops.concat_bwd(g(vs[0]), a["cs"])
            for v, part in zip(vs[1:], parts):
                env[v] = part
        elif op == "upsample_fwd":
            X, Y = vs
            env[Y] = ops.upsample_fwd(g(X))
        elif op == "upsample_bwd":
            dY, dX = vs
            env[dX] = ops.upsample_bwd(g(dY))
        elif op == "attention_fwd":
            X, Pv, Y = vs
            env[Pv], env[Y] = ops.attention_fwd(g(X), a["B"], a["T"], a["H"], bool(a["causal"]))
        elif op == "attention_bwd":
            # the probabilities are recomputed from q and k, not kept from the forward
            X, Pb, dY, dX, dS = vs
            env[Pb] = ops.attention_fwd(g(X), a["B"], a["T"], a["H"], bool(a["causal"]))[0]
            env[dX] = ops.attention_bwd(g(X), env[Pb], g(dY), a["B"], a["T"], a["H"])
            env[dS] = np.zeros_like(env[Pb])
        else:
            raise ValueError(f"unknown function {op}")
    return env

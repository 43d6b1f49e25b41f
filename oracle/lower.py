"""Oracle lowering: network description -> function sequence (Section 2, Fig. 1).

Test infrastructure.  The paper runs a network as the topologically ordered
sequence of its functions and lists, for each function, the variables it
uses.  One training step of a layer-sequential network becomes:

1. the forward functions in layer order;
2. the fused softmax cross-entropy (mean loss and the logits gradient);
3. for every layer in reverse order: its backward functions, then one SGD
   function for its parameters, then the sums of the gradient contributions
   of tensors with several consumers, in the order the contributions appear:
   a contribution is added in place into the tensor's running gradient
   (``acc_grad``), except while that running gradient variable is also the
   gradient of another tensor whose layer's backward is still to come (an
   addition passes its output gradient to both inputs); then it is added
   into a new variable (``add_grad``).

Variables are numbered by first appearance in the flattened sequence.  Each
function lists ``(variable, access)`` pairs in this fixed order:

=============  ======================================================================
linear_fwd     X R, W R, b R, Y W
conv_fwd       X R, W R, Y W
bn_fwd         X R, gamma R, beta R, Y W, stats W
relu_fwd       X R, Y W
maxpool_fwd    X R, Y W, idx W
avgpool_fwd    X R, Y W
add_fwd        A R, B R, Y W
softmax_ce     logits R, labels R, loss W, dlogits W
linear_bwd_w   X R, dY R, dW W, db W [, part W] (part only when split into > 1 slice)
linear_bwd_x   W R, dY R, dX W            (absent when X is the network input)
conv_bwd_w     X R, dY R, dW W [, part W] (part only when split into > 1 slice)
conv_bwd_x     W R, dY R, dX W            (absent when X is the network input)
bn_bwd         X R, gamma R, stats RW, dY R, dX W, dgamma W, dbeta W
relu_bwd       Y R, dY R, dX W            (Y = the ReLU output)
maxpool_bwd    idx R, dY R, dX W
avgpool_bwd    dY R, dX W
add_grad       g R, c R, g' W             (g' = g + c)
acc_grad       g RW, c R                  (g = g + c)
sgd            per parameter p in layer order: p RW, dp R [, m_p RW with momentum]
embed_fwd      ids R, E R, pos R, Y W
embed_bwd      ids R, dY R, dE W, dpos W
layernorm_fwd  X R, gamma R, beta R, Y W, stats W
layernorm_bwd  X R, gamma R, stats RW, dY R, dX W, dgamma W, dbeta W
gelu_fwd       X R, Y W
gelu_bwd       X R, dY R, dX W            (X = the GELU input)
attention_fwd  qkv R, P W, Y W            (P = the attention probabilities [B, H, T, T])
attention_bwd  qkv R, P' W, dY R, dqkv W, dS W  (P' = P recomputed, dS = scratch)
concat_fwd     X_1 R, ..., X_k R, Y W          (channel concatenation)
concat_bwd     dY R, dX_1 W, ..., dX_k W
upsample_fwd   X R, Y W                        (nearest, factor 2)
upsample_bwd   dY R, dX W
=============  ======================================================================

The backward of an addition is the identity, so both inputs receive the
output gradient itself and no function is emitted for it.

Sizes: float32 tensors except ``labels`` (int32) and ``idx`` (uint8);
``loss`` holds the per-row losses followed by their mean ([N + 1]);
``stats`` holds mean and 1/std per channel followed by two partial sums per
channel for each of S row slices, S = min(ceil(rows / 512), 2048) with rows =
N H W; a LayerNorm's ``stats`` holds mean and 1/std per row followed by two
partial sums per feature for each of S row slices, S = min(ceil(rows / 32),
2048); a convolution's
``part`` holds S_w slices of dW and a dense layer's S_w slices of dW then
S_w slices of db, S_w being given per layer by the caller (``lower``'s
``slices``).

Kinds: x and labels INPUT, parameters PARAM, momentum buffers STATE, loss
OUTPUT (parameter gradients too when ``keep_grads``), everything else TEMP.
Token inputs (``x`` of a transformer) are int32 [B, T]; there is one label per
row of the logits.
"""

from __future__ import annotations

import math

INPUT, PARAM, STATE, OUTPUT, TEMP = 0, 1, 2, 3, 4
R, W, RW = 1, 2, 3
ITEMSIZE = {"f32": 4, "i32": 4, "u8": 1}


def bn_slices(rows):
    return min(math.ceil(rows / 512), 2048)


def ln_slices(rows):
    return min(math.ceil(rows / 32), 2048)


def lower(spec, keep_grads=False, slices=None):
    """Returns ``{"vars": [...], "fns": [...]}``.

    ``slices`` maps a convolution or dense layer's name to the number S_w of
    partial sums its weight gradient is split into (1 when absent).  The count
    is a blocking choice of whoever computes the gradient, taken as an input:
    it only sizes the ``part`` variable, since the gradient is the same sum
    for every S_w.

    ``vars[i] = {"name", "shape", "dtype", "kind", "bytes"}``;
    ``fns[j] = {"op", "vars": [(id, access)], "attrs": {...}}``.
    """
    shapes = {"x": tuple(spec["input"])}
    decl = {}          # name -> (shape, dtype, kind)
    fns = []           # (op, [(name, access)], attrs)
    momentum = spec["optimizer"]["momentum"]
    grad_kind = OUTPUT if keep_grads else TEMP

    def var(name, shape, dtype="f32", kind=TEMP):
        decl[name] = (tuple(shape), dtype, kind)
        return name

    var("x", spec["input"], dtype="i32" if spec.get("tokens") else "f32", kind=INPUT)
    params_of = {}

    # ---------------- forward
    for L in spec["layers"]:
        op, name = L["op"], L["name"]
        ins = L["in"]
        X = ins[0]
        xs = shapes[X]
        if op == "linear":
            Wn = var(name + ".W", (L["out_features"], L["in_features"]), kind=PARAM)
            bn_ = var(name + ".b", (L["out_features"],), kind=PARAM)
            shapes[name] = (xs[0], L["out_features"])
            var(name, shapes[name])
            params_of[name] = [Wn, bn_]
            fns.append(("linear_fwd", [(X, R), (Wn, R), (bn_, R), (name, W)],
                        {"M": xs[0], "K": xs[1], "N": L["out_features"]}))
        elif op == "conv":
            n, h, w, c = xs
            k, st, pd = L["k"], L["stride"], L["pad"]
            P, Q = (h + 2 * pd - k) // st + 1, (w + 2 * pd - k) // st + 1
            Wn = var(name + ".W", (L["cout"], k, k, c), kind=PARAM)
            shapes[name] = (n, P, Q, L["cout"])
            var(name, shapes[name])
            params_of[name] = [Wn]
            fns.append(("conv_fwd", [(X, R), (Wn, R), (name, W)],
                        {"N": n, "H": h, "W": w, "C": c, "K": L["cout"], "R": k, "S": k,
                         "stride": st, "pad": pd, "P": P, "Q": Q}))
        elif op == "bn":
            c = xs[-1]
            rows = math.prod(xs[:-1])
            S = bn_slices(rows)
            g = var(name + ".gamma", (c,), kind=PARAM)
            bt = var(name + ".beta", (c,), kind=PARAM)
            st_ = var(name + ".stats", ((2 + 2 * S) * c,))
            shapes[name] = xs
            var(name, xs)
            params_of[name] = [g, bt]
            fns.append(("bn_fwd", [(X, R), (g, R), (bt, R), (name, W), (st_, W)],
                        {"rows": rows, "C": c, "slices": S}))
        elif op == "relu":
            shapes[name] = xs
            var(name, xs)
            fns.append(("relu_fwd", [(X, R), (name, W)], {"n": math.prod(xs)}))
        elif op == "maxpool":
            n, h, w, c = xs
            k, st, pd = L["k"], L["stride"], L["pad"]
            P, Q = (h + 2 * pd - k) // st + 1, (w + 2 * pd - k) // st + 1
            shapes[name] = (n, P, Q, c)
            var(name, shapes[name])
            ix = var(name + ".idx", shapes[name], dtype="u8")
            fns.append(("maxpool_fwd", [(X, R), (name, W), (ix, W)],
                        {"N": n, "H": h, "W": w, "C": c, "k": k, "stride": st, "pad": pd,
                         "P": P, "Q": Q}))
        elif op == "avgpool":
            n, h, w, c = xs
            shapes[name] = (n, c)
            var(name, shapes[name])
            fns.append(("avgpool_fwd", [(X, R), (name, W)], {"N": n, "H": h, "W": w, "C": c}))
        elif op == "add":
            B = ins[1]
            assert shapes[B] == xs
            shapes[name] = xs
            var(name, xs)
            fns.append(("add_fwd", [(X, R), (B, R), (name, W)], {"n": math.prod(xs)}))
        elif op == "embed":
            Bt, T = xs
            d = L["d"]
            E = var(name + ".E", (L["vocab"], d), kind=PARAM)
            pos = var(name + ".pos", (T, d), kind=PARAM)
            shapes[name] = (Bt * T, d)
            var(name, shapes[name])
            params_of[name] = [E, pos]
            fns.append(("embed_fwd", [(X, R), (E, R), (pos, R), (name, W)],
                        {"B": Bt, "T": T, "V": L["vocab"], "d": d}))
        elif op == "layernorm":
            rows, d = xs
            S = ln_slices(rows)
            g = var(name + ".gamma", (d,), kind=PARAM)
            bt = var(name + ".beta", (d,), kind=PARAM)
            st_ = var(name + ".stats", (2 * rows + 2 * S * d,))
            shapes[name] = xs
            var(name, xs)
            params_of[name] = [g, bt]
            fns.append(("layernorm_fwd", [(X, R), (g, R), (bt, R), (name, W), (st_, W)],
                        {"rows": rows, "d": d, "slices": S}))
        elif op == "gelu":
            shapes[name] = xs
            var(name, xs)
            fns.append(("gelu_fwd", [(X, R), (name, W)], {"n": math.prod(xs)}))
        elif op == "concat":
            lead = xs[:-1]
            assert all(shapes[s][:-1] == lead for s in ins) and len(set(ins)) == len(ins)
            cs = [shapes[s][-1] for s in ins]
            shapes[name] = lead + (sum(cs),)
            var(name, shapes[name])
            fns.append(("concat_fwd", [(s, R) for s in ins] + [(name, W)],
                        {"rows": math.prod(lead), "cs": cs}))
        elif op == "upsample":
            n, h, w, c = xs
            shapes[name] = (n, 2 * h, 2 * w, c)
            var(name, shapes[name])
            fns.append(("upsample_fwd", [(X, R), (name, W)], {"N": n, "H": h, "W": w, "C": c}))
        elif op == "attention":
            rows, d3 = xs
            d, H = d3 // 3, L["heads"]
            Bt, T = spec["input"]
            Pv = var(name + ".P", (Bt, H, T, T))
            shapes[name] = (rows, d)
            var(name, shapes[name])
            fns.append(("attention_fwd", [(X, R), (Pv, W), (name, W)],
                        {"B": Bt, "T": T, "H": H, "dh": d // H, "causal": int(L["causal"])}))
        else:
            raise ValueError(f"unknown layer kind {op}")

    # ---------------- loss
    logits = spec["logits"]
    N, ncls = math.prod(shapes[logits][:-1]), shapes[logits][-1]   # rows of the last axis
    var("labels", (N,), dtype="i32", kind=INPUT)
    var("loss", (N + 1,), kind=OUTPUT)
    dlog = var("d:" + logits, shapes[logits])
    fns.append(("softmax_ce", [(logits, R), ("labels", R), ("loss", W), (dlog, W)],
                {"N": N, "classes": ncls}))

    # ---------------- backward + update
    grad = {logits: dlog}
    count = {}

    def contribute(tensor, g, pending):
        if tensor == "x":
            return
        pending.append((tensor, g))

    done = set()        # tensors whose layer's backward is already in the sequence

    def held_elsewhere(g, tensor):
        """True when g is also the gradient of another tensor still waiting for its layer's
        backward, which will read it."""
        return any(t != tensor and t not in done and grad[t] == g for t in grad)

    def settle(pending):
        for tensor, g in pending:
            if tensor not in grad:
                grad[tensor] = g
            elif g != grad[tensor] and not held_elsewhere(grad[tensor], tensor):
                # running gradient += contribution, in place
                fns.append(("acc_grad", [(grad[tensor], RW), (g, R)],
                            {"n": math.prod(shapes[tensor])}))
            else:
                count[tensor] = count.get(tensor, 1) + 1
                new = var(f"d:{tensor}#{count[tensor]}", shapes[tensor])
                fns.append(("add_grad", [(grad[tensor], R), (g, R), (new, W)],
                            {"n": math.prod(shapes[tensor])}))
                grad[tensor] = new

    def update(layer_name):
        vs = []
        for p in params_of[layer_name]:
            vs.append((p, RW))
            vs.append(("d:" + p, R))
            if momentum:
                m = var("m:" + p, decl[p][0], kind=STATE)
                vs.append((m, RW))
        fns.append(("sgd", vs, {"lr": spec["optimizer"]["lr"], "momentum": momentum,
                                "sizes": [math.prod(decl[p][0]) for p in params_of[layer_name]]}))

    for L in reversed(spec["layers"]):
        op, name = L["op"], L["name"]
        if name not in grad:
            continue
        dY = grad[name]
        X = L["in"][0]
        xs = shapes[X]
        pending = []
        if op == "linear":
            Wn, bn_ = params_of[name]
            dW = var("d:" + Wn, decl[Wn][0], kind=grad_kind)
            db = var("d:" + bn_, decl[bn_][0], kind=grad_kind)
            attrs = {"M": xs[0], "K": xs[1], "N": L["out_features"]}
            Sw = int((slices or {}).get(name, 1))
            vs = [(X, R), (dY, R), (dW, W), (db, W)]
            if Sw > 1:
                vs.append((var(name + ".part", (Sw * (attrs["N"] * attrs["K"] + attrs["N"]),)), W))
            fns.append(("linear_bwd_w", vs, dict(attrs, slices=Sw)))
            if X != "x":
                dX = var(f"d:{X}@{name}", xs)
                fns.append(("linear_bwd_x", [(Wn, R), (dY, R), (dX, W)], attrs))
                contribute(X, dX, pending)
            update(name)
        elif op == "conv":
            (Wn,) = params_of[name]
            n, h, w, c = xs
            _, P, Q, K = shapes[name]
            k = L["k"]
            attrs = {"N": n, "H": h, "W": w, "C": c, "K": K, "R": k, "S": k,
                     "stride": L["stride"], "pad": L["pad"], "P": P, "Q": Q}
            dW = var("d:" + Wn, decl[Wn][0], kind=grad_kind)
            Sw = int((slices or {}).get(name, 1))
            vs = [(X, R), (dY, R), (dW, W)]
            if Sw > 1:
                vs.append((var(name + ".part", (Sw * K * k * k * c,)), W))
            fns.append(("conv_bwd_w", vs, dict(attrs, slices=Sw)))
            if X != "x":
                dX = var(f"d:{X}@{name}", xs)
                fns.append(("conv_bwd_x", [(Wn, R), (dY, R), (dX, W)], attrs))
                contribute(X, dX, pending)
            update(name)
        elif op == "bn":
            g, bt = params_of[name]
            dX = var(f"d:{X}@{name}", xs)
            dg = var("d:" + g, decl[g][0], kind=grad_kind)
            dbt = var("d:" + bt, decl[bt][0], kind=grad_kind)
            rows = math.prod(xs[:-1])
            fns.append(("bn_bwd", [(X, R), (g, R), (name + ".stats", RW), (dY, R), (dX, W),
                                   (dg, W), (dbt, W)],
                        {"rows": rows, "C": xs[-1], "slices": bn_slices(rows)}))
            contribute(X, dX, pending)
            update(name)
        elif op == "relu":
            dX = var(f"d:{X}@{name}", xs)
            fns.append(("relu_bwd", [(name, R), (dY, R), (dX, W)], {"n": math.prod(xs)}))
            contribute(X, dX, pending)
        elif op == "maxpool":
            n, h, w, c = xs
            _, P, Q, _ = shapes[name]
            dX = var(f"d:{X}@{name}", xs)
            fns.append(("maxpool_bwd", [(name + ".idx", R), (dY, R), (dX, W)],
                        {"N": n, "H": h, "W": w, "C": c, "k": L["k"], "stride": L["stride"],
                         "pad": L["pad"], "P": P, "Q": Q}))
            contribute(X, dX, pending)
        elif op == "avgpool":
            n, h, w, c = xs
            dX = var(f"d:{X}@{name}", xs)
            fns.append(("avgpool_bwd", [(dY, R), (dX, W)], {"N": n, "H": h, "W": w, "C": c}))
            contribute(X, dX, pending)
        elif op == "add":
            for src in L["in"]:
                contribute(src, dY, pending)
        elif op == "embed":
            E, pos = params_of[name]
            dE = var("d:" + E, decl[E][0], kind=grad_kind)
            dpos = var("d:" + pos, decl[pos][0], kind=grad_kind)
            fns.append(("embed_bwd", [(X, R), (dY, R), (dE, W), (dpos, W)],
                        {"B": xs[0], "T": xs[1], "V": L["vocab"], "d": L["d"]}))
            update(name)
        elif op == "layernorm":
            g, bt = params_of[name]
            rows, d = xs
            dX = var(f"d:{X}@{name}", xs)
            dg = var("d:" + g, decl[g][0], kind=grad_kind)
            dbt = var("d:" + bt, decl[bt][0], kind=grad_kind)
            fns.append(("layernorm_bwd", [(X, R), (g, R), (name + ".stats", RW), (dY, R),
                                          (dX, W), (dg, W), (dbt, W)],
                        {"rows": rows, "d": d, "slices": ln_slices(rows)}))
            contribute(X, dX, pending)
            update(name)
        elif op == "gelu":
            dX = var(f"d:{X}@{name}", xs)
            fns.append(("gelu_bwd", [(X, R), (dY, R), (dX, W)], {"n": math.prod(xs)}))
            contribute(X, dX, pending)
        elif op == "concat":
            cs = [shapes[s][-1] for s in L["in"]]
            dXs = [var(f"d:{s}@{name}", shapes[s]) for s in L["in"]]
            fns.append(("concat_bwd", [(dY, R)] + [(d, W) for d in dXs],
                        {"rows": math.prod(xs[:-1]), "cs": cs}))
            for s, d in zip(L["in"], dXs):
                contribute(s, d, pending)
        elif op == "upsample":
            n, h, w, c = xs
            dX = var(f"d:{X}@{name}", xs)
            fns.append(("upsample_bwd", [(dY, R), (dX, W)], {"N": n, "H": h, "W": w, "C": c}))
            contribute(X, dX, pending)
        elif op == "attention":
            rows, d3 = xs
            Bt, T = spec["input"]
            H = L["heads"]
            dX = var(f"d:{X}@{name}", xs)
            Pb = var(name + ".Pb", (Bt, H, T, T))
            dS = var(name + ".dS", (Bt, H, T, T))
            fns.append(("attention_bwd", [(X, R), (Pb, W), (dY, R), (dX, W), (dS, W)],
                        {"B": Bt, "T": T, "H": H, "dh": d3 // 3 // H,
                         "causal": int(L["causal"])}))
            contribute(X, dX, pending)
        done.add(name)
        settle(pending)

    # ---------------- number variables by first appearance
    ids = {}
    for _, vs, _ in fns:
        for nm, _ in vs:
            if nm not in ids:
                ids[nm] = len(ids)
    vars_ = [None] * len(ids)
    for nm, i in ids.items():
        shape, dtype, kind = decl[nm]
        vars_[i] = {"name": nm, "shape": shape, "dtype": dtype, "kind": kind,
                    "bytes": math.prod(shape) * ITEMSIZE[dtype]}
    fns_ = [{"op": op, "vars": [(ids[nm], a) for nm, a in vs], "attrs": attrs}
            for op, vs, attrs in fns]
    return {"vars": vars_, "fns": fns_, "name": spec["name"]}


def as_schedule_input(reg):
    """(var_bytes, var_kinds, fn_vars) as the scheduler takes them."""
    return ([v["bytes"] for v in reg["vars"]], [v["kind"] for v in reg["vars"]],
            [f["vars"] for f in reg["fns"]])

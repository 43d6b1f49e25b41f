"""Lowering of a network description to the library's function sequence.

The paper executes a network as the topological sequence of its functions,
each with the set of variables it uses (Section 2; Section 3,
variable-sequence).  ``Net`` builds that sequence for one training step and
registers it through the C interface:

* forward functions in layer order, then the fused softmax cross-entropy
  (one label per row of the logits);
* per layer in reverse order: its backward functions, one SGD function for
  its parameters, then the sums of the gradient contributions of tensors
  consumed more than once, in the order the contributions appear: each
  contribution is accumulated in place into the tensor's running gradient
  (``acc``), or, while another tensor whose backward is still to come holds
  that same gradient variable, added into a new variable (``add``); an
  addition's own backward is the identity and needs no function.

Variables are numbered by first appearance.  Variable lists, sizes and
kinds follow the operation table of ``include/ooc.h``; the auxiliary sizes are
fixed per shape: a BatchNorm keeps 2 + 2 S floats per channel with S =
min(ceil(rows / 512), 2048) row slices; a weight gradient (convolution or
dense layer) is split over S_w slices of its reduction, S_w being the count
the library's kernels ask for (``ooc_wgrad_slices``), with a partial-sum
variable of S_w copies of dW (a dense layer's then S_w copies of db) when
S_w > 1; a LayerNorm keeps mean and 1/std per row and 2 S floats per feature
with S = min(ceil(rows / 32), 2048) (its rows are d floats wide); attention
writes its probabilities [B, H, T, T] in the forward, where they die, and its
backward recomputes them into a variable of its own beside a scratch of the
same size.
"""

from __future__ import annotations

from math import ceil, prod

from . import ooc

FLOAT = 4


def bn_row_slices(rows):
    return min(ceil(rows / 512), 2048)


def ln_row_slices(rows):
    return min(ceil(rows / 32), 2048)


class Net:
    """Function sequence of one training step of ``spec``."""

    def __init__(self, spec, keep_grads=False):
        self.spec = spec
        self.keep_grads = keep_grads
        self.meta = {}        # name -> (shape, dtype, kind)
        self.calls = []       # (op, [(name, access)], attrs)
        self.shape = {}
        self.params = {}      # layer name -> [param names]
        self.slices = {}      # layer name -> split-K slices of its weight gradient
        self._lower()
        self._number()

    # ------------------------------------------------------------ helpers
    def _decl(self, name, shape, dtype="f32", kind=ooc.TEMP):
        self.meta[name] = (tuple(int(s) for s in shape), dtype, kind)
        return name

    def _call(self, op, pairs, attrs):
        self.calls.append((op, pairs, [int(a) for a in attrs]))

    # ------------------------------------------------------------ forward
    def _fwd_linear(self, L, X):
        n, fin = self.shape[X]
        fout = L["out_features"]
        W = self._decl(L["name"] + ".W", (fout, fin), kind=ooc.PARAM)
        b = self._decl(L["name"] + ".b", (fout,), kind=ooc.PARAM)
        self.params[L["name"]] = [W, b]
        Y = self._decl(L["name"], (n, fout))
        self._call("linear_fwd", [(X, ooc.R), (W, ooc.R), (b, ooc.R), (Y, ooc.W)], [n, fin, fout])
        return (n, fout)

    def _conv_attrs(self, L, xs):
        n, h, w, c = xs
        k, st, pd = L["k"], L["stride"], L["pad"]
        p_, q_ = (h + 2 * pd - k) // st + 1, (w + 2 * pd - k) // st + 1
        return [n, h, w, c, L["cout"], k, k, st, pd, p_, q_]

    def _fwd_conv(self, L, X):
        a = self._conv_attrs(L, self.shape[X])
        n, _, _, c, K, R, S, _, _, P, Q = a
        W = self._decl(L["name"] + ".W", (K, R, S, c), kind=ooc.PARAM)
        self.params[L["name"]] = [W]
        Y = self._decl(L["name"], (n, P, Q, K))
        self._call("conv_fwd", [(X, ooc.R), (W, ooc.R), (Y, ooc.W)], a)
        return (n, P, Q, K)

    def _fwd_bn(self, L, X):
        xs = self.shape[X]
        c, rows = xs[-1], prod(xs[:-1])
        S = bn_row_slices(rows)
        g = self._decl(L["name"] + ".gamma", (c,), kind=ooc.PARAM)
        bt = self._decl(L["name"] + ".beta", (c,), kind=ooc.PARAM)
        self.params[L["name"]] = [g, bt]
        Y = self._decl(L["name"], xs)
        st = self._decl(L["name"] + ".stats", ((2 + 2 * S) * c,))
        self._call("bn_fwd", [(X, ooc.R), (g, ooc.R), (bt, ooc.R), (Y, ooc.W), (st, ooc.W)],
                   [rows, c, S])
        return xs

    def _fwd_concat(self, L, X):
        srcs = L["in"]
        lead = self.shape[srcs[0]][:-1]
        if any(self.shape[s][:-1] != lead for s in srcs) or len(set(srcs)) != len(srcs):
            raise ValueError(f"{L['name']}: concatenated tensors must differ and share all but "
                             "their last axis")
        cs = [self.shape[s][-1] for s in srcs]
        ys = lead + (sum(cs),)
        Y = self._decl(L["name"], ys)
        self._call("concat_fwd", [(s, ooc.R) for s in srcs] + [(Y, ooc.W)], [prod(lead)] + cs)
        return ys

    def _fwd_upsample(self, L, X):
        n, h, w, c = self.shape[X]
        ys = (n, 2 * h, 2 * w, c)
        Y = self._decl(L["name"], ys)
        self._call("upsample_fwd", [(X, ooc.R), (Y, ooc.W)], [n, h, w, c])
        return ys

    def _fwd_relu(self, L, X):
        xs = self.shape[X]
        Y = self._decl(L["name"], xs)
        self._call("relu_fwd", [(X, ooc.R), (Y, ooc.W)], [prod(xs)])
        return xs

    def _pool_attrs(self, L, xs):
        n, h, w, c = xs
        k, st, pd = L["k"], L["stride"], L["pad"]
        return [n, h, w, c, k, st, pd, (h + 2 * pd - k) // st + 1, (w + 2 * pd - k) // st + 1]

    def _fwd_maxpool(self, L, X):
        a = self._pool_attrs(L, self.shape[X])
        ys = (a[0], a[7], a[8], a[3])
        Y = self._decl(L["name"], ys)
        ix = self._decl(L["name"] + ".idx", ys, dtype="u8")
        self._call("maxpool_fwd", [(X, ooc.R), (Y, ooc.W), (ix, ooc.W)], a)
        return ys

    def _fwd_avgpool(self, L, X):
        n, h, w, c = self.shape[X]
        Y = self._decl(L["name"], (n, c))
        self._call("avgpool_fwd", [(X, ooc.R), (Y, ooc.W)], [n, h, w, c])
        return (n, c)

    def _fwd_add(self, L, X):
        B = L["in"][1]
        xs = self.shape[X]
        if self.shape[B] != xs:
            raise ValueError(f"add {L['name']}: shapes differ")
        Y = self._decl(L["name"], xs)
        self._call("add", [(X, ooc.R), (B, ooc.R), (Y, ooc.W)], [prod(xs)])
        return xs

    def _fwd_embed(self, L, X):
        B, T = self.shape[X]
        d = L["d"]
        E = self._decl(L["name"] + ".E", (L["vocab"], d), kind=ooc.PARAM)
        pos = self._decl(L["name"] + ".pos", (T, d), kind=ooc.PARAM)
        self.params[L["name"]] = [E, pos]
        Y = self._decl(L["name"], (B * T, d))
        self._call("embed_fwd", [(X, ooc.R), (E, ooc.R), (pos, ooc.R), (Y, ooc.W)],
                   [B, T, L["vocab"], d])
        return (B * T, d)

    def _fwd_layernorm(self, L, X):
        rows, d = self.shape[X]
        S = ln_row_slices(rows)
        g = self._decl(L["name"] + ".gamma", (d,), kind=ooc.PARAM)
        bt = self._decl(L["name"] + ".beta", (d,), kind=ooc.PARAM)
        self.params[L["name"]] = [g, bt]
        Y = self._decl(L["name"], (rows, d))
        st = self._decl(L["name"] + ".stats", (2 * rows + 2 * S * d,))
        self._call("layernorm_fwd", [(X, ooc.R), (g, ooc.R), (bt, ooc.R), (Y, ooc.W),
                                     (st, ooc.W)], [rows, d, S])
        return (rows, d)

    def _fwd_gelu(self, L, X):
        xs = self.shape[X]
        Y = self._decl(L["name"], xs)
        self._call("gelu_fwd", [(X, ooc.R), (Y, ooc.W)], [prod(xs)])
        return xs

    def _attn_attrs(self, L, X):
        rows, d3 = self.shape[X]
        B, T = self.spec["input"]
        H = L["heads"]
        return [B, T, H, d3 // 3 // H, 1 if L["causal"] else 0]

    def _fwd_attention(self, L, X):
        a = self._attn_attrs(L, X)
        B, T, H, dh, _ = a
        Pr = self._decl(L["name"] + ".P", (B, H, T, T))
        Y = self._decl(L["name"], (B * T, H * dh))
        self._call("attention_fwd", [(X, ooc.R), (Pr, ooc.W), (Y, ooc.W)], a)
        return (B * T, H * dh)

    # ------------------------------------------------------------ backward
    def _grad_of_param(self, p):
        return self._decl("d:" + p, self.meta[p][0],
                          kind=ooc.OUTPUT if self.keep_grads else ooc.TEMP)

    def _sgd(self, layer):
        mom = self.spec["optimizer"]["momentum"]
        pairs = []
        for p in self.params[layer]:
            pairs += [(p, ooc.RW), ("d:" + p, ooc.R)]
            if mom:
                pairs.append((self._decl("m:" + p, self.meta[p][0], kind=ooc.STATE), ooc.RW))
        self._call("sgd", pairs, [len(self.params[layer]), 1 if mom else 0])

    def _bwd(self, L, dY, out):
        """Emits L's backward functions; appends (tensor, gradient) contributions to out."""
        name, X = L["name"], L["in"][0]
        xs = self.shape[X]
        op = L["op"]
        if op == "linear":
            W, b = self.params[name]
            n, fin = xs
            fout = L["out_features"]
            attrs = [n, fin, fout]
            sw = ooc.wgrad_slices("linear_bwd_w", attrs)
            self.slices[name] = sw
            pairs = [(X, ooc.R), (dY, ooc.R), (self._grad_of_param(W), ooc.W),
                     (self._grad_of_param(b), ooc.W)]
            if sw > 1:
                pairs.append((self._decl(name + ".part", (sw * (fout * fin + fout),)), ooc.W))
            self._call("linear_bwd_w", pairs, attrs + [sw])
            if X != "x":
                dX = self._decl(f"d:{X}@{name}", xs)
                self._call("linear_bwd_x", [(W, ooc.R), (dY, ooc.R), (dX, ooc.W)], attrs)
                out.append((X, dX))
            self._sgd(name)
        elif op == "conv":
            (W,) = self.params[name]
            a = self._conv_attrs(L, xs)
            n, _, _, c, K, R, S, _, _, P, Q = a
            sw = ooc.wgrad_slices("conv_bwd_w", a)
            self.slices[name] = sw
            pairs = [(X, ooc.R), (dY, ooc.R), (self._grad_of_param(W), ooc.W)]
            if sw > 1:
                pairs.append((self._decl(name + ".part", (sw * K * R * S * c,)), ooc.W))
            self._call("conv_bwd_w", pairs, a + [sw])
            if X != "x":
                dX = self._decl(f"d:{X}@{name}", xs)
                self._call("conv_bwd_x", [(W, ooc.R), (dY, ooc.R), (dX, ooc.W)], a)
                out.append((X, dX))
            self._sgd(name)
        elif op == "bn":
            g, bt = self.params[name]
            rows, c = prod(xs[:-1]), xs[-1]
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("bn_bwd", [(X, ooc.R), (g, ooc.R), (name + ".stats", ooc.RW), (dY, ooc.R),
                                  (dX, ooc.W), (self._grad_of_param(g), ooc.W),
                                  (self._grad_of_param(bt), ooc.W)],
                       [rows, c, bn_row_slices(rows)])
            out.append((X, dX))
            self._sgd(name)
        elif op == "relu":
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("relu_bwd", [(name, ooc.R), (dY, ooc.R), (dX, ooc.W)], [prod(xs)])
            out.append((X, dX))
        elif op == "maxpool":
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("maxpool_bwd", [(name + ".idx", ooc.R), (dY, ooc.R), (dX, ooc.W)],
                       self._pool_attrs(L, xs))
            out.append((X, dX))
        elif op == "avgpool":
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("avgpool_bwd", [(dY, ooc.R), (dX, ooc.W)], list(xs))
            out.append((X, dX))
        elif op == "add":
            for src in L["in"]:
                out.append((src, dY))
        elif op == "embed":
            E, pos = self.params[name]
            B, T = xs
            self._call("embed_bwd", [(X, ooc.R), (dY, ooc.R), (self._grad_of_param(E), ooc.W),
                                     (self._grad_of_param(pos), ooc.W)],
                       [B, T, L["vocab"], L["d"]])
            self._sgd(name)
        elif op == "layernorm":
            g, bt = self.params[name]
            rows, d = xs
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("layernorm_bwd", [(X, ooc.R), (g, ooc.R), (name + ".stats", ooc.RW),
                                         (dY, ooc.R), (dX, ooc.W),
                                         (self._grad_of_param(g), ooc.W),
                                         (self._grad_of_param(bt), ooc.W)],
                       [rows, d, ln_row_slices(rows)])
            out.append((X, dX))
            self._sgd(name)
        elif op == "gelu":
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("gelu_bwd", [(X, ooc.R), (dY, ooc.R), (dX, ooc.W)], [prod(xs)])
            out.append((X, dX))
        elif op == "concat":
            srcs = L["in"]
            cs = [self.shape[s][-1] for s in srcs]
            dXs = [self._decl(f"d:{s}@{name}", self.shape[s]) for s in srcs]
            self._call("concat_bwd", [(dY, ooc.R)] + [(d, ooc.W) for d in dXs],
                       [prod(self.shape[name][:-1])] + cs)
            out.extend(zip(srcs, dXs))
        elif op == "upsample":
            n, h, w, c = xs
            dX = self._decl(f"d:{X}@{name}", xs)
            self._call("upsample_bwd", [(dY, ooc.R), (dX, ooc.W)], [n, h, w, c])
            out.append((X, dX))
        elif op == "attention":
            a = self._attn_attrs(L, X)
            B, T, H, dh, _ = a
            dX = self._decl(f"d:{X}@{name}", xs)
            Pb = self._decl(name + ".Pb", (B, H, T, T))
            dS = self._decl(name + ".dS", (B, H, T, T))
            self._call("attention_bwd", [(X, ooc.R), (Pb, ooc.W), (dY, ooc.R),
                                         (dX, ooc.W), (dS, ooc.W)], a)
            out.append((X, dX))

    # ------------------------------------------------------------ whole step
    def _lower(self):
        spec = self.spec
        self.shape["x"] = tuple(spec["input"])
        self._decl("x", spec["input"], dtype="i32" if spec.get("tokens") else "f32",
                   kind=ooc.INPUT)
        fwd = {"linear": self._fwd_linear, "conv": self._fwd_conv, "bn": self._fwd_bn,
               "relu": self._fwd_relu, "maxpool": self._fwd_maxpool,
               "avgpool": self._fwd_avgpool, "add": self._fwd_add, "embed": self._fwd_embed,
               "layernorm": self._fwd_layernorm, "gelu": self._fwd_gelu,
               "attention": self._fwd_attention, "concat": self._fwd_concat,
               "upsample": self._fwd_upsample}
        for L in spec["layers"]:
            self.shape[L["name"]] = fwd[L["op"]](L, L["in"][0])
        logits = spec["logits"]
        ls = self.shape[logits]
        n, classes = prod(ls[:-1]), ls[-1]          # one row (and label) per position
        self._decl("labels", (n,), dtype="i32", kind=ooc.INPUT)
        self._decl("loss", (n + 1,), kind=ooc.OUTPUT)
        dlogits = self._decl("d:" + logits, ls)
        self._call("softmax_ce", [(logits, ooc.R), ("labels", ooc.R), ("loss", ooc.W),
                                  (dlogits, ooc.W)], [n, classes])
        grads = {logits: dlogits}
        sums = {}
        visited = set()      # layers whose backward has been emitted
        for L in reversed(spec["layers"]):
            if L["name"] not in grads:
                continue
            contributions = []
            self._bwd(L, grads[L["name"]], contributions)
            visited.add(L["name"])
            for tensor, g in contributions:
                if tensor == "x":
                    continue
                if tensor not in grads:
                    grads[tensor] = g
                    continue
                cur = grads[tensor]
                # the running sum is accumulated in place unless another tensor whose
                # backward is still to come holds the same gradient variable (an addition's
                # backward hands its output gradient to both inputs)
                shared = any(u != tensor and gv == cur and u not in visited
                             for u, gv in grads.items())
                n = prod(self.shape[tensor])
                if not shared and cur != g:
                    self._call("acc", [(cur, ooc.RW), (g, ooc.R)], [n])
                    continue
                sums[tensor] = sums.get(tensor, 1) + 1
                acc = self._decl(f"d:{tensor}#{sums[tensor]}", self.shape[tensor])
                self._call("add", [(cur, ooc.R), (g, ooc.R), (acc, ooc.W)], [n])
                grads[tensor] = acc

    def _number(self):
        self.ids = {}
        for _, pairs, _ in self.calls:
            for nm, _ in pairs:
                self.ids.setdefault(nm, len(self.ids))
        self.names = sorted(self.ids, key=self.ids.get)
        itemsize = {"f32": 4, "i32": 4, "u8": 1}
        self.var_bytes = [prod(self.meta[n][0]) * itemsize[self.meta[n][1]] for n in self.names]
        self.var_kinds = [self.meta[n][2] for n in self.names]
        self.fn_vars = [[(self.ids[nm], a) for nm, a in pairs] for _, pairs, _ in self.calls]
        self.fn_ops = [op for op, _, _ in self.calls]
        self.fn_attrs = [attrs for _, _, attrs in self.calls]

    # ------------------------------------------------------------ C interface
    def register(self, ctx):
        """Adds every variable and function to ``ctx`` (an ``ooc.Context``)."""
        for nb, kd in zip(self.var_bytes, self.var_kinds):
            ctx.add_var(nb, kd)
        for op, vs, attrs in zip(self.fn_ops, self.fn_vars, self.fn_attrs):
            ctx.add_fn(op, [v for v, _ in vs], [a for _, a in vs], attrs)
        return self

    def var(self, name):
        return self.ids[name]

    def view(self, ctx, name):
        """Host slot of a persistent variable as an array of its shape."""
        shape, dtype, _ = self.meta[name]
        return ctx.host_view(self.ids[name], dtype, shape)

    def param_names(self):
        return [n for n in self.names if self.meta[n][2] == ooc.PARAM]

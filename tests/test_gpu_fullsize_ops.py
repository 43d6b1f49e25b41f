"""Every distinct function of the full-size workloads, alone, against the float64 oracle (GPU).

The out-of-core steps at the benchmark sizes are compared bit for bit with the in-core step
of the same kernels (``test_gpu_step``).  A defect that only shows at full size (a 32-bit
offset past 2^31 bytes, BatchNorm with more rows per slice once the slice count is capped,
a grid dimension at its limit) would be the same in both runs, so here each distinct
(operation, attributes) launch of ResNet-50 at batch 256 and 1440 and of the 48-layer
transformer at batch 64 runs once, in-core, at its full shape, on seeded inputs, and its
results are compared element by element with ``oracle.sampled`` / ``oracle.ops``:

* reductions (convolutions, dense layers, sums over rows): at least 4096 sampled outputs
  (all of them when there are fewer), each within sqrt(T) u mag + 4 u |ref|, where T is the
  number of terms of its sum, mag the sum of their absolute values and u = 2^-24;
* every BatchNorm / LayerNorm statistic (mean and 1/std per channel or row, and the
  dgamma / dbeta sums), within the same kind of bound;
* elementwise and data-movement results (ReLU, addition, embedding rows, max-pool values and
  indices): every element, exactly;
* transcendental results (softmax cross-entropy, GELU, attention): every element of the
  sampled heads or of the whole tensor, within a bound built the same way from the
  magnitudes of the formula's terms.

Inputs are windows of one seeded standard-normal pool (``synth.normal_pool``); indices
(labels, token ids, max-pool taps) are drawn valid.  The worst ratio error / bound of each
case is printed.
"""

from __future__ import annotations

import contextlib
import math
import zlib

import numpy as np
import pytest

from scipy.special import erfc

from oracle import ops, sampled
from paper_2010_14109_amd import netdef, ooc, synth

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
NSAMPLE = 4096
SCRATCH = {("conv_bwd_w", 3), ("linear_bwd_w", 4), ("attention_bwd", 4)}   # (op, var position)
WORKLOADS = (("resnet50_b256", {}), ("resnet50_b1440", {}), ("transformer", {}))


def distinct_functions():
    """[(id, op, attrs, [(bytes, access)])] over the workloads, first occurrence of each."""
    seen, out = set(), []
    for name, kw in WORKLOADS:
        net = netdef.Net(synth.workload(name, **kw))
        for op, vs, attrs in zip(net.fn_ops, net.fn_vars, net.fn_attrs):
            sig = [(net.var_bytes[v], a) for v, a in vs]
            key = (op, tuple(attrs), tuple(sig))
            if key in seen:
                continue
            seen.add(key)
            out.append((f"{name}-{op}-{'x'.join(map(str, attrs))}", op, list(attrs), sig))
    return out


CASES = distinct_functions()


# ---------------------------------------------------------------- inputs
class Pool:
    """One seeded normal pool of twice the largest tensor of the cases; input j of a case
    with k inputs is the window starting at j / (k - 1) of the free span, so a case's inputs
    overlap as little as the pool allows.  The pool's size is fixed by the case list, so every
    case sees the same values however the tests are selected or ordered."""
    data = None
    SIZE = 2 * max(b for _, _, _, sig in CASES for b, _ in sig) // 4

    @classmethod
    def window(cls, n, slot, slots):
        if cls.data is None:
            cls.data = synth.normal_pool(cls.SIZE, seed=2024)
        span = cls.data.size - n
        off = 0 if slots <= 1 else span * slot // (slots - 1)
        return cls.data[off:off + n]


@contextlib.contextmanager
def run_case(op, attrs, sig, fill):
    """Registers the function alone (reads: INPUT or PARAM, writes: OUTPUT, scratch: TEMP),
    fills the host slots with ``fill(position, view)``, runs it once in-core and yields the
    host views of every variable (None for scratch), valid inside the ``with`` block."""
    ctx = ooc.Context(0)
    try:
        ids, kinds = [], []
        for j, (nb, acc) in enumerate(sig):
            kind = (ooc.TEMP if (op, j) in SCRATCH else ooc.OUTPUT if acc == ooc.W
                    else ooc.INPUT if acc == ooc.R else ooc.PARAM)
            ids.append(ctx.add_var(nb, kind))
            kinds.append(kind)
        ctx.add_fn(op, ids, [a for _, a in sig], attrs)
        ctx.set_chunk(2 << 20)
        ctx.build_schedule()
        ctx.prepare()
        views = [None if k == ooc.TEMP else ctx.host_view(v, np.uint8) for v, k in zip(ids, kinds)]
        for j, (v, k) in enumerate(zip(views, kinds)):
            if k in (ooc.INPUT, ooc.PARAM):
                fill(j, v)
        ctx.upload()
        ctx.step(0.01, 0.9)
        ctx.download()
        yield views
    finally:
        ctx.close()


def as_f32(b):
    return b.view(np.float32)


class Report:
    def __init__(self, case):
        self.case, self.worst = case, 0.0

    def close(self, name, got, ref, bound, offset=0):
        ref = np.asarray(ref, np.float64)
        bound = np.broadcast_to(np.asarray(bound, np.float64), ref.shape).reshape(-1)
        got = np.asarray(got, np.float64).reshape(-1)
        ref = ref.reshape(-1)
        assert got.shape == ref.shape, (name, got.shape, ref.shape)
        assert np.all(np.isfinite(got)), name
        err = np.abs(got - ref)
        ratio = err / np.maximum(bound, 1e-300)
        worst = int(np.argmax(ratio))
        assert ratio[worst] <= 1.0, (f"{self.case} {name}: element {offset + worst} got {got[worst]!r} "
                                     f"ref {ref[worst]!r} bound {bound[worst]!r}")
        self.worst = max(self.worst, float(ratio[worst]))

    def exact(self, name, got, ref, offset=0):
        """Equal values (a zero's sign is not compared); offset = index of got[0] in the whole
        result, for the message."""
        got, ref = np.asarray(got).reshape(-1), np.asarray(ref).reshape(-1)
        assert got.shape == ref.shape, (name, got.shape, ref.shape)
        bad = np.flatnonzero(got != ref)
        assert bad.size == 0, (f"{self.case} {name}: {bad.size} elements differ, first "
                               f"{offset + bad[0]}")


# Whole-tensor comparisons run over pieces of this many elements: each piece's reference and
# comparison stay small, so a tensor of 2^30 elements does not need several more of its size.
PIECE = 1 << 24


def pieces(n):
    return ((lo, min(n, lo + PIECE)) for lo in range(0, n, PIECE))


def sample(shape, rng, n=NSAMPLE):
    """n random coordinates of an array of ``shape`` (every one when it has fewer), plus the
    first and last element."""
    total = math.prod(shape)
    if total <= n:
        flat = np.arange(total)
    else:
        flat = np.unique(np.concatenate([rng.integers(0, total, n), [0, total - 1]]))
    return np.unravel_index(flat, shape)


def reduction_bound(mag, terms, ref):
    return math.sqrt(terms) * U * mag + 4 * U * np.abs(ref)


# ---------------------------------------------------------------- per-op checks
def check_conv(op, a, sig, rep, rng):
    N, H, W, C, K, R, S, st, pd, P, Q = a[:11]
    xs, ws, ys = (N, H, W, C), (K, R, S, C), (N, P, Q, K)
    shapes = {"conv_fwd": [xs, ws, ys], "conv_bwd_x": [ws, ys, xs], "conv_bwd_w": [xs, ys, ws]}[op]
    inputs = {}

    def fill(j, v):
        inputs[j] = Pool.window(v.size // 4, j, 2).reshape(shapes[j])
        as_f32(v)[...] = inputs[j].reshape(-1)

    with run_case(op, a, sig, fill) as out:
        got = as_f32(out[2]).reshape(shapes[2])
        if op == "conv_fwd":
            idx = sample(ys, rng)
            val, mag, T = sampled.conv_fwd_at(inputs[0], inputs[1], st, pd, *idx)
            rep.close("Y", got[idx], val, reduction_bound(mag, T, val))
        elif op == "conv_bwd_x":
            idx = sample(xs, rng)
            val, mag, T = sampled.conv_bwd_x_at(inputs[0], inputs[1], st, pd, *idx)
            rep.close("dX", got[idx], val, reduction_bound(mag, T, val))
        else:
            # a block of dW: nk output channels x nc input channels x nt taps >= 4096 entries
            taps = [(r, s) for r in range(R) for s in range(S)]
            nk = min(K, 64)
            nc = min(C, 64, -(-NSAMPLE // (nk * len(taps))))
            nt = min(len(taps), -(-NSAMPLE // (nk * nc)))
            ks = np.sort(rng.choice(K, nk, replace=False))
            cs = np.sort(rng.choice(C, nc, replace=False))
            pick = [taps[i] for i in np.sort(rng.choice(len(taps), nt, replace=False))]
            sub = np.stack([got[ks][:, r, s, :][:, cs] for r, s in pick])
            val, mag, T = sampled.conv_bwd_w_at(inputs[0], inputs[1], st, pd, R, S, ks, cs, pick)
            rep.close("dW", sub, val, reduction_bound(mag, T, val))


def check_linear(op, a, sig, rep, rng):
    M, K, N = a[:3]
    shapes = {"linear_fwd": [(M, K), (N, K), (N,), (M, N)],
              "linear_bwd_x": [(N, K), (M, N), (M, K)],
              "linear_bwd_w": [(M, K), (M, N), (N, K), (N,)]}[op]
    inputs = {}

    def fill(j, v):
        inputs[j] = Pool.window(v.size // 4, j, 3).reshape(shapes[j])
        as_f32(v)[...] = inputs[j].reshape(-1)

    with run_case(op, a, sig, fill) as out:
        if op == "linear_fwd":
            got = as_f32(out[3]).reshape(M, N)
            idx = sample((M, N), rng)
            val, mag, T = sampled.linear_fwd_at(inputs[0], inputs[1], inputs[2], *idx)
            rep.close("Y", got[idx], val, reduction_bound(mag, T, val))
        elif op == "linear_bwd_x":
            got = as_f32(out[2]).reshape(M, K)
            idx = sample((M, K), rng)
            val, mag, T = sampled.linear_bwd_x_at(inputs[0], inputs[1], *idx)
            rep.close("dX", got[idx], val, reduction_bound(mag, T, val))
        else:
            dW, db = as_f32(out[2]).reshape(N, K), as_f32(out[3])
            js = np.sort(rng.choice(N, min(N, 64), replace=False))
            cols = np.sort(rng.choice(K, min(K, 64), replace=False))
            (w, wm), (b, bm), T = sampled.linear_bwd_w_at(inputs[0], inputs[1], js, cols)
            rep.close("dW", dW[js][:, cols], w, reduction_bound(wm, T, w))
            rep.close("db", db[js], b, reduction_bound(bm, T, b))


def check_bn(op, a, sig, rep, rng):
    """The statistics' bounds follow the kernels' summation: each slice's rows go to 16 float32
    chains (ceil(rows / 16 S) terms each, of x - x[0] and its square, or of dY and dY xhat) and
    chains and slices are combined in float64, so a sum carries the error of a float32 sum of
    ceil(rows / 16 S) terms (4 sqrt(that) u of its magnitude, the bound of a one-signed running
    sum with room to spare).  The variance is E[d^2] - E[d]^2 with d = x - x[0], which divides
    the error of E[d^2] by var / E[d^2].  Elementwise results carry the error of the statistics
    they use plus their own rounding."""
    rows, C, S = a
    chain = 4 * math.sqrt(-(-rows // (16 * S))) * U
    idx = sample((rows, C), rng)
    c = idx[1]
    gamma = (1.0 + 0.25 * Pool.window(C, 1, 7)).astype(np.float32)
    X = Pool.window(rows * C, 0, 7).reshape(rows, C)
    if op == "bn_fwd":
        beta = Pool.window(C, 2, 7).copy()

        def fill(j, v):
            as_f32(v)[...] = (X.reshape(-1), gamma, beta)[j]

        with run_case(op, a, sig, fill) as out:
            mean, invstd, absmean = sampled.bn_stats(X)
            shift = X[0].astype(np.float64)
            ed2 = 1.0 / invstd ** 2 + (mean - shift) ** 2        # E[d^2], d = x - x[0] (+ eps)
            dmean = chain * (absmean + np.abs(shift)) + 4 * U * np.abs(mean)
            drel = 0.5 * chain * ed2 * invstd ** 2 + 8 * U    # relative error of invstd
            st = as_f32(out[4])
            rep.close("mean", st[:C], mean, dmean)
            rep.close("invstd", st[C:2 * C], invstd, drel * invstd)
            ref = sampled.bn_fwd_at(X, gamma, beta, mean, invstd, *idx)
            xh = np.abs((X[idx].astype(np.float64) - mean[c]) * invstd[c])
            bound = np.abs(gamma[c]) * (xh * drel[c] + dmean[c] * invstd[c]) \
                + 8 * U * (np.abs(gamma[c]) * xh + np.abs(beta[c]))
            rep.close("Y", as_f32(out[3]).reshape(rows, C)[idx], ref, bound)
        return
    # bn_bwd: stats hold mean and invstd as the forward leaves them (here the oracle's, rounded
    # to float32); the rest of stats is the kernels' scratch
    G = Pool.window(rows * C, 6, 7).reshape(rows, C)
    m64, r64, _ = sampled.bn_stats(X)
    mean32, inv32 = m64.astype(np.float32), r64.astype(np.float32)

    def fill(j, v):
        f = as_f32(v)
        if j == 2:
            f[...] = 0
            f[:C], f[C:2 * C] = mean32, inv32
        else:
            f[...] = {0: X.reshape(-1), 1: gamma, 3: G.reshape(-1)}[j]

    with run_case(op, a, sig, fill) as out:
        mean, invstd = mean32.astype(np.float64), inv32.astype(np.float64)
        db, dg, dbm, dgm = sampled.bn_bwd_sums(X, G, mean, invstd)
        ddb = chain * dbm + 4 * U * np.abs(db)
        ddg = (chain + 8 * U) * dgm + 4 * U * np.abs(dg)
        rep.close("dbeta", as_f32(out[6]), db, ddb)
        rep.close("dgamma", as_f32(out[5]), dg, ddg)
        ref = sampled.bn_bwd_at(X, G, gamma, mean, invstd, db, dg, *idx)
        xh = np.abs((X[idx].astype(np.float64) - mean[c]) * invstd[c])
        scale = np.abs(gamma[c]) * invstd[c]
        bound = scale * ((ddb[c] + xh * ddg[c]) / rows
                         + 8 * U * (np.abs(G[idx]) + (np.abs(db[c]) + xh * np.abs(dg[c])) / rows))
        rep.close("dX", as_f32(out[4]).reshape(rows, C)[idx], ref, bound)


def check_elementwise(op, a, sig, rep, rng):
    n = a[0]
    ins = [Pool.window(n, j, 2) for j in range(2)]

    def fill(j, v):
        as_f32(v)[...] = ins[j]

    with run_case(op, a, sig, fill) as out:
        got = as_f32(out[0] if op == "acc" else out[-1])     # acc: in place, A += B
        for lo, hi in pieces(n):
            x, y = ins[0][lo:hi], ins[1][lo:hi]
            if op == "relu_fwd":
                ref = np.maximum(x, np.float32(0))
            elif op == "relu_bwd":
                ref = np.where(x > 0, y, np.float32(0))
            else:
                ref = x + y                         # one float32 addition, correctly rounded
            rep.exact({"relu_bwd": "dX", "acc": "A"}.get(op, "Y"), got[lo:hi], ref, lo)


def pool_taps(N, P, Q, C, k, st, pd, H, W, rng):
    """Valid max-pool indices r k + s: for every output, a uniformly drawn tap inside the image."""
    def axis(n_out, n_in):
        o = np.arange(n_out)
        return np.maximum(0, pd - o * st), np.minimum(k - 1, n_in - 1 + pd - o * st)

    (rlo, rhi), (slo, shi) = axis(P, H), axis(Q, W)
    r = rlo[None, :, None, None] + np.floor(rng.random((N, P, Q, C), dtype=np.float32)
                                            * (rhi - rlo + 1)[None, :, None, None]).astype(np.int64)
    s = slo[None, None, :, None] + np.floor(rng.random((N, P, Q, C), dtype=np.float32)
                                            * (shi - slo + 1)[None, None, :, None]).astype(np.int64)
    return (np.minimum(r, rhi[None, :, None, None]) * k
            + np.minimum(s, shi[None, None, :, None])).astype(np.uint8)


def check_pool(op, a, sig, rep, rng):
    if op.startswith("avgpool"):
        N, H, W, C = a
        shp = (N, H, W, C) if op == "avgpool_fwd" else (N, C)
        X = Pool.window(math.prod(shp), 0, 1).reshape(shp)

        def fill(j, v):
            as_f32(v)[...] = X.reshape(-1)

        with run_case(op, a, sig, fill) as out:
            x = X.astype(np.float64)
            if op == "avgpool_fwd":
                ref = ops.avgpool_fwd(x)
                rep.close("Y", as_f32(out[1]), ref,
                          reduction_bound(np.abs(x).mean(axis=(1, 2)), H * W, ref))
            else:
                ref = ops.avgpool_bwd(x, (N, H, W, C))
                rep.close("dX", as_f32(out[1]), ref, 4 * U * np.abs(ref))
        return
    N, H, W, C, k, st, pd, P, Q = a
    if op == "maxpool_fwd":
        X = Pool.window(N * H * W * C, 0, 1).reshape(N, H, W, C)

        def fill(j, v):
            as_f32(v)[...] = X.reshape(-1)

        with run_case(op, a, sig, fill) as out:
            idx = sample((N, P, Q, C), rng)
            val, tap = sampled.maxpool_fwd_at(X, k, st, pd, *idx)
            rep.exact("Y", as_f32(out[1]).reshape(N, P, Q, C)[idx], val.astype(np.float32))
            rep.exact("idx", out[2].reshape(N, P, Q, C)[idx], tap.astype(np.uint8))
        return
    taps = pool_taps(N, P, Q, C, k, st, pd, H, W, rng)
    G = Pool.window(N * P * Q * C, 1, 2).reshape(N, P, Q, C)

    def fill(j, v):
        if j == 0:
            v[...] = taps.reshape(-1)
        else:
            as_f32(v)[...] = G.reshape(-1)

    with run_case(op, a, sig, fill) as out:
        idx = sample((N, H, W, C), rng)
        val, T = sampled.maxpool_bwd_at(taps, G, k, st, pd, *idx)
        mag, _ = sampled.maxpool_bwd_at(taps, np.abs(G), k, st, pd, *idx)
        rep.close("dX", as_f32(out[2]).reshape(N, H, W, C)[idx], val, T * U * mag)


def check_softmax(op, a, sig, rep, rng):
    """exp of z - max - lse in float32: its argument carries u (|z| + |max| + |lse|) of error,
    the sum of the exponentials sqrt(classes) u of its own, expf a few ulp."""
    N, classes = a
    logits = (3 * Pool.window(N * classes, 0, 1)).reshape(N, classes)
    labels = rng.integers(0, classes, N).astype(np.int32)

    def fill(j, v):
        if j == 0:
            as_f32(v)[...] = logits.reshape(-1)
        else:
            v.view(np.int32)[...] = labels

    with run_case(op, a, sig, fill) as out:
        z = logits.astype(np.float64)
        rows, mean, d = ops.softmax_ce(z, labels)
        zmax = z.max(axis=1)
        lse = np.log(np.exp(z - zmax[:, None]).sum(axis=1)) + zmax
        p = np.exp(z - lse[:, None])
        rel = (math.sqrt(classes) + 16 + 2 * np.abs(z).max(axis=1) + np.abs(lse))[:, None] * U
        rep.close("dlogits", as_f32(out[3]).reshape(N, classes), d,
                  rel * p / N + 4 * U * np.abs(d))
        zl = z[np.arange(N), labels]
        rb = rel[:, 0] * (np.abs(lse) + np.abs(zl) + 1)
        loss = as_f32(out[2])
        rep.close("row losses", loss[:N], rows, rb)
        rep.close("mean loss", loss[N:], [mean],
                  [rb.max() + math.sqrt(N) * U * np.abs(rows).mean() + 4 * U * abs(mean)])


def check_sgd(op, a, sig, rep, rng):
    count, mom = a
    step = 3 if mom else 2
    ins = {}

    def fill(j, v):
        ins[j] = Pool.window(v.size // 4, j, 3 * count)
        as_f32(v)[...] = ins[j]

    with run_case(op, a, sig, fill) as out:
        lr, mu = float(np.float32(0.01)), float(np.float32(0.9))
        for t in range(count):
            p, g = ins[step * t].astype(np.float64), ins[step * t + 1].astype(np.float64)
            if mom:
                v = ins[step * t + 2].astype(np.float64)
                ref_w, ref_v = ops.sgd_momentum(p, g, v, lr, mu)
                vm = mu * np.abs(v) + np.abs(g)
                rep.close(f"v{t}", as_f32(out[step * t + 2]), ref_v, 4 * U * vm)
                rep.close(f"w{t}", as_f32(out[step * t]), ref_w, 4 * U * (np.abs(p) + lr * vm))
            else:
                rep.close(f"w{t}", as_f32(out[step * t]), ops.sgd(p, g, lr),
                          4 * U * (np.abs(p) + lr * np.abs(g)))


def check_embed(op, a, sig, rep, rng):
    B, T, V, d = a
    ids = rng.integers(0, V, (B, T)).astype(np.int32)
    if op == "embed_fwd":
        E = Pool.window(V * d, 1, 3).reshape(V, d)
        pos = Pool.window(T * d, 2, 3).reshape(T, d)

        def fill(j, v):
            if j == 0:
                v.view(np.int32)[...] = ids.reshape(-1)
            else:
                as_f32(v)[...] = (E if j == 1 else pos).reshape(-1)

        with run_case(op, a, sig, fill) as out:
            rep.exact("Y", as_f32(out[3]), (E[ids] + pos[None]).reshape(-1))
        return
    G = Pool.window(B * T * d, 1, 2).reshape(B * T, d)

    def fill(j, v):
        if j == 0:
            v.view(np.int32)[...] = ids.reshape(-1)
        else:
            as_f32(v)[...] = G.reshape(-1)

    with run_case(op, a, sig, fill) as out:
        dE, dpos = ops.embed_bwd(ids, G.astype(np.float64), V)
        mE, mpos = ops.embed_bwd(ids, np.abs(G).astype(np.float64), V)
        cnt = np.bincount(ids.reshape(-1), minlength=V)[:, None]
        rep.close("dE", as_f32(out[2]).reshape(V, d), dE,
                  np.sqrt(np.maximum(cnt, 1)) * U * mE + 4 * U * np.abs(dE))
        rep.close("dpos", as_f32(out[3]).reshape(T, d), dpos, reduction_bound(mpos, B, dpos))


def check_layernorm(op, a, sig, rep, rng):
    """Row statistics are sums of d terms (sqrt(d) u of their magnitude), the dgamma / dbeta
    sums run over the rows (sqrt(rows) u); elementwise results carry the statistics' error
    plus their own rounding, as for BatchNorm."""
    rows, d, S = a
    X = Pool.window(rows * d, 0, 7).reshape(rows, d)
    gamma = (1.0 + 0.25 * Pool.window(d, 1, 7)).astype(np.float32)
    beta = Pool.window(d, 2, 7).copy()
    x64 = X.astype(np.float64)
    mean = x64.mean(axis=1)
    rstd = 1.0 / np.sqrt(((x64 - mean[:, None]) ** 2).mean(axis=1) + ops.LN_EPS)
    absmean = np.abs(x64).mean(axis=1)
    root = math.sqrt(d) * U
    if op == "layernorm_fwd":
        def fill(j, v):
            as_f32(v)[...] = (X.reshape(-1), gamma, beta)[j]

        with run_case(op, a, sig, fill) as out:
            st = as_f32(out[4])
            dmean = root * absmean + 4 * U * np.abs(mean)
            drel = root * (1 + (mean * rstd) ** 2) + 8 * U
            rep.close("mean", st[:rows], mean, dmean)
            rep.close("rstd", st[rows:2 * rows], rstd, drel * rstd)
            Y, _, _ = ops.layernorm_fwd(x64, gamma.astype(np.float64), beta.astype(np.float64))
            xh = np.abs((x64 - mean[:, None]) * rstd[:, None])
            bound = np.abs(gamma) * (xh * drel[:, None] + (dmean * rstd)[:, None]) \
                + 8 * U * (np.abs(gamma) * xh + np.abs(beta))
            rep.close("Y", as_f32(out[3]).reshape(rows, d), Y, bound)
        return
    G = Pool.window(rows * d, 6, 7).reshape(rows, d)
    m32, r32 = mean.astype(np.float32), rstd.astype(np.float32)

    def fill(j, v):
        f = as_f32(v)
        if j == 2:
            f[...] = 0
            f[:rows], f[rows:2 * rows] = m32, r32
        else:
            f[...] = {0: X.reshape(-1), 1: gamma, 3: G.reshape(-1)}[j]

    with run_case(op, a, sig, fill) as out:
        m64, rs64 = m32.astype(np.float64), r32.astype(np.float64)
        g64 = G.astype(np.float64)
        dX, dg, db = ops.layernorm_bwd(x64, gamma.astype(np.float64), m64, rs64, g64)
        xh = (x64 - m64[:, None]) * rs64[:, None]
        rr = math.sqrt(rows) * U
        rep.close("dbeta", as_f32(out[6]), db, rr * np.abs(g64).sum(axis=0) + 4 * U * np.abs(db))
        rep.close("dgamma", as_f32(out[5]), dg,
                  (rr + 8 * U) * np.abs(g64 * xh).sum(axis=0) + 4 * U * np.abs(dg))
        gg = np.abs(g64 * gamma)
        mag = rs64[:, None] * (gg + gg.mean(axis=1, keepdims=True)
                               + np.abs(xh) * (gg * np.abs(xh)).mean(axis=1, keepdims=True))
        rep.close("dX", as_f32(out[4]).reshape(rows, d), dX, (root + 16 * U) * mag)


def check_gelu(op, a, sig, rep, rng):
    """x Phi(x) with Phi = erfc(-x / sqrt 2) / 2: rounding -x / sqrt 2 moves Phi by up to
    |x| phi(x) u, erfcf and expf err by a few ulp, and the backward's exp(-x^2 / 2) carries
    x^2 u of error from its argument; bounds are 8 u times the magnitudes of those terms."""
    n = a[0]
    X = (2 * Pool.window(n, 0, 2)).astype(np.float32)
    G = Pool.window(n, 1, 2)

    def fill(j, v):
        as_f32(v)[...] = X if j == 0 else G

    with run_case(op, a, sig, fill) as out:
        got = as_f32(out[1] if op == "gelu_fwd" else out[2])
        tiny = 2.0 ** -126
        for lo, hi in pieces(n):
            x = X[lo:hi].astype(np.float64)
            cdf = 0.5 * erfc(-x / math.sqrt(2.0))
            xpdf = np.abs(x) * np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
            if op == "gelu_fwd":
                rep.close("Y", got[lo:hi], ops.gelu_fwd(x), 8 * U * np.abs(x) * (cdf + xpdf) + tiny,
                          lo)
            else:
                g = G[lo:hi]
                rep.close("dX", got[lo:hi], ops.gelu_bwd(x, g.astype(np.float64)),
                          8 * U * np.abs(g) * (cdf + xpdf * (x * x + 2)) + tiny, lo)


def check_attention(op, a, sig, rep, rng):
    """Scores are sums of dh products (sqrt(dh) u of their magnitude); exp of score - max adds
    u of the score's magnitude; the row normalisation and P v sum T terms.  The backward's
    bound is 4 sqrt(T) u times the magnitude of each output, formed by the same products on
    absolute values: every stage (dP = dY v^T, the row sums of dS, dS k, dS^T q, P^T dY) sums
    at most T terms; the backward recomputes P, so the forward's relative bound on P is added
    through both factors of P in dS and through P^T dY."""
    B, T, H, dh, causal = a
    d = H * dh
    qkv = Pool.window(B * T * 3 * d, 0, 3).reshape(B * T, 3 * d)
    heads = sorted({(0, 0), (B - 1, H - 1)} | {(int(b), int(h)) for b, h in
                                                zip(rng.integers(0, B, 4), rng.integers(0, H, 4))})

    def head(M, b, h):
        """[T, 3 dh] columns of one head (its q, k and v) in batch b's rows."""
        rows = M[b * T:(b + 1) * T]
        return np.concatenate([rows[:, p * d + h * dh:p * d + (h + 1) * dh] for p in range(3)],
                              axis=1)

    def p_rel(x):
        """Relative bound on each row of one head's P (x = its q, k, v columns)."""
        q, k = np.abs(x[:, :dh]), np.abs(x[:, dh:2 * dh])
        smag = (q @ k.T).max(axis=1, keepdims=True) / math.sqrt(dh)
        return (2 * math.sqrt(dh) + 4) * U * smag + (math.sqrt(T) + 16) * U

    if op == "attention_fwd":
        def fill(j, v):
            as_f32(v)[...] = qkv.reshape(-1)

        with run_case(op, a, sig, fill) as out:
            Pg = as_f32(out[1]).reshape(B, H, T, T)
            Yg = as_f32(out[2]).reshape(B * T, d)
            for b, h in heads:
                x = head(qkv, b, h).astype(np.float64)
                P, Y = ops.attention_fwd(x, 1, T, 1, bool(causal))
                rel = p_rel(x)
                rep.close(f"P[{b},{h}]", Pg[b, h], P[0, 0], rel * P[0, 0])
                rep.close(f"Y[{b},{h}]", Yg[b * T:(b + 1) * T, h * dh:(h + 1) * dh], Y,
                          (rel + math.sqrt(T) * U) * (P[0, 0] @ np.abs(x[:, 2 * dh:])))
        return
    # backward: P is recomputed from q and k into a variable of its own; dY normal
    G = Pool.window(B * T * d, 2, 3).reshape(B * T, d)

    def fill(j, v):
        as_f32(v)[...] = (qkv.reshape(-1), None, G.reshape(-1))[j]

    with run_case(op, a, sig, fill) as out:
        Pg = as_f32(out[1]).reshape(B, H, T, T)
        dg = as_f32(out[3]).reshape(B * T, 3 * d)
        for b, h in heads:
            x = head(qkv, b, h).astype(np.float64)
            P = ops.attention_fwd(x, 1, T, 1, bool(causal))[0]
            p, rel = P[0, 0], p_rel(x)
            rep.close(f"P[{b},{h}]", Pg[b, h], p, rel * p)
            g = G[b * T:(b + 1) * T, h * dh:(h + 1) * dh].astype(np.float64)
            ref = ops.attention_bwd(x, P, g, 1, T, 1)
            q, k, v = np.abs(x[:, :dh]), np.abs(x[:, dh:2 * dh]), np.abs(x[:, 2 * dh:])
            ga = np.abs(g)
            dP = ga @ v.T
            dS = p * (dP + (dP * p).sum(axis=1, keepdims=True)) / math.sqrt(dh)
            mag = np.concatenate([dS @ k, dS.T @ q, p.T @ ga], axis=1)
            # the recomputed P's error (rel per row) enters dS through both of its factors
            # of P and dv through P^T dY
            carried = np.concatenate([(2 * rel * dS) @ k, (2 * rel * dS).T @ q,
                                      (rel * p).T @ ga], axis=1)
            rep.close(f"dqkv[{b},{h}]", head(dg, b, h), ref,
                      4 * math.sqrt(T) * U * mag + carried)


CHECKS = {"conv_fwd": check_conv, "conv_bwd_x": check_conv, "conv_bwd_w": check_conv,
          "linear_fwd": check_linear, "linear_bwd_x": check_linear,
          "linear_bwd_w": check_linear, "bn_fwd": check_bn, "bn_bwd": check_bn,
          "relu_fwd": check_elementwise, "relu_bwd": check_elementwise,
          "add": check_elementwise, "acc": check_elementwise, "maxpool_fwd": check_pool, "maxpool_bwd": check_pool,
          "avgpool_fwd": check_pool, "avgpool_bwd": check_pool, "softmax_ce": check_softmax,
          "sgd": check_sgd, "embed_fwd": check_embed, "embed_bwd": check_embed,
          "layernorm_fwd": check_layernorm, "layernorm_bwd": check_layernorm,
          "gelu_fwd": check_gelu, "gelu_bwd": check_gelu,
          "attention_fwd": check_attention, "attention_bwd": check_attention}


@pytest.mark.parametrize("cid,op,attrs,sig", CASES, ids=[c[0] for c in CASES])
def test_full_size_function_matches_oracle(cid, op, attrs, sig):
    print(f"{cid}: {sum(b for b, _ in sig) / 2 ** 30:.2f} GiB", flush=True)
    rep = Report(cid)
    CHECKS[op](op, attrs, sig, rep, np.random.default_rng(zlib.crc32(cid.encode())))
    print(f"{cid}: worst error / bound {rep.worst:.3f}", flush=True)

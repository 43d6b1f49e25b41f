"""Every kernel against the float64 oracle, one function at a time (GPU).

Each case registers one function whose inputs are INPUT/PARAM variables and
whose results are OUTPUT variables, runs it in-core through the C interface
and compares with ``oracle.ops``.  Shapes are ragged on purpose: they span
several 128 x 128 tiles and end in partial tiles, use channel counts that are
and are not multiples of 4, and include empty split-K slices.

Tolerance: relative L2 error <= 2e-5.  An fp32 sum of n terms carries a
relative rounding error of order sqrt(n) * 6e-8; the longest reductions here
(n <= 4608) stay below 5e-6, so 2e-5 leaves margin without hiding a wrong
term (a dropped tap or a transposed operand is an O(1) error).
"""

import numpy as np
import pytest

from oracle import mixop, ops
from paper_2010_14109_amd import ooc
from tests.gpu_util import rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-5
rng = np.random.default_rng(77)

NPT = {"f32": np.float32, "i32": np.int32, "u8": np.uint8, "u32": np.uint32}


def run_fn(op, args, attrs, chunk=4096):
    """args: list of (array or (shape, dtype), access); arrays are inputs, tuples outputs.
    Returns the final value of every variable, in order.  Variables of tens of MiB need a
    chunk larger than the 4 KiB default: tens of thousands of 4 KiB mappings are refused."""
    ctx = ooc.Context(0)
    try:
        ids, dts = [], []
        for a, acc in args:
            if isinstance(a, np.ndarray):
                kind = ooc.INPUT if acc == ooc.R else ooc.PARAM
                ids.append(ctx.add_var(a.nbytes, kind))
                dts.append((a.shape, a.dtype))
            else:
                shape, dt = a
                nb = int(np.prod(shape)) * np.dtype(NPT[dt]).itemsize
                ids.append(ctx.add_var(nb, ooc.OUTPUT))
                dts.append((shape, np.dtype(NPT[dt])))
        ctx.add_fn(op, ids, [acc for _, acc in args], attrs)
        ctx.set_chunk(chunk)
        ctx.build_schedule()
        ctx.prepare()
        for (a, _), v, (shape, dt) in zip(args, ids, dts):
            if isinstance(a, np.ndarray):
                ctx.host_view(v, dt)[...] = a.reshape(-1)
        ctx.upload()
        ctx.step(0.0, 0.0)
        ctx.download()
        out = []
        for (a, acc), v, (shape, dt) in zip(args, ids, dts):
            if acc == ooc.R:
                out.append(None)
            else:
                out.append(np.array(ctx.host_view(v, dt)).reshape(shape))
        return out
    finally:
        ctx.close()


def f32(*shape, scale=1.0):
    return (rng.standard_normal(shape) * scale).astype(np.float32)


def d(a):
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------- dense
@pytest.mark.parametrize("M,K,N,S", [(300, 200, 130, 1), (5, 147, 10, 1), (256, 1024, 1024, 1),
                                     (1, 3, 1, 1), (3000, 200, 132, 3), (2500, 64, 1000, 2),
                                     (4100, 36, 7, 5), (100, 40, 20, 3),
                                     # reductions of at most 128 (the persistent form) over more
                                     # tiles than workgroups, ragged rows and columns: forward,
                                     # input gradient, and a scalar-loader forward on 256 x 64
                                     (70001, 100, 130, 1), (70001, 130, 100, 1),
                                     (200001, 37, 45, 1),
                                     # few output tiles (64 x 64 tiles), reductions of at most
                                     # 128 among them, ragged rows and columns
                                     (640, 96, 640, 1), (333, 120, 257, 1)])
def test_linear(M, K, N, S):
    """S > 1 cuts the rows of the weight gradient into slices (the last one of
    (100, 40, 20, 3) is empty)."""
    X, Wt, b, G = f32(M, K), f32(N, K), f32(N), f32(M, N)
    print(f"linear M={M} K={K} N={N} slices={S}", flush=True)
    chunk = 2 << 20 if M * max(K, N) > (1 << 22) else 4096
    (_, _, _, Y) = run_fn("linear_fwd", [(X, ooc.R), (Wt, ooc.R), (b, ooc.R),
                                          (((M, N), "f32"), ooc.W)], [M, K, N], chunk)
    assert rel_err(Y, ops.linear_fwd(d(X), d(Wt), d(b))) < TOL
    wargs = [(X, ooc.R), (G, ooc.R), (((N, K), "f32"), ooc.W), (((N,), "f32"), ooc.W)]
    if S > 1:
        wargs.append((((S * (N * K + N),), "f32"), ooc.W))
    dW, db = run_fn("linear_bwd_w", wargs, [M, K, N, S], chunk)[2:4]
    rdW, rdb = ops.linear_bwd_w(d(X), d(G))
    assert rel_err(dW, rdW) < TOL and rel_err(db, rdb) < TOL
    (_, _, dX) = run_fn("linear_bwd_x", [(Wt, ooc.R), (G, ooc.R), (((M, K), "f32"), ooc.W)],
                        [M, K, N], chunk)
    assert rel_err(dX, ops.linear_bwd_x(d(Wt), d(G))) < TOL


# ---------------------------------------------------------------- conv
CONVS = [  # N, H, W, C, K, k, stride, pad
    (2, 9, 9, 4, 8, 3, 1, 1),
    (2, 9, 9, 4, 8, 3, 2, 1),
    (2, 15, 13, 3, 8, 7, 2, 3),
    (2, 9, 9, 8, 12, 1, 1, 0),
    (2, 9, 10, 8, 12, 1, 2, 0),
    (3, 8, 8, 64, 64, 3, 1, 1),
    (1, 5, 5, 132, 136, 3, 1, 1),
    # channel counts that are multiples of 32 (one filter tap per K tile), strided input
    # gradients split into stride classes, classes no tap reaches (1x1 stride 2), stride 3
    (2, 11, 9, 32, 64, 3, 2, 1),
    (2, 10, 7, 64, 32, 1, 2, 0),
    (1, 9, 9, 64, 40, 3, 2, 1),
    (2, 7, 7, 32, 36, 5, 2, 2),
    (1, 8, 7, 4, 6, 3, 3, 1),
    (1, 4, 4, 32, 32, 1, 3, 0),
    # filter gradients on 64 x 192 tiles whose last tile is ragged (RSC 540 and 180)
    (2, 9, 9, 60, 20, 3, 1, 1),
    (1, 7, 6, 20, 64, 3, 2, 1),
    # filter gradients on 64 x 64 tiles (3 input channels, RSC 27; a 1 x 1 64 -> 64 filter) and on
    # 32 x 256 tiles with a ragged last tile (128 -> 32 channels, RSC 1152); forward on 128 x 32
    (2, 10, 9, 3, 64, 3, 1, 1),
    (2, 6, 5, 64, 64, 1, 1, 0),
    (1, 6, 6, 128, 32, 3, 1, 1),
    # at most 32 output channels over at least 256 x 256 output rows: forward on 256 x 32, one
    # filter tap per K tile and (ragged, 66560 rows) four channels per load
    (4, 128, 128, 32, 32, 3, 1, 1),
    (4, 128, 130, 4, 16, 3, 1, 1),
    # at least 65536 output rows and 64 columns: 256 x 64 tiles with a ragged last tile
    # (66825 rows), for the 3 x 3 forward and input gradient, the stride-2 classes and the
    # pointwise (dense) path
    (33, 45, 45, 64, 64, 3, 1, 1),
    (33, 90, 90, 64, 64, 3, 2, 1),
    (33, 45, 45, 64, 64, 1, 1, 0),
]


@pytest.mark.parametrize("shape", CONVS, ids=lambda s: "x".join(map(str, s)))
def test_conv(shape):
    N, H, Wd, C, K, k, st, pd = shape
    print(f"conv {shape}", flush=True)
    P, Q = (H + 2 * pd - k) // st + 1, (Wd + 2 * pd - k) // st + 1
    a = [N, H, Wd, C, K, k, k, st, pd, P, Q]
    # variables are virtually contiguous whatever the chunk; 2 MiB chunks keep the tensors of
    # millions of elements to a few hundred mappings (each one a driver call) per run
    chunk = 2 << 20 if max(N * H * Wd * C, N * P * Q * K) > (1 << 20) else 4096
    X, Wt, G = f32(N, H, Wd, C), f32(K, k, k, C), f32(N, P, Q, K)
    (_, _, Y) = run_fn("conv_fwd", [(X, ooc.R), (Wt, ooc.R), (((N, P, Q, K), "f32"), ooc.W)], a,
                       chunk)
    assert rel_err(Y, ops.conv_fwd(d(X), d(Wt), st, pd)) < TOL
    ref_dW = ops.conv_bwd_w(d(X), d(G), Wt.shape, st, pd)
    for slices in sorted({1, ooc.wgrad_slices("conv_bwd_w", a), 3, 7}):
        slices = min(slices, N * P * Q)
        args = [(X, ooc.R), (G, ooc.R), (((K, k, k, C), "f32"), ooc.W)]
        if slices > 1:
            args.append((((slices * K * k * k * C,), "f32"), ooc.W))
        out = run_fn("conv_bwd_w", args, a + [slices], chunk)
        assert rel_err(out[2], ref_dW) < TOL, slices
    if C % 4 == 0:
        (_, _, dX) = run_fn("conv_bwd_x", [(Wt, ooc.R), (G, ooc.R),
                                            (((N, H, Wd, C), "f32"), ooc.W)], a, chunk)
        assert rel_err(dX, ops.conv_bwd_x(d(Wt), d(G), X.shape, st, pd)) < TOL


def test_conv_bwd_x_fills_unreached_classes():
    """A 1 x 1 stride-2 input gradient reaches one stride class of four; the other pixels must
    be written as zeros, not left as they were.  Out of core at the smallest budget the output
    is mapped onto chunks that held the ones a ReLU wrote just before."""
    N, H, Wd, C, K = 2, 10, 7, 64, 32
    P, Q = 5, 4
    n = N * H * Wd * C
    Wt, G = f32(K, 1, 1, C), f32(N, P, Q, K)
    ctx = ooc.Context(0)
    try:
        x1 = ctx.add_var(n * 4, ooc.INPUT)
        t = ctx.add_var(n * 4, ooc.TEMP)
        w = ctx.add_var(Wt.nbytes, ooc.INPUT)
        g = ctx.add_var(G.nbytes, ooc.INPUT)
        dx = ctx.add_var(n * 4, ooc.OUTPUT)
        ctx.add_fn("relu_fwd", [x1, t], [ooc.R, ooc.W], [n])
        ctx.add_fn("conv_bwd_x", [w, g, dx], [ooc.R, ooc.R, ooc.W],
                   [N, H, Wd, C, K, 1, 1, 2, 0, P, Q])
        ctx.set_chunk(4096)
        ctx.set_budget(ctx.working_set_max())
        ctx.build_schedule()
        held = {iv["var"]: set(iv["chunks"]) for iv in ctx.plan()}
        assert held[dx] & (held[x1] | held[t]), "the output must reuse chunks that held ones"
        ctx.prepare()
        ctx.host_view(x1, np.float32)[...] = 1.0
        ctx.host_view(w, np.float32)[...] = Wt.reshape(-1)
        ctx.host_view(g, np.float32)[...] = G.reshape(-1)
        ctx.upload()
        ctx.step(0.0, 0.0)
        ctx.download()
        got = np.array(ctx.host_view(dx, np.float32)).reshape(N, H, Wd, C)
    finally:
        ctx.close()
    ref = ops.conv_bwd_x(d(Wt), d(G), (N, H, Wd, C), 2, 0)
    assert np.all(got[:, 1::2] == 0) and np.all(got[:, :, 1::2] == 0)
    assert rel_err(got, ref) < TOL


# ---------------------------------------------------------------- BatchNorm
@pytest.mark.parametrize("rows,C,slices", [(162, 12, 1), (162, 12, 5), (162, 6, 4), (4096, 64, 8),
                                           (3, 128, 3),
                                           # above 256 slices the reduction runs in two passes:
                                           # empty trailing slices, a ragged last slice group
                                           (4096, 64, 300), (5000, 12, 513), (3000, 5, 257),
                                           # the plain CNN's shape, slices of ragged length, 4
                                           # and 128 channels, 1024 slices
                                           (131072, 64, 256), (1000, 64, 2), (9999, 4, 20),
                                           (1000, 128, 4), (524288, 64, 1024)])
def test_batchnorm(rows, C, slices):
    X = f32(rows, C, scale=2.0) + 0.5
    g, b, G = f32(C), f32(C), f32(rows, C)
    sb = (2 + 2 * slices) * C
    chunk = 2 << 20 if rows * C > (1 << 22) else 4096
    print(f"bn rows={rows} C={C} slices={slices}", flush=True)
    (_, _, _, Y, st) = run_fn("bn_fwd", [(X, ooc.R), (g, ooc.R), (b, ooc.R),
                                          (((rows, C), "f32"), ooc.W), (((sb,), "f32"), ooc.W)],
                              [rows, C, slices], chunk)
    rY, mean, invstd = ops.bn_fwd(d(X), d(g), d(b))
    assert rel_err(Y, rY) < TOL
    assert rel_err(st[:C], mean) < TOL and rel_err(st[C:2 * C], invstd) < TOL
    out = run_fn("bn_bwd", [(X, ooc.R), (g, ooc.R), (st.astype(np.float32), ooc.RW), (G, ooc.R),
                            (((rows, C), "f32"), ooc.W), (((C,), "f32"), ooc.W),
                            (((C,), "f32"), ooc.W)], [rows, C, slices], chunk)
    rdX, rdg, rdb = ops.bn_bwd(d(X), d(g), d(st[:C]), d(st[C:2 * C]), d(G))
    assert rel_err(out[4], rdX) < TOL and rel_err(out[5], rdg) < TOL and rel_err(out[6], rdb) < TOL


# ---------------------------------------------------------------- elementwise
@pytest.mark.parametrize("n", [1003, 4096, 1, 4 * 262144 + 3])
def test_relu_add(n):
    x, y, g = f32(n), f32(n), f32(n)
    (_, r) = run_fn("relu_fwd", [(x, ooc.R), (((n,), "f32"), ooc.W)], [n])
    assert np.array_equal(r, ops.relu_fwd(x))
    (_, _, dx) = run_fn("relu_bwd", [(r, ooc.R), (g, ooc.R), (((n,), "f32"), ooc.W)], [n])
    assert np.array_equal(dx, ops.relu_bwd(r, g))
    (_, _, s) = run_fn("add", [(x, ooc.R), (y, ooc.R), (((n,), "f32"), ooc.W)], [n])
    assert np.array_equal(s, x + y)
    (a, _) = run_fn("acc", [(x, ooc.RW), (y, ooc.R)], [n])      # in place: x += y
    assert np.array_equal(a, x + y)


def test_sgd_plain_and_momentum():
    n = 1001
    ctx_args = []
    w, g, v = f32(n), f32(n), f32(n)
    ctx = ooc.Context(0)
    try:
        iw, ig, iv = ctx.add_var(n * 4, ooc.PARAM), ctx.add_var(n * 4, ooc.INPUT), \
            ctx.add_var(n * 4, ooc.STATE)
        iw2 = ctx.add_var(n * 4, ooc.PARAM)
        ctx.add_fn("sgd", [iw, ig, iv], [ooc.RW, ooc.R, ooc.RW], [1, 1])
        ctx.add_fn("sgd", [iw2, ig], [ooc.RW, ooc.R], [1, 0])
        ctx.set_chunk(4096)
        ctx.build_schedule()
        ctx.prepare()
        for i, a in ((iw, w), (ig, g), (iv, v), (iw2, w)):
            ctx.host_view(i)[...] = a
        ctx.upload()
        ctx.step(0.1, 0.9)
        ctx.download()
        rw, rv = ops.sgd_momentum(d(w), d(g), d(v), 0.1, 0.9)
        assert rel_err(ctx.host_view(iw), rw) < 1e-6 and rel_err(ctx.host_view(iv), rv) < 1e-6
        assert rel_err(ctx.host_view(iw2), ops.sgd(d(w), d(g), 0.1)) < 1e-6
    finally:
        ctx.close()
    del ctx_args


@pytest.mark.parametrize("mom", [1, 0])
def test_sgd_many_tensors_in_one_function(mom):
    """One update function over 11 tensors (more than one launch's set of 8), sizes from 1 to
    70001 elements, so that each tensor's grid row differs from the launch's widest."""
    sizes = [1, 3, 4, 5000, 70001, 64, 7, 12288, 2, 999, 4096]
    lr, mu = 0.05, 0.9 if mom else 0.0
    ws, gs, vs = [f32(n) for n in sizes], [f32(n) for n in sizes], [f32(n) for n in sizes]
    ctx = ooc.Context(0)
    try:
        ids, acc = [], []
        for n in sizes:
            ids.append(ctx.add_var(n * 4, ooc.PARAM))
            ids.append(ctx.add_var(n * 4, ooc.INPUT))
            acc += [ooc.RW, ooc.R]
            if mom:
                ids.append(ctx.add_var(n * 4, ooc.STATE))
                acc.append(ooc.RW)
        ctx.add_fn("sgd", ids, acc, [len(sizes), mom])
        ctx.set_chunk(4096)
        ctx.build_schedule()
        ctx.prepare()
        per = 3 if mom else 2
        for k in range(len(sizes)):
            ctx.host_view(ids[per * k])[...] = ws[k]
            ctx.host_view(ids[per * k + 1])[...] = gs[k]
            if mom:
                ctx.host_view(ids[per * k + 2])[...] = vs[k]
        ctx.upload()
        ctx.step(lr, mu)
        ctx.download()
        for k in range(len(sizes)):
            if mom:
                rw, rv = ops.sgd_momentum(d(ws[k]), d(gs[k]), d(vs[k]), lr, mu)
                assert rel_err(ctx.host_view(ids[per * k + 2]), rv) < 1e-6
            else:
                rw = ops.sgd(d(ws[k]), d(gs[k]), lr)
            assert rel_err(ctx.host_view(ids[per * k]), rw) < 1e-6, k
    finally:
        ctx.close()


# ---------------------------------------------------------------- pooling
@pytest.mark.parametrize("C", [8, 6, 64])   # four channels per thread; one per thread (C % 4)
def test_maxpool_with_ties(C):
    N, H, Wd, k, st, pd = 2, 9, 8, 3, 2, 1
    P, Q = (H + 2 * pd - k) // st + 1, (Wd + 2 * pd - k) // st + 1
    X = f32(N, H, Wd, C)
    X[0, 0, 0, :] = X[0, 0, 1, :] = 7.0
    X[1, 4, 4, 3] = X[1, 4, 5, 3] = X[1, 5, 4, 3] = 9.0
    a = [N, H, Wd, C, k, st, pd, P, Q]
    (_, Y, idx) = run_fn("maxpool_fwd", [(X, ooc.R), (((N, P, Q, C), "f32"), ooc.W),
                                         (((N, P, Q, C), "u8"), ooc.W)], a)
    rY, ridx = ops.maxpool_fwd(d(X), k, st, pd)
    assert np.array_equal(Y, rY.astype(np.float32)) and np.array_equal(idx, ridx)
    G = f32(N, P, Q, C)
    (_, _, dX) = run_fn("maxpool_bwd", [(ridx, ooc.R), (G, ooc.R),
                                        (((N, H, Wd, C), "f32"), ooc.W)], a)
    assert rel_err(dX, ops.maxpool_bwd(ridx, d(G), X.shape, k, st, pd)) < 1e-6


@pytest.mark.parametrize("H,Wd,C", [(7, 5, 12), (17, 19, 70)])   # 4 and 16 waves per workgroup
def test_avgpool(H, Wd, C):
    N = 3
    X, G = f32(N, H, Wd, C), f32(N, C)
    (_, Y) = run_fn("avgpool_fwd", [(X, ooc.R), (((N, C), "f32"), ooc.W)], [N, H, Wd, C])
    assert rel_err(Y, ops.avgpool_fwd(d(X))) < TOL
    (_, dX) = run_fn("avgpool_bwd", [(G, ooc.R), (((N, H, Wd, C), "f32"), ooc.W)], [N, H, Wd, C])
    assert rel_err(dX, ops.avgpool_bwd(d(G), X.shape)) < TOL


# ---------------------------------------------------------------- loss
@pytest.mark.parametrize("N,C", [(37, 10), (5, 1000), (1, 1), (70001, 3), (16387, 2)])
def test_softmax_ce(N, C):
    Z = f32(N, C, scale=3.0)
    y = rng.integers(0, C, N).astype(np.int32)
    (_, _, loss, dZ) = run_fn("softmax_ce", [(Z, ooc.R), (y, ooc.R), (((N + 1,), "f32"), ooc.W),
                                             (((N, C), "f32"), ooc.W)], [N, C])
    rows, mean, rdZ = ops.softmax_ce(d(Z), y)
    assert rel_err(loss[:N], rows) < TOL and abs(loss[N] - mean) <= TOL * abs(mean) + 1e-7
    assert rel_err(dZ, rdZ) < TOL or np.abs(dZ - rdZ).max() < 1e-7


def test_softmax_ce_out_of_range_label():
    N, C = 4, 6
    Z = f32(N, C)
    y = np.array([0, 6, -1, 5], dtype=np.int32)
    (_, _, loss, dZ) = run_fn("softmax_ce", [(Z, ooc.R), (y, ooc.R), (((N + 1,), "f32"), ooc.W),
                                             (((N, C), "f32"), ooc.W)], [N, C])
    assert np.isnan(loss[1]) and np.isnan(loss[2]) and np.isnan(loss[N])
    assert np.all(dZ[1] == 0) and np.all(dZ[2] == 0)
    rows, _, rdZ = ops.softmax_ce(d(Z[[0, 3]]), y[[0, 3]])
    assert rel_err(loss[[0, 3]], rows) < TOL


# ---------------------------------------------------------------- integrity op
def test_mix_op():
    a = rng.integers(0, 2 ** 32, 17, dtype=np.uint64).astype(np.uint32)
    b = rng.integers(0, 2 ** 32, 5, dtype=np.uint64).astype(np.uint32)
    y0 = rng.integers(0, 2 ** 32, 9, dtype=np.uint64).astype(np.uint32)
    (_, _, y) = run_fn("mix", [(a, ooc.R), (b, ooc.R), (y0, ooc.RW)], [12345])
    assert np.array_equal(y, mixop.mix([a, b, y0], 9, 12345))
    (_, y) = run_fn("mix", [(a, ooc.R), (((33,), "u32"), ooc.W)], [7])
    assert np.array_equal(y, mixop.mix([a], 33, 7))


# ---------------------------------------------------------------- concatenation, upsampling
@pytest.mark.parametrize("rows,cs", [(37, (8, 12)), (37, (3, 5, 1)), (1, (4,)), (1000, (64, 32, 32)),
                                     (50, (64,) + (32,) * 14 + (3, 4, 5, 32))])
def test_concat(rows, cs):
    parts = [f32(rows, c) for c in cs]
    ct = sum(cs)
    print(f"concat rows={rows} cs={cs}", flush=True)
    out = run_fn("concat_fwd", [(p, ooc.R) for p in parts] + [(((rows, ct), "f32"), ooc.W)],
                 [rows] + list(cs))
    assert np.array_equal(out[-1], np.concatenate(parts, axis=1))
    G = f32(rows, ct)
    back = run_fn("concat_bwd", [(G, ooc.R)] + [(((rows, c), "f32"), ooc.W) for c in cs],
                  [rows] + list(cs))
    for got, ref in zip(back[1:], ops.concat_bwd(G, list(cs))):
        assert np.array_equal(got, ref)


@pytest.mark.parametrize("N,H,W,C", [(2, 3, 5, 8), (1, 4, 4, 3), (2, 16, 16, 64)])
def test_upsample(N, H, W, C):
    X = f32(N, H, W, C)
    print(f"upsample {N}x{H}x{W}x{C}", flush=True)
    (_, Y) = run_fn("upsample_fwd", [(X, ooc.R), (((N, 2 * H, 2 * W, C), "f32"), ooc.W)],
                    [N, H, W, C])
    assert np.array_equal(Y, ops.upsample_fwd(X))
    G = f32(N, 2 * H, 2 * W, C)
    (_, dX) = run_fn("upsample_bwd", [(G, ooc.R), (((N, H, W, C), "f32"), ooc.W)], [N, H, W, C])
    g = G.reshape(N, H, 2, W, 2, C)
    ref = ((g[:, :, 0, :, 0] + g[:, :, 0, :, 1]) + g[:, :, 1, :, 0]) + g[:, :, 1, :, 1]
    assert np.array_equal(dX, ref)         # same fp32 order as the kernel: bit-exact


# ---------------------------------------------------------------- transformer layers
@pytest.mark.parametrize("rows,d,slices", [(37, 64, 1), (37, 100, 3), (130, 1024, 4), (5, 4096, 2),
                                          (2000, 1024, 63), (999, 100, 37), (40, 66, 2),
                                          (300, 2048, 9)])
def test_layernorm(rows, d, slices):
    X = f32(rows, d, scale=2.0) + 0.3
    g, b, G = f32(d), f32(d), f32(rows, d)
    sb = 2 * rows + 2 * slices * d
    print(f"layernorm rows={rows} d={d} slices={slices}", flush=True)
    (_, _, _, Y, st) = run_fn("layernorm_fwd", [(X, ooc.R), (g, ooc.R), (b, ooc.R),
                                                 (((rows, d), "f32"), ooc.W),
                                                 (((sb,), "f32"), ooc.W)], [rows, d, slices])
    rY, mean, rstd = ops.layernorm_fwd(X.astype(np.float64), g.astype(np.float64),
                                       b.astype(np.float64))
    assert rel_err(Y, rY) < TOL
    assert rel_err(st[:rows], mean) < TOL and rel_err(st[rows:2 * rows], rstd) < TOL
    out = run_fn("layernorm_bwd", [(X, ooc.R), (g, ooc.R), (st.astype(np.float32), ooc.RW),
                                   (G, ooc.R), (((rows, d), "f32"), ooc.W),
                                   (((d,), "f32"), ooc.W), (((d,), "f32"), ooc.W)],
                 [rows, d, slices])
    rdX, rdg, rdb = ops.layernorm_bwd(X.astype(np.float64), g.astype(np.float64), mean, rstd,
                                      G.astype(np.float64))
    assert rel_err(out[4], rdX) < TOL and rel_err(out[5], rdg) < TOL and rel_err(out[6], rdb) < TOL


@pytest.mark.parametrize("n", [1003, 1, 64, 4 * (16384 * 256 + 5)])
def test_gelu(n):
    """n = 64 spans the lower tail (x down to -12), where GELU is tiny but not 0.  Sizes that are
    multiples of 4 take the four-wide kernel; the largest needs two grid-stride passes."""
    x, g = f32(n, scale=3.0), f32(n)
    if n == 64:
        x = np.linspace(-12.0, 4.0, n).astype(np.float32)
    chunk = 4096 if n < 1 << 20 else 2 << 20
    (_, y) = run_fn("gelu_fwd", [(x, ooc.R), (((n,), "f32"), ooc.W)], [n], chunk)
    assert rel_err(y, ops.gelu_fwd(x.astype(np.float64))) < TOL
    (_, _, dx) = run_fn("gelu_bwd", [(x, ooc.R), (g, ooc.R), (((n,), "f32"), ooc.W)], [n], chunk)
    assert rel_err(dx, ops.gelu_bwd(x.astype(np.float64), g.astype(np.float64))) < TOL


@pytest.mark.parametrize("B,T,V,dm", [(3, 5, 17, 64), (2, 7, 40, 48), (4, 64, 1000, 1024)])
def test_embedding(B, T, V, dm):
    ids = rng.integers(0, V, (B, T)).astype(np.int32)
    ids[0, 0] = ids[-1, -1] = 3                        # a repeated token
    E, pos, G = f32(V, dm), f32(T, dm), f32(B * T, dm)
    (_, _, _, Y) = run_fn("embed_fwd", [(ids, ooc.R), (E, ooc.R), (pos, ooc.R),
                                        (((B * T, dm), "f32"), ooc.W)], [B, T, V, dm])
    assert np.array_equal(Y, ops.embed_fwd(ids, E, pos))
    (_, _, dE, dpos) = run_fn("embed_bwd", [(ids, ooc.R), (G, ooc.R), (((V, dm), "f32"), ooc.W),
                                            (((T, dm), "f32"), ooc.W)], [B, T, V, dm])
    rdE, rdpos = ops.embed_bwd(ids, G.astype(np.float64), V)
    assert rel_err(dE, rdE) < TOL and rel_err(dpos, rdpos) < TOL


def test_embedding_out_of_range_id():
    B, T, V, dm = 1, 3, 5, 64
    ids = np.array([[0, 7, -2]], dtype=np.int32)
    E, pos = f32(V, dm), f32(T, dm)
    (_, _, _, Y) = run_fn("embed_fwd", [(ids, ooc.R), (E, ooc.R), (pos, ooc.R),
                                        (((B * T, dm), "f32"), ooc.W)], [B, T, V, dm])
    assert np.array_equal(Y[0], E[0] + pos[0]) and np.isnan(Y[1]).all() and np.isnan(Y[2]).all()


@pytest.mark.parametrize("B,T,H,dh,causal", [(2, 6, 2, 8, 1), (2, 64, 4, 16, 1), (1, 130, 2, 64, 1),
                                            (2, 33, 3, 8, 0), (1, 512, 2, 64, 1),
                                            (1, 260, 2, 8, 1), (2, 256, 2, 16, 0),
                                            (1, 392, 1, 16, 0), (1, 1024, 1, 32, 1)])
def test_attention(B, T, H, dh, causal):
    dmod = H * dh
    qkv, G = f32(B * T, 3 * dmod), f32(B * T, dmod)
    print(f"attention B={B} T={T} H={H} dh={dh} causal={causal}", flush=True)
    (_, P, Y) = run_fn("attention_fwd", [(qkv, ooc.R), (((B, H, T, T), "f32"), ooc.W),
                                         (((B * T, dmod), "f32"), ooc.W)], [B, T, H, dh, causal])
    rP, rY = ops.attention_fwd(qkv.astype(np.float64), B, T, H, bool(causal))
    assert rel_err(P, rP) < TOL and rel_err(Y, rY) < TOL
    if causal:   # masked scores are exact zeros, also in tiles the products skip
        assert not np.triu(P.reshape(B * H, T, T), 1).any()
    # the backward recomputes P into its own buffer with the forward's kernels: bit for bit
    out = run_fn("attention_bwd", [(qkv, ooc.R), (((B, H, T, T), "f32"), ooc.W), (G, ooc.R),
                                   (((B * T, 3 * dmod), "f32"), ooc.W),
                                   (((B, H, T, T), "f32"), ooc.W)], [B, T, H, dh, causal])
    assert np.array_equal(out[1], P)
    rd = ops.attention_bwd(qkv.astype(np.float64), rP, G.astype(np.float64), B, T, H)
    assert rel_err(out[3], rd) < TOL

"""Pins of the oracle's float64 training step (CPU only).

Nothing here retypes an oracle formula: each op is checked against central
finite differences of its forward, a library routine for a special case
(scipy correlation, numpy matmul), a brute-force loop, or an identity the
mathematics fixes (BatchNorm gradients are orthogonal to 1 and x_hat; a
stride-1 convolution's input gradient is the correlation with the flipped,
channel-swapped kernel).  Whole tiny networks are checked end to end by
finite differences of the loss against the gradients the function sequence
produces, which pins the lowering's wiring as well.
"""

import zlib

import numpy as np
import pytest
from scipy import signal

from oracle import ops
from oracle.interp import run
from oracle.lower import lower
from paper_2010_14109_amd import synth

rng = np.random.default_rng(1234)


def fd_grad(f, x, h=1e-6, n=None, seed=0):
    """Central finite differences of scalar f at (a sample of) the entries of x."""
    flat = x.reshape(-1)
    idx = np.arange(flat.size)
    if n is not None and n < flat.size:
        idx = np.random.default_rng(seed).choice(flat.size, n, replace=False)
    g = np.zeros(len(idx))
    for j, i in enumerate(idx):
        old = flat[i]
        flat[i] = old + h
        fp = f()
        flat[i] = old - h
        fm = f()
        flat[i] = old
        g[j] = (fp - fm) / (2 * h)
    return idx, g


def assert_close(a, b, rtol=1e-6):
    a, b = np.asarray(a), np.asarray(b)
    err = np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30)
    assert err <= rtol, f"relative error {err:.3e}"


# ---------------------------------------------------------------- per op
def test_linear_matches_matmul_and_fd():
    X, W, b = rng.standard_normal((5, 7)), rng.standard_normal((3, 7)), rng.standard_normal(3)
    Y = ops.linear_fwd(X, W, b)
    ref = np.array([[sum(X[n, k] * W[o, k] for k in range(7)) + b[o] for o in range(3)]
                    for n in range(5)])
    assert_close(Y, ref, 1e-12)
    G = rng.standard_normal((5, 3))
    dW, db = ops.linear_bwd_w(X, G)
    dX = ops.linear_bwd_x(W, G)
    loss = lambda: float((ops.linear_fwd(X, W, b) * G).sum())
    for arr, got in ((X, dX), (W, dW), (b, db)):
        idx, g = fd_grad(loss, arr)
        assert_close(got.reshape(-1)[idx], g)


@pytest.mark.parametrize("stride,pad,k", [(1, 1, 3), (2, 1, 3), (2, 3, 7), (1, 0, 1), (2, 0, 1)])
def test_conv_forward_matches_scipy(stride, pad, k):
    N, H, Wd, C, K = 2, 9, 8, 3, 4
    X = rng.standard_normal((N, H, Wd, C))
    Wt = rng.standard_normal((K, k, k, C))
    Y = ops.conv_fwd(X, Wt, stride, pad)
    for n in range(N):
        for o in range(K):
            acc = 0
            for c in range(C):
                xp = np.pad(X[n, :, :, c], pad)
                acc = acc + signal.correlate2d(xp, Wt[o, :, :, c], mode="valid")
            assert_close(Y[n, :, :, o], acc[::stride, ::stride], 1e-12)


@pytest.mark.parametrize("stride,pad,k", [(1, 1, 3), (2, 1, 3), (2, 3, 7), (2, 0, 1)])
def test_conv_backward_fd(stride, pad, k):
    N, H, Wd, C, K = 2, 7, 6, 3, 2
    X = rng.standard_normal((N, H, Wd, C))
    Wt = rng.standard_normal((K, k, k, C))
    Y = ops.conv_fwd(X, Wt, stride, pad)
    G = rng.standard_normal(Y.shape)
    loss = lambda: float((ops.conv_fwd(X, Wt, stride, pad) * G).sum())
    dX = ops.conv_bwd_x(Wt, G, X.shape, stride, pad)
    dW = ops.conv_bwd_w(X, G, Wt.shape, stride, pad)
    for arr, got in ((X, dX), (Wt, dW)):
        idx, g = fd_grad(loss, arr, n=60)
        assert_close(got.reshape(-1)[idx], g)


def test_conv_input_gradient_is_flipped_correlation():
    """Stride 1: dX = correlation of dY with the kernel flipped in space and with input and
    output channels swapped, padding k - 1 - pad."""
    N, H, Wd, C, K, k, pad = 2, 6, 5, 3, 4, 3, 1
    Wt = rng.standard_normal((K, k, k, C))
    G = rng.standard_normal((N, H, Wd, K))
    dX = ops.conv_bwd_x(Wt, G, (N, H, Wd, C), 1, pad)
    flipped = Wt[:, ::-1, ::-1, :].transpose(3, 1, 2, 0).copy()   # [C, R, S, K]
    assert_close(dX, ops.conv_fwd(G, flipped, 1, k - 1 - pad), 1e-12)


def test_batchnorm_identities_and_fd():
    X = rng.standard_normal((3, 4, 5, 6)) * 2 + 0.5
    gamma, beta = rng.standard_normal(6), rng.standard_normal(6)
    Y, mean, invstd = ops.bn_fwd(X, gamma, beta)
    # normalised output has zero mean and (biased) unit variance per channel
    xhat = (Y - beta) / gamma
    assert np.allclose(xhat.mean(axis=(0, 1, 2)), 0, atol=1e-12)
    assert np.allclose((xhat ** 2).mean(axis=(0, 1, 2)), 1 - ops.BN_EPS * invstd ** 2, atol=1e-12)
    assert np.allclose(mean, X.reshape(-1, 6).mean(axis=0))
    assert np.allclose(1 / invstd ** 2 - ops.BN_EPS, X.reshape(-1, 6).var(axis=0))
    G = rng.standard_normal(X.shape)
    dX, dg, db = ops.bn_bwd(X, gamma, mean, invstd, G)
    # dX is orthogonal to 1 per channel; against x_hat only up to the eps term:
    # sum(dX x_hat) = gamma dgamma eps invstd^3 (it vanishes as eps -> 0)
    assert np.allclose(dX.sum(axis=(0, 1, 2)), 0, atol=1e-10)
    assert np.allclose((dX * xhat).sum(axis=(0, 1, 2)), gamma * dg * ops.BN_EPS * invstd ** 3,
                       rtol=1e-6, atol=1e-13)
    loss = lambda: float((ops.bn_fwd(X, gamma, beta)[0] * G).sum())
    for arr, got in ((X, dX), (gamma, dg), (beta, db)):
        idx, g = fd_grad(loss, arr, n=60)
        assert_close(got.reshape(-1)[idx], g, 1e-6)


def test_relu_fd():
    X = rng.standard_normal((4, 9))
    G = rng.standard_normal(X.shape)
    dX = ops.relu_bwd(ops.relu_fwd(X), G)
    idx, g = fd_grad(lambda: float((ops.relu_fwd(X) * G).sum()), X)
    assert_close(dX.reshape(-1)[idx], g)


def test_maxpool_brute_force_and_ties():
    X = rng.standard_normal((2, 7, 6, 3))
    X[0, 0, 0, 0] = X[0, 0, 1, 0] = 5.0          # a tie inside one window
    Y, idx = ops.maxpool_fwd(X, 3, 2, 1)
    N, H, Wd, C = X.shape
    for n in range(N):
        for p in range(Y.shape[1]):
            for q in range(Y.shape[2]):
                for c in range(C):
                    best, bi = None, None
                    for r in range(3):
                        for s in range(3):
                            h, w = 2 * p + r - 1, 2 * q + s - 1
                            if 0 <= h < H and 0 <= w < Wd and (best is None or X[n, h, w, c] > best):
                                best, bi = X[n, h, w, c], r * 3 + s
                    assert Y[n, p, q, c] == best and idx[n, p, q, c] == bi
    # first of the tied taps (row-major) wins: window (0,0) has taps (r,s) = (1,1) and (1,2)
    assert idx[0, 0, 0, 0] == 4
    G = rng.standard_normal(Y.shape)
    dX = ops.maxpool_bwd(idx, G, X.shape, 3, 2, 1)
    X2 = X.copy()
    X2[0, 0, 1, 0] = 4.0                           # remove the tie for the FD check
    Y2, idx2 = ops.maxpool_fwd(X2, 3, 2, 1)
    dX2 = ops.maxpool_bwd(idx2, G, X2.shape, 3, 2, 1)
    i_, g = fd_grad(lambda: float((ops.maxpool_fwd(X2, 3, 2, 1)[0] * G).sum()), X2)
    assert_close(dX2.reshape(-1)[i_], g)
    assert np.isclose(dX.sum(), G.sum())           # every output gradient lands exactly once


def test_avgpool_fd():
    X = rng.standard_normal((2, 3, 4, 5))
    G = rng.standard_normal((2, 5))
    dX = ops.avgpool_bwd(G, X.shape)
    assert_close(ops.avgpool_fwd(X), X.reshape(2, 12, 5).mean(axis=1), 1e-14)
    idx, g = fd_grad(lambda: float((ops.avgpool_fwd(X) * G).sum()), X)
    assert_close(dX.reshape(-1)[idx], g)


def test_softmax_ce_fd_and_properties():
    Z = rng.standard_normal((6, 5)) * 3
    y = rng.integers(0, 5, 6)
    rows, mean, dZ = ops.softmax_ce(Z, y)
    # closed form of the loss on a direct (unshifted) softmax
    p = np.exp(Z) / np.exp(Z).sum(axis=1, keepdims=True)
    assert_close(rows, -np.log(p[np.arange(6), y]), 1e-12)
    assert np.isclose(mean, rows.mean())
    assert np.allclose(dZ.sum(axis=1), 0, atol=1e-15)
    idx, g = fd_grad(lambda: float(ops.softmax_ce(Z, y)[1]), Z)
    assert_close(dZ.reshape(-1)[idx], g)
    # shift invariance and extreme logits stay finite
    big = Z + 1e4
    assert_close(ops.softmax_ce(big, y)[0], rows, 1e-9)


def test_sgd_steps():
    w, g, v = rng.standard_normal(5), rng.standard_normal(5), rng.standard_normal(5)
    assert np.allclose(ops.sgd(w, g, 0.0), w)
    w1, v1 = ops.sgd_momentum(w, g, np.zeros(5), 0.1, 0.9)
    assert np.allclose(v1, g) and np.allclose(w1, ops.sgd(w, g, 0.1))   # v0 = 0: plain SGD
    w2, v2 = ops.sgd_momentum(w, g, v, 0.1, 0.0)
    assert np.allclose(w2, ops.sgd(w, g, 0.1))                           # mu = 0: plain SGD


def test_concat_and_upsample_brute_force_and_fd():
    A, B, C = (rng.standard_normal((2, 3, 4, c)) for c in (2, 5, 1))
    Y = ops.concat_fwd([A, B, C])
    for n in range(2):
        for h in range(3):
            for w in range(4):
                assert list(Y[n, h, w]) == list(A[n, h, w]) + list(B[n, h, w]) + list(C[n, h, w])
    G = rng.standard_normal(Y.shape)
    parts = ops.concat_bwd(G, [2, 5, 1])
    for arr, got in zip((A, B, C), parts):
        idx, g = fd_grad(lambda: float((ops.concat_fwd([A, B, C]) * G).sum()), arr)
        assert_close(got.reshape(-1)[idx], g)
    X = rng.standard_normal((2, 3, 2, 4))
    U = ops.upsample_fwd(X)
    assert U.shape == (2, 6, 4, 4)
    for h in range(6):
        for w in range(4):
            assert np.array_equal(U[:, h, w], X[:, h // 2, w // 2])
    G = rng.standard_normal(U.shape)
    dX = ops.upsample_bwd(G)
    assert np.allclose(dX[1, 2, 1], G[1, 4:6, 2:4].sum(axis=(0, 1)))
    idx, g = fd_grad(lambda: float((ops.upsample_fwd(X) * G).sum()), X)
    assert_close(dX.reshape(-1)[idx], g)


# ---------------------------------------------------------------- whole networks
def tiny_specs():
    return [
        synth.mlp(batch=5, width=6, depth=3, classes=4),
        synth.plain_cnn(batch=3, channels=4, depth=2, hw=5, in_ch=2, classes=3),
        synth.resnet(batch=2, hw=16, classes=5, blocks=(1, 1), width=2, momentum=0.9),
        synth.densenet(batch=2, hw=8, growth=3, blocks=(3, 2), stem=4, classes=4),
        synth.unet(batch=2, hw=8, base=2, depth=2, classes=3),
    ]


@pytest.mark.parametrize("spec", tiny_specs(), ids=lambda s: s["name"])
def test_network_gradients_by_finite_differences(spec):
    reg = lower(spec, keep_grads=True)
    x, labels = synth.make_inputs(spec, seed=3)
    params = {k: v.astype(np.float64) for k, v in synth.make_params(spec, seed=4).items()}
    # zero biases put dead ReLU rows exactly on the kink, where finite differences
    # see half a slope; move every parameter off it
    noise = np.random.default_rng(9)
    for k in params:
        params[k] += 0.1 * noise.standard_normal(params[k].shape)
    env = run(reg, x, labels, params)

    def loss():
        return float(run(reg, x, labels, params)["loss"][-1])

    for name, arr in params.items():
        idx, g = fd_grad(loss, arr, n=6, seed=zlib.crc32(name.encode()) % 1000)
        got = env["d:" + name].reshape(-1)[idx]
        assert np.allclose(got, g, rtol=1e-5, atol=1e-8), name


def test_mlp_loss_matches_direct_forward():
    spec = synth.mlp(batch=7, width=5, depth=3, classes=4)
    x, labels = synth.make_inputs(spec, 0)
    p = {k: v.astype(np.float64) for k, v in synth.make_params(spec, 1).items()}
    h = x.astype(np.float64)
    for i in range(1, 4):
        h = h @ p[f"fc{i}.W"].T + p[f"fc{i}.b"]
        if i < 3:
            h = np.where(h > 0, h, 0)
    logp = h - np.log(np.exp(h).sum(axis=1, keepdims=True))
    direct = -logp[np.arange(7), labels].mean()
    env = run(lower(spec), x, labels, p)
    assert np.isclose(env["loss"][-1], direct, rtol=1e-12)
    # one SGD step by hand for the last layer
    g = np.exp(logp)
    g[np.arange(7), labels] -= 1
    g /= 7
    assert np.allclose(env["fc3.b"], p["fc3.b"] - 0.01 * g.sum(axis=0))


def test_momentum_step_changes_state():
    spec = synth.resnet(batch=2, hw=16, classes=5, blocks=(1, 1), width=2, momentum=0.9)
    reg = lower(spec, keep_grads=True)
    x, labels = synth.make_inputs(spec, 0)
    params = {k: v.astype(np.float64) for k, v in synth.make_params(spec, 1).items()}
    env = run(reg, x, labels, params)
    for name in params:
        assert np.allclose(env["m:" + name], env["d:" + name])        # v1 = g (v0 = 0)
        assert np.allclose(env[name], params[name] - spec["optimizer"]["lr"] * env["d:" + name])


# ---------------------------------------------------------------- transformer ops
def test_layernorm_identities_and_fd():
    X = rng.standard_normal((5, 12)) * 3 + 1
    gamma, beta = rng.standard_normal(12), rng.standard_normal(12)
    Y, mean, rstd = ops.layernorm_fwd(X, gamma, beta)
    xhat = (Y - beta) / gamma
    assert np.allclose(xhat.mean(axis=1), 0, atol=1e-12)
    assert np.allclose(mean, X.mean(axis=1)) and np.allclose(1 / rstd ** 2 - ops.LN_EPS, X.var(axis=1))
    G = rng.standard_normal(X.shape)
    dX, dg, db = ops.layernorm_bwd(X, gamma, mean, rstd, G)
    assert np.allclose(dX.sum(axis=1), 0, atol=1e-12)        # orthogonal to 1 per row
    loss = lambda: float((ops.layernorm_fwd(X, gamma, beta)[0] * G).sum())
    for arr, got in ((X, dX), (gamma, dg), (beta, db)):
        idx, g = fd_grad(loss, arr)
        assert_close(got.reshape(-1)[idx], g)


def test_gelu_closed_form_and_fd():
    from scipy.stats import norm
    X = rng.standard_normal(50) * 3
    assert_close(ops.gelu_fwd(X), X * norm.cdf(X), 1e-13)
    assert ops.gelu_fwd(np.array([0.0]))[0] == 0.0
    # lower tail: GELU(x) = x Phi(x) is tiny but not zero; elementwise relative error
    T = np.array([-6.0, -9.0, -15.0, -30.0])
    assert np.all(np.abs(ops.gelu_fwd(T) / (T * norm.cdf(T)) - 1) < 1e-12)
    assert np.all(np.abs(ops.gelu_bwd(T, np.ones(4)) / (norm.cdf(T) + T * norm.pdf(T)) - 1) < 1e-9)
    G = rng.standard_normal(50)
    idx, g = fd_grad(lambda: float((ops.gelu_fwd(X) * G).sum()), X)
    assert_close(ops.gelu_bwd(X, G)[idx], g)


def test_attention_brute_force_and_fd():
    import math
    B, T, H, dh = 2, 5, 3, 4
    d = H * dh
    qkv = rng.standard_normal((B * T, 3 * d))
    P, ctx = ops.attention_fwd(qkv, B, T, H, causal=True)
    for b in range(B):
        for h in range(H):
            for i in range(T):
                q = qkv[b * T + i, h * dh:(h + 1) * dh]
                sc = []
                for j in range(i + 1):                          # causal: keys up to i
                    k = qkv[b * T + j, d + h * dh:d + (h + 1) * dh]
                    sc.append(sum(q[u] * k[u] for u in range(dh)) / math.sqrt(dh))
                m = max(sc)
                e = [math.exp(s - m) for s in sc]
                p = [x / sum(e) for x in e]
                assert np.allclose(P[b, h, i, :i + 1], p) and np.all(P[b, h, i, i + 1:] == 0)
                out = sum(p[j] * qkv[b * T + j, 2 * d + h * dh:2 * d + (h + 1) * dh]
                          for j in range(i + 1))
                assert np.allclose(ctx[b * T + i, h * dh:(h + 1) * dh], out)
    G = rng.standard_normal(ctx.shape)
    dqkv = ops.attention_bwd(qkv, P, G, B, T, H)
    idx, g = fd_grad(lambda: float((ops.attention_fwd(qkv, B, T, H)[1] * G).sum()), qkv, n=80)
    assert_close(dqkv.reshape(-1)[idx], g)


def test_embedding_fd():
    B, T, V, d = 3, 4, 7, 5
    ids = rng.integers(0, V, (B, T))
    ids[0, 0] = ids[1, 2] = 3                                   # a repeated token
    E, pos = rng.standard_normal((V, d)), rng.standard_normal((T, d))
    X = ops.embed_fwd(ids, E, pos)
    assert np.allclose(X[1 * T + 2], E[3] + pos[2])
    G = rng.standard_normal(X.shape)
    dE, dpos = ops.embed_bwd(ids, G, V)
    loss = lambda: float((ops.embed_fwd(ids, E, pos) * G).sum())
    for arr, got in ((E, dE), (pos, dpos)):
        idx, g = fd_grad(loss, arr)
        assert_close(got.reshape(-1)[idx], g)


def test_tiny_transformer_gradients_by_finite_differences():
    spec = synth.transformer(batch=2, seq=6, d=16, heads=2, ffn=24, layers=2, vocab=11)
    reg = lower(spec, keep_grads=True)
    x, labels = synth.make_inputs(spec, 3)
    params = {k: v.astype(np.float64) for k, v in synth.make_params(spec, 4).items()}
    noise = np.random.default_rng(5)
    for k in params:
        params[k] += 0.05 * noise.standard_normal(params[k].shape)
    env = run(reg, x, labels, params)

    def loss():
        return float(run(reg, x, labels, params)["loss"][-1])

    for name, arr in params.items():
        idx, g = fd_grad(loss, arr, n=4, seed=len(name))
        got = env["d:" + name].reshape(-1)[idx]
        assert np.allclose(got, g, rtol=1e-5, atol=1e-9), name

"""Pins of ``oracle.sampled`` (per-output evaluations used at full size) against the
whole-layer definitions of ``oracle.ops`` on small shapes, and of the tolerance the
full-size GPU checks apply."""

import numpy as np
import pytest

from oracle import ops, sampled

rng = np.random.default_rng(5)


def every_index(shape):
    return [a.reshape(-1) for a in np.indices(shape)]


CONVS = [(2, 9, 7, 5, 6, 3, 1, 1), (2, 10, 9, 3, 4, 7, 2, 3), (1, 8, 8, 4, 5, 3, 2, 1),
         (3, 5, 6, 8, 3, 1, 1, 0), (1, 7, 7, 2, 2, 1, 2, 0)]


@pytest.mark.parametrize("shape", CONVS, ids=lambda s: "x".join(map(str, s)))
def test_conv_elements_match_whole_layer(shape):
    N, H, W, C, K, k, st, pd = shape
    X = rng.standard_normal((N, H, W, C)).astype(np.float32)
    Wt = rng.standard_normal((K, k, k, C)).astype(np.float32)
    Y = ops.conv_fwd(X.astype(np.float64), Wt.astype(np.float64), st, pd)
    Ya = ops.conv_fwd(np.abs(X).astype(np.float64), np.abs(Wt).astype(np.float64), st, pd)
    P, Q = Y.shape[1:3]
    val, mag, terms = sampled.conv_fwd_at(X, Wt, st, pd, *every_index(Y.shape))
    assert terms == k * k * C
    np.testing.assert_allclose(val, Y.reshape(-1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mag, Ya.reshape(-1), rtol=1e-12, atol=1e-12)

    G = rng.standard_normal((N, P, Q, K)).astype(np.float32)
    dX = ops.conv_bwd_x(Wt.astype(np.float64), G.astype(np.float64), X.shape, st, pd)
    dXa = ops.conv_bwd_x(np.abs(Wt).astype(np.float64), np.abs(G).astype(np.float64), X.shape,
                         st, pd)
    val, mag, terms = sampled.conv_bwd_x_at(Wt, G, st, pd, *every_index(X.shape))
    np.testing.assert_allclose(val, dX.reshape(-1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mag, dXa.reshape(-1), rtol=1e-12, atol=1e-12)

    dW = ops.conv_bwd_w(X.astype(np.float64), G.astype(np.float64), Wt.shape, st, pd)
    dWa = ops.conv_bwd_w(np.abs(X).astype(np.float64), np.abs(G).astype(np.float64), Wt.shape,
                         st, pd)
    ks, cs = [K - 1, 0], list(range(C))[::-1]
    taps = [(r, s) for r in range(k) for s in range(k)][::2]
    val, mag, terms = sampled.conv_bwd_w_at(X, G, st, pd, k, k, ks, cs, taps, batch_block=1)
    assert terms == N * P * Q
    for t, (r, s) in enumerate(taps):
        np.testing.assert_allclose(val[t], dW[ks][:, r, s, :][:, cs], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(mag[t], dWa[ks][:, r, s, :][:, cs], rtol=1e-12, atol=1e-12)


def test_dense_elements_match_whole_layer():
    M, K, N = 37, 19, 11
    X = rng.standard_normal((M, K)).astype(np.float32)
    Wt = rng.standard_normal((N, K)).astype(np.float32)
    b = rng.standard_normal(N).astype(np.float32)
    G = rng.standard_normal((M, N)).astype(np.float32)
    d = lambda a: a.astype(np.float64)                      # noqa: E731
    m, j = every_index((M, N))
    val, mag, terms = sampled.linear_fwd_at(X, Wt, b, m, j)
    np.testing.assert_allclose(val, ops.linear_fwd(d(X), d(Wt), d(b)).reshape(-1), rtol=1e-12)
    np.testing.assert_allclose(mag, (np.abs(d(X)) @ np.abs(d(Wt)).T + np.abs(d(b))).reshape(-1),
                               rtol=1e-12)
    m, i = every_index((M, K))
    val, mag, _ = sampled.linear_bwd_x_at(Wt, G, m, i)
    np.testing.assert_allclose(val, ops.linear_bwd_x(d(Wt), d(G)).reshape(-1), rtol=1e-12)
    dW, db = ops.linear_bwd_w(d(X), d(G))
    (w, wm), (bb, bm), terms = sampled.linear_bwd_w_at(X, G, [3, 0, 10], [18, 2], row_block=5)
    assert terms == M
    np.testing.assert_allclose(w, dW[[3, 0, 10]][:, [18, 2]], rtol=1e-12)
    np.testing.assert_allclose(bb, db[[3, 0, 10]], rtol=1e-12)
    np.testing.assert_allclose(bm, np.abs(d(G)).sum(axis=0)[[3, 0, 10]], rtol=1e-12)


def test_batchnorm_elements_match_whole_layer():
    X = (rng.standard_normal((3, 5, 4, 6)) * 2 + 1).astype(np.float32)
    G = rng.standard_normal(X.shape).astype(np.float32)
    gamma = rng.standard_normal(6).astype(np.float32)
    beta = rng.standard_normal(6).astype(np.float32)
    Y, mean, invstd = ops.bn_fwd(X.astype(np.float64), gamma.astype(np.float64),
                                 beta.astype(np.float64))
    X2, G2 = X.reshape(-1, 6), G.reshape(-1, 6)
    m2, r2, absmean = sampled.bn_stats(X2, row_block=7)
    np.testing.assert_allclose(m2, mean, rtol=1e-12)
    np.testing.assert_allclose(r2, invstd, rtol=1e-12)
    np.testing.assert_allclose(absmean, np.abs(X2.astype(np.float64)).mean(axis=0), rtol=1e-12)
    row, c = every_index(X2.shape)
    np.testing.assert_allclose(sampled.bn_fwd_at(X2, gamma, beta, mean, invstd, row, c),
                               Y.reshape(-1), rtol=1e-12, atol=1e-12)
    dX, dg, db = ops.bn_bwd(X.astype(np.float64), gamma.astype(np.float64), mean, invstd,
                            G.astype(np.float64))
    b2, g2, _, _ = sampled.bn_bwd_sums(X2, G2, mean, invstd, row_block=7)
    np.testing.assert_allclose(b2, db, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(g2, dg, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sampled.bn_bwd_at(X2, G2, gamma, mean, invstd, b2, g2, row, c),
                               dX.reshape(-1), rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("k,st,pd", [(3, 2, 1), (2, 2, 0), (3, 1, 1)])
def test_maxpool_elements_match_whole_layer(k, st, pd):
    X = rng.standard_normal((2, 9, 8, 3)).astype(np.float32)
    X[0, 2, 2, 1] = X[0, 2, 3, 1] = X[0, 3, 2, 1] = 9.0          # ties: the first tap wins
    Y, idx = ops.maxpool_fwd(X, k, st, pd)
    v, i = sampled.maxpool_fwd_at(X, k, st, pd, *every_index(Y.shape))
    assert np.array_equal(v, Y.reshape(-1).astype(np.float64))
    assert np.array_equal(i, idx.reshape(-1))
    G = rng.standard_normal(Y.shape).astype(np.float32)
    dX = ops.maxpool_bwd(idx, G.astype(np.float64), X.shape, k, st, pd)
    val, _ = sampled.maxpool_bwd_at(idx, G, k, st, pd, *every_index(X.shape))
    np.testing.assert_allclose(val, dX.reshape(-1), rtol=1e-12, atol=0)


def test_tolerance_separates_rounding_from_dropped_terms():
    """The full-size checks accept |gpu - ref| <= sqrt(T) u mag + 4 u |ref| (u = 2^-24, T
    terms, mag = sum of |terms|).  A float32 evaluation in one running sum, the least accurate
    common order, meets it both for terms of random sign and for terms of one sign (where the
    running sum grows and its rounding errors with it).  A block of T / 64 terms left out (a
    lost split-K slice, tile row or tap) fails it at every T; a single term left out fails it
    for the sums of up to 4608 terms (a convolution's R S C), where one term is larger than
    the bound."""
    u = 2.0 ** -24
    for T in (27, 576, 4608, 200_704):
        for positive in (False, True):
            a = rng.standard_normal((64, T)).astype(np.float32)
            b = rng.standard_normal((64, T)).astype(np.float32)
            if positive:
                a, b = np.abs(a), np.abs(b)
            terms = a.astype(np.float64) * b.astype(np.float64)
            ref, mag = terms.sum(axis=1), np.abs(terms).sum(axis=1)
            seq = np.zeros(64, np.float32)
            for t in range(T):
                seq = seq + a[:, t] * b[:, t]
            bound = np.sqrt(T) * u * mag + 4 * u * np.abs(ref)
            assert np.all(np.abs(seq - ref) <= bound), (T, positive)
            block = ref - terms[:, :max(1, T // 64)].sum(axis=1)
            assert np.mean(np.abs(block - ref) > bound) > 0.9, (T, positive)
            if T <= 4608:
                one = ref - terms[:, T // 3]
                assert np.mean(np.abs(one - ref) > bound) > 0.9, (T, positive)

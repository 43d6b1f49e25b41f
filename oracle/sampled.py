"""Single outputs of the layer definitions, for checks at full size (test infrastructure).

At the full batch sizes a whole layer is too large to recompute on the CPU in
float64, but each output element is one defining sum that the oracle can
evaluate on its own.  These functions take arrays of output coordinates and
return, per coordinate, the value of that sum in float64 together with its
magnitude, the sum of the absolute values of its terms.  The magnitude is what
bounds the rounding error of any float32 evaluation of the same sum, whatever
its order; the caller's tolerance is stated in units of it.

The formulas are those of ``oracle.ops`` (the module docstring there lists
them), written per element:

* conv forward:   Y[n,p,q,k] = sum_{r,s,c} X[n, p st + r - pad, q st + s - pad, c] W[k,r,s,c]
                  over the taps inside the image (zero padding contributes nothing);
* conv input gradient: dX[n,h,w,c] = sum over taps (r, s) and channels k of
                  dY[n,p,q,k] W[k,r,s,c] for the outputs (p, q) with
                  p st + r - pad = h and q st + s - pad = w;
* conv filter gradient: dW[k,r,s,c] = sum_{n,p,q} dY[n,p,q,k] X[n, p st + r - pad, q st + s - pad, c];
* dense:          Y = X W^T + b, dX = dY W, dW = dY^T X, db = column sums of dY;
* BatchNorm:      per-channel batch mean and biased variance; y = gamma (x - mean) invstd + beta;
                  dX = gamma invstd (dY - mean(dY) - xhat mean(dY xhat)), with the statistics
                  of the forward as given;
* max pool:       the first maximal valid tap in row-major window order; the input gradient
                  of a pixel sums dY over the windows whose chosen tap it is.

Every evaluation here is pinned against the whole-layer functions of
``oracle.ops`` on small shapes (``tests/test_oracle_sampled.py``).
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F64 = np.float64
WORKERS = min(16, os.cpu_count() or 1)


def _block_sum(fn, starts):
    """sum of fn(start) over the blocks, evaluated on a thread pool (NumPy releases the
    interpreter lock inside its array operations) and added in block order."""
    with ThreadPoolExecutor(WORKERS) as ex:
        parts = list(ex.map(fn, starts))
    total = parts[0]
    for p in parts[1:]:
        total = tuple(a + b for a, b in zip(total, p))
    return total


def _i(a):
    return np.asarray(a, dtype=np.int64)


# ---------------------------------------------------------------- conv
def conv_fwd_at(X, Wt, stride, pad, n, p, q, k):
    """(values, magnitudes, terms) of Y[n, p, q, k]; terms = R S C."""
    n, p, q, k = map(_i, (n, p, q, k))
    _, H, Wd, C = X.shape
    K, R, S, _ = Wt.shape
    val = np.zeros(n.size, F64)
    mag = np.zeros(n.size, F64)
    for r in range(R):
        h = p * stride + r - pad
        for s in range(S):
            w = q * stride + s - pad
            ok = (h >= 0) & (h < H) & (w >= 0) & (w < Wd)
            prod = X[n[ok], h[ok], w[ok], :].astype(F64) * Wt[k[ok], r, s, :].astype(F64)
            val[ok] += prod.sum(axis=1)
            mag[ok] += np.abs(prod).sum(axis=1)
    return val, mag, R * S * C


def conv_bwd_x_at(Wt, dY, stride, pad, n, h, w, c):
    """(values, magnitudes, terms) of dX[n, h, w, c]; terms = K R S (the most any pixel has)."""
    n, h, w, c = map(_i, (n, h, w, c))
    _, P, Q, K = dY.shape
    _, R, S, _ = Wt.shape
    val = np.zeros(n.size, F64)
    mag = np.zeros(n.size, F64)
    for r in range(R):
        hp = h + pad - r                      # = p * stride when output row p uses tap r
        p = hp // stride
        for s in range(S):
            wq = w + pad - s
            q = wq // stride
            ok = (hp >= 0) & (hp % stride == 0) & (p < P) & (wq >= 0) & (wq % stride == 0) & (q < Q)
            prod = dY[n[ok], p[ok], q[ok], :].astype(F64) * Wt[:, r, s, :][:, c[ok]].T.astype(F64)
            val[ok] += prod.sum(axis=1)
            mag[ok] += np.abs(prod).sum(axis=1)
    return val, mag, K * R * S


def conv_bwd_w_at(X, dY, stride, pad, R, S, ks, cs, taps, batch_block=16):
    """(values, magnitudes, terms) of dW[k, r, s, c] for every k in ``ks``, c in ``cs`` and
    (r, s) in ``taps``, as arrays [len(taps), len(ks), len(cs)]; terms = N P Q.  The sum over
    the batch runs in blocks of ``batch_block`` images (float64 throughout)."""
    N, H, Wd, C = X.shape
    _, P, Q, K = dY.shape
    ks, cs = _i(ks), _i(cs)

    def block(n0):
        n1 = min(N, n0 + batch_block)
        val = np.zeros((len(taps), ks.size, cs.size), F64)
        mag = np.zeros_like(val)
        g = dY[n0:n1][..., ks].astype(F64).reshape(-1, ks.size)          # [b P Q, |ks|]
        ga = np.abs(g)
        xp = np.zeros((n1 - n0, H + 2 * pad, Wd + 2 * pad, cs.size), F64)
        xp[:, pad:pad + H, pad:pad + Wd, :] = X[n0:n1][..., cs]
        for t, (r, s) in enumerate(taps):
            tap = xp[:, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride, :]
            tap = tap.reshape(-1, cs.size)
            val[t] = g.T @ tap
            mag[t] = ga.T @ np.abs(tap)
        return val, mag

    val, mag = _block_sum(block, range(0, N, batch_block))
    return val, mag, N * P * Q


# ---------------------------------------------------------------- dense
def linear_fwd_at(X, Wt, b, m, j):
    """(values, magnitudes, terms) of Y[m, j] = sum_i X[m, i] W[j, i] + b[j]; terms = K + 1."""
    m, j = _i(m), _i(j)
    prod = X[m, :].astype(F64) * Wt[j, :].astype(F64)
    bias = b[j].astype(F64)
    return prod.sum(axis=1) + bias, np.abs(prod).sum(axis=1) + np.abs(bias), X.shape[1] + 1


def linear_bwd_x_at(Wt, dY, m, i):
    """(values, magnitudes, terms) of dX[m, i] = sum_j dY[m, j] W[j, i]; terms = N."""
    m, i = _i(m), _i(i)
    prod = dY[m, :].astype(F64) * Wt[:, i].T.astype(F64)
    return prod.sum(axis=1), np.abs(prod).sum(axis=1), dY.shape[1]


def linear_bwd_w_at(X, dY, js, cols, row_block=1 << 14):
    """dW[j, i] for j in ``js`` and i in ``cols`` ([|js|, |cols|]) and db[j] for j in ``js``,
    each as (values, magnitudes); terms = M (the rows)."""
    js, cols = _i(js), _i(cols)

    def block(m0):
        g = dY[m0:m0 + row_block][:, js].astype(F64)
        x = X[m0:m0 + row_block][:, cols].astype(F64)
        return g.T @ x, np.abs(g).T @ np.abs(x), g.sum(axis=0), np.abs(g).sum(axis=0)

    dw, dwm, db, dbm = _block_sum(block, range(0, X.shape[0], row_block))
    return (dw, dwm), (db, dbm), X.shape[0]


# ---------------------------------------------------------------- BatchNorm
def bn_stats(X2, row_block=1 << 18):
    """Per-channel statistics of [rows, C]: (mean, invstd, mean of |x|), in float64."""
    rows, C = X2.shape
    starts = range(0, rows, row_block)

    def sums(r0):
        x = X2[r0:r0 + row_block].astype(F64)
        return x.sum(axis=0), np.abs(x).sum(axis=0)

    s, sa = _block_sum(sums, starts)
    mean = s / rows

    def squares(r0):
        d = X2[r0:r0 + row_block].astype(F64) - mean
        return ((d * d).sum(axis=0),)

    (ss,) = _block_sum(squares, starts)
    return mean, 1.0 / np.sqrt(ss / rows + 1e-5), sa / rows


def bn_fwd_at(X2, gamma, beta, mean, invstd, row, c):
    """y[row, c] = gamma (x - mean) invstd + beta with the statistics given."""
    row, c = _i(row), _i(c)
    xhat = (X2[row, c].astype(F64) - mean[c]) * invstd[c]
    return gamma[c].astype(F64) * xhat + beta[c].astype(F64)


def bn_bwd_sums(X2, dY2, mean, invstd, row_block=1 << 18):
    """(dbeta, dgamma, |dbeta| magnitude, |dgamma| magnitude) per channel: the sums of dY and
    of dY xhat over the rows, xhat from the statistics given."""
    rows, C = X2.shape

    def sums(r0):
        g = dY2[r0:r0 + row_block].astype(F64)
        gx = g * ((X2[r0:r0 + row_block].astype(F64) - mean) * invstd)
        return g.sum(axis=0), gx.sum(axis=0), np.abs(g).sum(axis=0), np.abs(gx).sum(axis=0)

    return _block_sum(sums, range(0, rows, row_block))


def bn_bwd_at(X2, dY2, gamma, mean, invstd, dbeta, dgamma, row, c):
    """dX[row, c] = gamma invstd / m (m dY - dbeta - xhat dgamma), m = rows."""
    row, c = _i(row), _i(c)
    m = X2.shape[0]
    xhat = (X2[row, c].astype(F64) - mean[c]) * invstd[c]
    return gamma[c].astype(F64) * invstd[c] / m * (m * dY2[row, c].astype(F64) - dbeta[c]
                                                   - xhat * dgamma[c])


# ---------------------------------------------------------------- max pool
def maxpool_fwd_at(X, k, stride, pad, n, p, q, c):
    """(max, index r k + s of its first maximal valid tap) at output [n, p, q, c]."""
    n, p, q, c = map(_i, (n, p, q, c))
    _, H, Wd, _ = X.shape
    best = np.full(n.size, -np.inf)
    idx = np.zeros(n.size, np.int64)
    for r in range(k):
        h = p * stride + r - pad
        for s in range(k):
            w = q * stride + s - pad
            ok = (h >= 0) & (h < H) & (w >= 0) & (w < Wd)
            v = np.full(n.size, -np.inf)
            v[ok] = X[n[ok], h[ok], w[ok], c[ok]]
            better = v > best
            best = np.where(better, v, best)
            idx = np.where(better, r * k + s, idx)
    return best, idx


def maxpool_bwd_at(idx, dY, k, stride, pad, n, h, w, c):
    """(values, terms) of dX[n, h, w, c]: dY summed over the windows (p, q) that contain the
    pixel and chose it (idx[n, p, q, c] = (h - p st + pad) k + (w - q st + pad))."""
    n, h, w, c = map(_i, (n, h, w, c))
    _, P, Q, _ = dY.shape
    val = np.zeros(n.size, F64)
    for r in range(k):
        hp = h + pad - r
        p = hp // stride
        for s in range(k):
            wq = w + pad - s
            q = wq // stride
            ok = (hp >= 0) & (hp % stride == 0) & (p < P) & (wq >= 0) & (wq % stride == 0) & (q < Q)
            hit = np.zeros(n.size, bool)
            hit[ok] = idx[n[ok], p[ok], q[ok], c[ok]] == r * k + s
            val[hit] += dY[n[hit], p[hit], q[hit], c[hit]]
    return val, k * k

"""Textbook forward, backward and SGD of every layer kind, in NumPy (test infrastructure).

The paper trains ordinary networks (ResNet-50 and others, Section 5); it
fixes none of these formulas, so each is the standard definition, computed in
the dtype of its inputs (float64 for parity).  Layouts follow the library
boundary: images NHWC, conv weights [K, R, S, C], dense weights [out, in].

* dense:        Y = X W^T + b
* conv:         cross-correlation with zero padding,
                Y[n,p,q,k] = sum_{r,s,c} Xpad[n, p*st + r, q*st + s, c] W[k,r,s,c]
* BatchNorm:    training mode, batch mean and biased variance over N, H, W,
                eps = 1e-5, y = gamma * (x - mean) / sqrt(var + eps) + beta
* ReLU:         y = max(x, 0); backward through the output: dx = dy * [y > 0]
* max pool:     window max over valid taps; ties go to the first tap in
                row-major window order; backward routes dy to that tap
* global average pool over H, W
* softmax cross-entropy, mean over the batch
* SGD:          w -= lr g;  with momentum mu: v = mu v + g, w -= lr v
* LayerNorm:    per row over the features, biased variance, eps = 1e-5
* GELU:         exact, x Phi(x) with the normal CDF Phi
* attention:    per batch and head, P = softmax(q k^T / sqrt(dh)) with future
                positions masked (causal), context = P v; q, k, v are the
                column thirds of one [rows, 3 d] projection, head h owning
                columns h dh .. (h + 1) dh of each third
* embedding:    x[b, t] = E[id[b, t]] + pos[t]
* concat:       channel (last axis) concatenation; its backward hands each input
                its own channel range of the output gradient
* upsample:     nearest, factor 2: y[n, 2h + i, 2w + j] = x[n, h, w]; backward sums
                each 2 x 2 block of the output gradient
"""

from __future__ import annotations

import numpy as np
from scipy.special import erfc

BN_EPS = 1e-5
LN_EPS = 1e-5


# ---------------------------------------------------------------- dense
def linear_fwd(X, W, b):
    return X @ W.T + b


def linear_bwd_w(X, dY):
    """dW = dY^T X, db = sum_n dY."""
    return dY.T @ X, dY.sum(axis=0)


def linear_bwd_x(W, dY):
    """dX = dY W."""
    return dY @ W


# ---------------------------------------------------------------- conv
def _out_size(h, k, stride, pad):
    return (h + 2 * pad - k) // stride + 1


def conv_fwd(X, Wt, stride, pad):
    N, H, Wd, C = X.shape
    K, R, S, C2 = Wt.shape
    assert C == C2
    P, Q = _out_size(H, R, stride, pad), _out_size(Wd, S, stride, pad)
    Xp = np.pad(X, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    Y = np.zeros((N, P, Q, K), dtype=X.dtype)
    for r in range(R):
        for s in range(S):
            tap = Xp[:, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride, :]
            Y += tap @ Wt[:, r, s, :].T
    return Y


def conv_bwd_x(Wt, dY, x_shape, stride, pad):
    """dX: every output gradient is sent back through the tap that produced it."""
    N, H, Wd, C = x_shape
    K, R, S, _ = Wt.shape
    _, P, Q, _ = dY.shape
    dXp = np.zeros((N, H + 2 * pad, Wd + 2 * pad, C), dtype=dY.dtype)
    for r in range(R):
        for s in range(S):
            dXp[:, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride, :] += \
                dY @ Wt[:, r, s, :]
    return dXp[:, pad:pad + H, pad:pad + Wd, :]


def conv_bwd_w(X, dY, w_shape, stride, pad):
    """dW[k,r,s,c] = sum_{n,p,q} dY[n,p,q,k] Xpad[n, p*st + r, q*st + s, c]."""
    K, R, S, C = w_shape
    _, P, Q, _ = dY.shape
    Xp = np.pad(X, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    dW = np.zeros(w_shape, dtype=dY.dtype)
    for r in range(R):
        for s in range(S):
            tap = Xp[:, r:r + stride * (P - 1) + 1:stride, s:s + stride * (Q - 1) + 1:stride, :]
            dW[:, r, s, :] = np.tensordot(dY, tap, axes=([0, 1, 2], [0, 1, 2]))
    return dW


# ---------------------------------------------------------------- BatchNorm
def bn_fwd(X, gamma, beta):
    """Returns (Y, mean, invstd); statistics over every axis but the channel (last) one."""
    axes = tuple(range(X.ndim - 1))
    mean = X.mean(axis=axes)
    var = ((X - mean) ** 2).mean(axis=axes)
    invstd = 1.0 / np.sqrt(var + BN_EPS)
    xhat = (X - mean) * invstd
    return gamma * xhat + beta, mean, invstd


def bn_bwd(X, gamma, mean, invstd, dY):
    """Returns (dX, dgamma, dbeta) of the training-mode normalisation."""
    axes = tuple(range(X.ndim - 1))
    m = X.size // X.shape[-1]
    xhat = (X - mean) * invstd
    dbeta = dY.sum(axis=axes)
    dgamma = (dY * xhat).sum(axis=axes)
    dX = gamma * invstd / m * (m * dY - dbeta - xhat * dgamma)
    return dX, dgamma, dbeta


# ---------------------------------------------------------------- ReLU
def relu_fwd(X):
    return np.maximum(X, 0)


def relu_bwd(Y, dY):
    return dY * (Y > 0)


# ---------------------------------------------------------------- pooling
def maxpool_fwd(X, k, stride, pad):
    """Returns (Y, idx): idx = r*k + s of the first maximal valid tap (uint8)."""
    N, H, Wd, C = X.shape
    P, Q = _out_size(H, k, stride, pad), _out_size(Wd, k, stride, pad)
    Y = np.full((N, P, Q, C), -np.inf, dtype=X.dtype)
    idx = np.zeros((N, P, Q, C), dtype=np.uint8)
    for p in range(P):
        for q in range(Q):
            for r in range(k):
                for s in range(k):
                    h, w = p * stride + r - pad, q * stride + s - pad
                    if 0 <= h < H and 0 <= w < Wd:
                        v = X[:, h, w, :]
                        better = v > Y[:, p, q, :]
                        Y[:, p, q, :] = np.where(better, v, Y[:, p, q, :])
                        idx[:, p, q, :] = np.where(better, r * k + s, idx[:, p, q, :])
    return Y, idx


def maxpool_bwd(idx, dY, x_shape, k, stride, pad):
    N, H, Wd, C = x_shape
    _, P, Q, _ = dY.shape
    dX = np.zeros(x_shape, dtype=dY.dtype)
    for p in range(P):
        for q in range(Q):
            for r in range(k):
                for s in range(k):
                    h, w = p * stride + r - pad, q * stride + s - pad
                    if 0 <= h < H and 0 <= w < Wd:
                        dX[:, h, w, :] += np.where(idx[:, p, q, :] == r * k + s, dY[:, p, q, :], 0)
    return dX


def avgpool_fwd(X):
    return X.mean(axis=(1, 2))


def avgpool_bwd(dY, x_shape):
    N, H, Wd, C = x_shape
    return np.broadcast_to(dY[:, None, None, :] / (H * Wd), x_shape).copy()


# ---------------------------------------------------------------- loss
def softmax_ce(logits, labels):
    """Returns (per-row losses, mean loss, dlogits) of the mean softmax cross-entropy."""
    N = logits.shape[0]
    z = logits - logits.max(axis=1, keepdims=True)
    lse = np.log(np.exp(z).sum(axis=1))
    rows = lse - z[np.arange(N), labels]
    prob = np.exp(z - lse[:, None])
    onehot = np.zeros_like(prob)
    onehot[np.arange(N), labels] = 1.0
    return rows, rows.mean(), (prob - onehot) / N


# ---------------------------------------------------------------- update
def sgd(w, g, lr):
    return w - lr * g


def sgd_momentum(w, g, v, lr, mu):
    v_new = mu * v + g
    return w - lr * v_new, v_new


# ---------------------------------------------------------------- LayerNorm
def layernorm_fwd(X, gamma, beta):
    """Returns (Y, mean, rstd) over the last axis."""
    mean = X.mean(axis=-1, keepdims=True)
    var = ((X - mean) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + LN_EPS)
    return (X - mean) * rstd * gamma + beta, mean[..., 0], rstd[..., 0]


def layernorm_bwd(X, gamma, mean, rstd, dY):
    """Returns (dX, dgamma, dbeta)."""
    xhat = (X - mean[..., None]) * rstd[..., None]
    g = dY * gamma
    dX = rstd[..., None] * (g - g.mean(axis=-1, keepdims=True)
                            - xhat * (g * xhat).mean(axis=-1, keepdims=True))
    return dX, (dY * xhat).sum(axis=0), dY.sum(axis=0)


# ---------------------------------------------------------------- GELU
def _normal_cdf(X):
    """Phi(x) = erfc(-x / sqrt 2) / 2; the erfc form keeps full relative precision in the
    lower tail, where 1 + erf(x / sqrt 2) cancels."""
    return 0.5 * erfc(-X / np.sqrt(2.0))


def gelu_fwd(X):
    return X * _normal_cdf(X)


def gelu_bwd(X, dY):
    cdf = _normal_cdf(X)
    pdf = np.exp(-0.5 * X * X) / np.sqrt(2.0 * np.pi)
    return dY * (cdf + X * pdf)


# ---------------------------------------------------------------- attention
def _heads(qkv, B, T, H):
    """Split [B T, 3 d] into q, k, v of shape [B, H, T, dh]."""
    d = qkv.shape[1] // 3
    dh = d // H
    t = qkv.reshape(B, T, 3, H, dh)
    return t[:, :, 0].transpose(0, 2, 1, 3), t[:, :, 1].transpose(0, 2, 1, 3), \
        t[:, :, 2].transpose(0, 2, 1, 3)


def attention_fwd(qkv, B, T, H, causal=True):
    """Returns (P [B, H, T, T], context [B T, d])."""
    q, k, v = _heads(qkv, B, T, H)
    dh = q.shape[-1]
    S = q @ k.transpose(0, 1, 3, 2) / np.sqrt(dh)
    if causal:
        S = np.where(np.tril(np.ones((T, T), dtype=bool)), S, -np.inf)
    S = S - S.max(axis=-1, keepdims=True)
    P = np.exp(S)
    P /= P.sum(axis=-1, keepdims=True)
    ctx = P @ v                                    # [B, H, T, dh]
    return P, ctx.transpose(0, 2, 1, 3).reshape(B * T, H * dh)


def attention_bwd(qkv, P, dctx, B, T, H):
    """Returns dqkv [B T, 3 d] for context = softmax(q k^T / sqrt(dh)) v."""
    q, k, v = _heads(qkv, B, T, H)
    dh = q.shape[-1]
    dO = dctx.reshape(B, T, H, dh).transpose(0, 2, 1, 3)
    dv = P.transpose(0, 1, 3, 2) @ dO
    dP = dO @ v.transpose(0, 1, 3, 2)
    dS = P * (dP - (dP * P).sum(axis=-1, keepdims=True)) / np.sqrt(dh)
    dq = dS @ k
    dk = dS.transpose(0, 1, 3, 2) @ q
    out = np.stack([dq, dk, dv], axis=2)           # [B, H, 3, T, dh]
    return out.transpose(0, 3, 2, 1, 4).reshape(B * T, 3 * H * dh)


# ---------------------------------------------------------------- embedding
def embed_fwd(ids, E, pos):
    B, T = ids.shape
    return (E[ids] + pos[None, :T]).reshape(B * T, E.shape[1])


def concat_fwd(Xs):
    return np.concatenate(Xs, axis=-1)


def concat_bwd(dY, channels):
    edges = np.cumsum([0] + list(channels))
    return [dY[..., edges[j]:edges[j + 1]].copy() for j in range(len(channels))]


def upsample_fwd(X):
    return X.repeat(2, axis=1).repeat(2, axis=2)


def upsample_bwd(dY):
    N, H2, W2, C = dY.shape
    return dY.reshape(N, H2 // 2, 2, W2 // 2, 2, C).sum(axis=(2, 4))


def embed_bwd(ids, dX, vocab):
    B, T = ids.shape
    d = dX.shape[1]
    dE = np.zeros((vocab, d), dtype=dX.dtype)
    np.add.at(dE, ids.reshape(-1), dX)
    return dE, dX.reshape(B, T, d).sum(axis=0)

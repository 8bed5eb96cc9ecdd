"""Layer forward functions and their vector-Jacobian products in fp64 numpy.

TEST INFRASTRUCTURE ONLY (the CPU oracle; see oracle/__init__.py).

The paper runs stock framework layers (Sec. IV-A, IV-C) and defines none of
them; each function below is the textbook definition written out.  Layouts:
activations NHWC (or [n, C]), conv weights [K, R, S, C], linear weights
[out, in].  Convolutions are stride 1 with zero padding k//2 (cross-
correlation).  ReLU'(0) = 0.  Max pooling sends the gradient to the first
maximum in row-major window order.  3x3 average pooling counts the zero
padding (divides by 9).  Batch normalisation uses the batch mean and the
biased batch variance of the micro-batch, eps 1e-5.
"""
from __future__ import annotations

import numpy as np

BN_EPS = 1e-5


def _shifted(xp, r, s, H, W):
    """The H x W window of padded input xp starting at (r, s), as [n*H*W, C]."""
    return np.ascontiguousarray(xp[:, r:r + H, s:s + W, :]).reshape(-1, xp.shape[3])


# ---------------------------------------------------------------- conv / linear
def conv2d(x, w, b=None):
    """y[n,h,w,k] = sum_{r,s,c} x[n, h+r-p, w+s-p, c] * w[k,r,s,c] (+ b[k])."""
    n, H, W, C = x.shape
    K, R, S, _ = w.shape
    p = R // 2
    xp = np.pad(x, ((0, 0), (p, p), (p, p), (0, 0)))
    y = np.zeros((n * H * W, K))
    for r in range(R):
        for s in range(S):
            y += _shifted(xp, r, s, H, W) @ w[:, r, s, :].T
    if b is not None:
        y += b
    return y.reshape(n, H, W, K)


def conv2d_vjp(x, w, dy, need_dx=True, has_bias=False):
    """Gradients of conv2d w.r.t. x, w and b for cotangent dy."""
    n, H, W, C = x.shape
    K, R, S, _ = w.shape
    p = R // 2
    xp = np.pad(x, ((0, 0), (p, p), (p, p), (0, 0)))
    dy2 = dy.reshape(-1, K)
    dw = np.zeros_like(w)
    dxp = np.zeros_like(xp) if need_dx else None
    for r in range(R):
        for s in range(S):
            dw[:, r, s, :] = dy2.T @ _shifted(xp, r, s, H, W)
            if need_dx:
                dxp[:, r:r + H, s:s + W, :] += (dy2 @ w[:, r, s, :]).reshape(n, H, W, C)
    db = dy2.sum(axis=0) if has_bias else None
    dx = dxp[:, p:p + H, p:p + W, :] if need_dx else None
    return dx, dw, db


def linear(x, w, b=None):
    """y = x w^T (+ b)."""
    y = x @ w.T
    if b is not None:
        y = y + b
    return y


def linear_vjp(x, w, dy, need_dx=True, has_bias=False):
    dx = dy @ w if need_dx else None
    dw = dy.T @ x
    db = dy.sum(axis=0) if has_bias else None
    return dx, dw, db


# ---------------------------------------------------------------- activations
def relu(x):
    return np.maximum(x, 0.0)


def relu_vjp(x, dy):
    """ReLU'(x) = 1 for x > 0, else 0 (x is the ReLU input or its output)."""
    return dy * (x > 0)


# ---------------------------------------------------------------- batch norm
def batchnorm(z, gamma, beta, eps=BN_EPS):
    """Training-mode batch normalisation over all axes but the channel axis.
    Returns (y, xhat, rstd)."""
    axes = tuple(range(z.ndim - 1))
    mu = z.mean(axis=axes)
    var = ((z - mu) ** 2).mean(axis=axes)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mu) * rstd
    return gamma * xhat + beta, xhat, rstd


def batchnorm_vjp(xhat, rstd, gamma, dy):
    """VJP of batchnorm: with M the reduced count, dbeta = sum dy,
    dgamma = sum dy*xhat, dz = gamma*rstd*(dy - dbeta/M - xhat*dgamma/M)."""
    axes = tuple(range(dy.ndim - 1))
    M = dy.size // dy.shape[-1]
    dbeta = dy.sum(axis=axes)
    dgamma = (dy * xhat).sum(axis=axes)
    dz = gamma * rstd * (dy - dbeta / M - xhat * dgamma / M)
    return dz, dgamma, dbeta


# ---------------------------------------------------------------- pooling
def _windows2(x):
    """[n,H,W,C] -> [n,H/2,W/2,4,C], window elements in row-major order."""
    n, H, W, C = x.shape
    Ho, Wo = H // 2, W // 2
    x = x[:, :2 * Ho, :2 * Wo, :]
    return x.reshape(n, Ho, 2, Wo, 2, C).transpose(0, 1, 3, 2, 4, 5).reshape(n, Ho, Wo, 4, C)


def maxpool2(x):
    """2x2 max pooling, stride 2.  Returns (y, argmax index 0..3 per output)."""
    win = _windows2(x)
    idx = np.argmax(win, axis=3)  # first maximum in row-major window order
    y = np.take_along_axis(win, idx[:, :, :, None, :], axis=3)[:, :, :, 0, :]
    return y, idx


def maxpool2_vjp(x_shape, idx, dy):
    n, H, W, C = x_shape
    Ho, Wo = H // 2, W // 2
    win = np.zeros((n, Ho, Wo, 4, C))
    np.put_along_axis(win, idx[:, :, :, None, :], dy[:, :, :, None, :], axis=3)
    dx = np.zeros((n, H, W, C))
    dx[:, :2 * Ho, :2 * Wo, :] = (win.reshape(n, Ho, Wo, 2, 2, C)
                                  .transpose(0, 1, 3, 2, 4, 5).reshape(n, 2 * Ho, 2 * Wo, C))
    return dx


def avgpool3(x):
    """3x3 average pooling, stride 1, zero padding 1, divisor always 9."""
    n, H, W, C = x.shape
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    y = np.zeros_like(x)
    for r in range(3):
        for s in range(3):
            y += xp[:, r:r + H, s:s + W, :]
    return y / 9.0


def avgpool3_vjp(dy):
    n, H, W, C = dy.shape
    dxp = np.zeros((n, H + 2, W + 2, C))
    for r in range(3):
        for s in range(3):
            dxp[:, r:r + H, s:s + W, :] += dy / 9.0
    return dxp[:, 1:H + 1, 1:W + 1, :]


def gap(x):
    """Global average pool over H, W: [n,H,W,C] -> [n,C]."""
    return x.mean(axis=(1, 2))


def gap_vjp(x_shape, dy):
    n, H, W, C = x_shape
    return np.broadcast_to(dy[:, None, None, :] / (H * W), x_shape).copy()


# ---------------------------------------------------------------- loss
def softmax_ce(z, labels, N):
    """Sum over the rows of z of the cross-entropy -log softmax(z)[label],
    divided by N (the mini-batch size).  Returns (loss, dloss/dz)."""
    zmax = z.max(axis=1, keepdims=True)
    e = np.exp(z - zmax)
    ssum = e.sum(axis=1, keepdims=True)
    logp = (z - zmax) - np.log(ssum)
    rows = np.arange(z.shape[0])
    loss = -logp[rows, labels].sum() / N
    p = e / ssum
    p[rows, labels] -= 1.0
    return loss, p / N

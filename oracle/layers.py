"""Layer forward functions and their vector-Jacobian products in fp64 numpy.

TEST INFRASTRUCTURE ONLY (the CPU oracle; see oracle/__init__.py).

The paper runs stock framework layers (Sec. IV-A, IV-C) and defines none of
them; each function below is the textbook definition written out.  Layouts:
activations NHWC (or [n, C]), conv weights [K, R, S, C], linear weights
[out, in].  Convolutions (cross-correlation) have an R x S kernel (square, or
Inception-V3's 1 x n / n x 1), stride 1 or 2, and either "same" zero padding
(R//2, S//2) or none ("valid", Inception-V3's stem and grid reductions); output
size floor((H + 2p - R) / stride) + 1.  ReLU'(0) = 0.  Max pooling sends the
gradient to the first maximum in row-major window order (the 3x3 stride-2 pool
pads with -inf, or not at all when "valid").  3x3 average pooling counts the zero
padding (divides by 9).  Batch normalisation uses the batch mean and the
biased batch variance of the micro-batch, eps 1e-5.
"""
from __future__ import annotations

import numpy as np

BN_EPS = 1e-5


def _win(r, s, Ho, Wo, stride):
    """Index of the Ho x Wo output grid's taps (r, s) in the padded input."""
    return (slice(None), slice(r, r + stride * (Ho - 1) + 1, stride),
            slice(s, s + stride * (Wo - 1) + 1, stride), slice(None))


def _shifted(xp, r, s, Ho, Wo, stride=1):
    """Tap (r, s) of every output position, from padded input xp, as [n*Ho*Wo, C]."""
    return np.ascontiguousarray(xp[_win(r, s, Ho, Wo, stride)]).reshape(-1, xp.shape[3])


def conv_out(H, k, stride=1, valid=False):
    """Output size of a convolution: floor((H + 2p - k) / stride) + 1, p = k//2 or 0."""
    p = 0 if valid else k // 2
    return (H + 2 * p - k) // stride + 1


# ---------------------------------------------------------------- conv / linear
def conv2d(x, w, b=None, stride=1, valid=False):
    """y[n,h,w,k] = sum_{r,s,c} x[n, h*st+r-ph, w*st+s-pw, c] * w[k,r,s,c] (+ b[k]),
    (ph, pw) = (R//2, S//2), or (0, 0) when valid."""
    n, H, W, C = x.shape
    K, R, S, _ = w.shape
    ph, pw = (0, 0) if valid else (R // 2, S // 2)
    Ho, Wo = conv_out(H, R, stride, valid), conv_out(W, S, stride, valid)
    xp = np.pad(x, ((0, 0), (ph, ph), (pw, pw), (0, 0)))
    y = np.zeros((n * Ho * Wo, K))
    for r in range(R):
        for s in range(S):
            y += _shifted(xp, r, s, Ho, Wo, stride) @ w[:, r, s, :].T
    if b is not None:
        y += b
    return y.reshape(n, Ho, Wo, K)


def conv2d_vjp(x, w, dy, need_dx=True, has_bias=False, stride=1, valid=False):
    """Gradients of conv2d w.r.t. x, w and b for cotangent dy."""
    n, H, W, C = x.shape
    K, R, S, _ = w.shape
    ph, pw = (0, 0) if valid else (R // 2, S // 2)
    Ho, Wo = dy.shape[1], dy.shape[2]
    xp = np.pad(x, ((0, 0), (ph, ph), (pw, pw), (0, 0)))
    dy2 = dy.reshape(-1, K)
    dw = np.zeros_like(w)
    dxp = np.zeros_like(xp) if need_dx else None
    for r in range(R):
        for s in range(S):
            dw[:, r, s, :] = dy2.T @ _shifted(xp, r, s, Ho, Wo, stride)
            if need_dx:
                dxp[_win(r, s, Ho, Wo, stride)] += (dy2 @ w[:, r, s, :]).reshape(n, Ho, Wo, C)
    db = dy2.sum(axis=0) if has_bias else None
    dx = dxp[:, ph:ph + H, pw:pw + W, :] if need_dx else None
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


def maxpool3s2(x, valid=False):
    """3x3 max pooling, stride 2, padding 1 with -inf (never chosen: the window
    centre is always inside), or no padding when valid.  Output
    floor((H + 2p - 3) / 2) + 1.  Returns (y, argmax index 0..8 per output, the
    first maximum in row-major order)."""
    n, H, W, C = x.shape
    p = 0 if valid else 1
    Ho, Wo = (H + 2 * p - 3) // 2 + 1, (W + 2 * p - 3) // 2 + 1
    xp = np.pad(x, ((0, 0), (p, p), (p, p), (0, 0)), constant_values=-np.inf)
    win = np.stack([xp[_win(r, s, Ho, Wo, 2)] for r in range(3) for s in range(3)], axis=3)
    idx = np.argmax(win, axis=3)
    y = np.take_along_axis(win, idx[:, :, :, None, :], axis=3)[:, :, :, 0, :]
    return y, idx


def maxpool3s2_vjp(x_shape, idx, dy, valid=False):
    """Each output's gradient goes to its window's first maximum; windows overlap,
    so an input adds the gradients of every output that chose it."""
    n, H, W, C = x_shape
    p = 0 if valid else 1
    Ho, Wo = dy.shape[1], dy.shape[2]
    dxp = np.zeros((n, H + 2 * p, W + 2 * p, C))
    for j in range(9):
        r, s = divmod(j, 3)
        dxp[_win(r, s, Ho, Wo, 2)] += np.where(idx == j, dy, 0.0)
    return dxp[:, p:p + H, p:p + W, :]


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

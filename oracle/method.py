"""XPipe's method steps in plain fp64 numpy: version difference, weight
prediction, the Adam update, and the other update rules the paper trains
with while predicting from Adam moments (momentum SGD, RMSProp).

TEST INFRASTRUCTURE ONLY.  This module is the CPU oracle that the GPU path is
checked against; it is never part of the product path.  Only tests/,
__graft_entry__.smoke() and bench.py's cpu_baseline leg may import it.

Notation: the paper calls the first moment v (decay gamma) and the second
moment m (decay lambda) in Eq. 4.  Here, as in Adam, m is the first moment
(beta1 = gamma = 0.9) and v the second (beta2 = lambda = 0.999).
"""
from __future__ import annotations

import math

import numpy as np

# rounding rules for the "round" of Eq. 1 and Eq. 2 (the paper does not define it)
HALF_UP = "half_up"        # round half away from zero (the default reading)
HALF_EVEN = "half_even"    # Python's round()
HALF_DOWN = "half_down"

PRED_EQ3 = "eq3"           # Eq. 3: m_hat / sqrt(v_hat + eps), bias correction 1 - beta^t
PRED_ADAMDIR = "adamdir"   # Adam's own direction m_hat / (sqrt(v_hat) + eps)
PRED_LITERAL = "literal"   # Eq. 4 as printed: m / (1 - beta1), v / (1 - beta2)
PRED_SMOOTHED = "smoothed" # SpecTrain's smoothed gradient (Sec. II): m / (1 - beta1), no v


def _round(x: float, rule: str) -> int:
    """Round a non-negative real to an integer under the named tie rule."""
    lo = math.floor(x)
    frac = x - lo
    if frac > 0.5:
        return lo + 1
    if frac < 0.5:
        return lo
    if rule == HALF_UP:
        return lo + 1
    if rule == HALF_DOWN:
        return lo
    if rule == HALF_EVEN:
        return lo if lo % 2 == 0 else lo + 1
    raise ValueError(rule)


def version_difference_fwd(size: int, T: int, rank: int, rule: str = HALF_UP,
                           ceil_half_rank: bool = False) -> int:
    """Eq. 1 (Sec. III-B): s = round((size + T - rank/2 - 2) / T) for the forward
    bellwether.  rank/2 is real-valued as printed; ceil_half_rank reads it as
    ceil(rank/2) instead."""
    half = math.ceil(rank / 2) if ceil_half_rank else rank / 2
    return _round((size + T - half - 2) / T, rule)


def version_difference_bwd(size: int, T: int, rank: int, rule: str = HALF_UP) -> int:
    """Eq. 2 (Sec. III-B): s = round((T + floor(rank/2) - 1) / T) for the backward
    bellwether.  It does not depend on size."""
    return _round((T + rank // 2 - 1) / T, rule)


def predict(W, m, v, t: int, s: int, lr: float, beta1: float, beta2: float, eps: float,
            mode: str = PRED_EQ3) -> np.ndarray:
    """Eq. 3 (Sec. III-B): W_hat = W - s * lr * dW with dW built from the Adam
    moments of Eq. 4.

    The moments are the optimizer state after t completed updates (the gradient
    of the mini-batch being predicted for does not exist yet).  With t = 0 the
    bias corrections 1 - beta^t vanish and no update has happened, so the
    prediction is W itself; s = 0 is likewise W.

    PRED_SMOOTHED is the predictor Sec. II attributes to SpecTrain: the weights
    moved s steps along momentum SGD's smoothed gradient.  Heavy-ball momentum
    without dampening keeps buf = sum_j mu^(k-j) g_j, and the first moment with
    beta1 = mu is (1 - mu) times the same sum, so m / (1 - beta1) is that
    buffer and the prediction is W - s lr buf.
    """
    W = np.asarray(W, np.float64)
    if s == 0 or (t == 0 and mode != PRED_LITERAL):
        return W.copy()
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    if mode == PRED_EQ3:
        m_hat = m / (1.0 - beta1 ** t)
        v_hat = v / (1.0 - beta2 ** t)
        dW = m_hat / np.sqrt(v_hat + eps)
    elif mode == PRED_ADAMDIR:
        m_hat = m / (1.0 - beta1 ** t)
        v_hat = v / (1.0 - beta2 ** t)
        dW = m_hat / (np.sqrt(v_hat) + eps)
    elif mode == PRED_LITERAL:
        dW = (m / (1.0 - beta1)) / np.sqrt(v / (1.0 - beta2) + eps)
    elif mode == PRED_SMOOTHED:
        dW = m / (1.0 - beta1)
    else:
        raise ValueError(mode)
    return W - s * lr * dW


def adam_update(W, m, v, G, t_next: int, lr: float, beta1: float, beta2: float,
                eps: float):
    """One Adam update (Kingma and Ba, Algorithm 1, which Sec. III-B and the
    robustness study of Sec. IV-D cite) applied at the mini-batch boundary with
    the accumulated gradient G (Sec. III-A).  t_next is the index of this update
    (1 for the first).  Returns (W, m, v) in fp64.

    The moment recurrences are Eq. 4's; the step uses Adam's bias-corrected
    estimates with eps outside the square root."""
    W = np.asarray(W, np.float64)
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    G = np.asarray(G, np.float64)
    m_new = beta1 * m + (1.0 - beta1) * G
    v_new = beta2 * v + (1.0 - beta2) * G * G
    m_hat = m_new / (1.0 - beta1 ** t_next)
    v_hat = v_new / (1.0 - beta2 ** t_next)
    W_new = W - lr * m_hat / (np.sqrt(v_hat) + eps)
    return W_new, m_new, v_new


# update rules besides Adam; the prediction always uses Adam moments
RULE_ADAM = "adam"
RULE_MOMENTUM_SGD = "momentum_sgd"
RULE_RMSPROP = "rmsprop"


def adam_moments(m, v, g, beta1: float, beta2: float):
    """Eq. 4's running averages of the gradient and of its square, the state
    XPipe's prediction reads (Sec. III-B), advanced by one gradient g."""
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    g = np.asarray(g, np.float64)
    return beta1 * m + (1.0 - beta1) * g, beta2 * v + (1.0 - beta2) * g * g


def momentum_sgd_update(W, buf, m, v, G, lr: float, momentum: float, weight_decay: float,
                        beta1: float, beta2: float):
    """Momentum SGD with weight decay, the update rule of the paper's main
    experiments (Sec. IV-D: momentum 0.9, weight decay 5e-4), with the Adam
    moments that the prediction of Eq. 3 keeps (Sec. III-B) advanced by the same
    gradient.  Heavy-ball form without dampening: g = G + wd * W,
    buf = momentum * buf + g, W = W - lr * buf.  Returns (W, buf, m, v) in fp64."""
    W = np.asarray(W, np.float64)
    buf = np.asarray(buf, np.float64)
    g = np.asarray(G, np.float64) + weight_decay * W
    buf_new = momentum * buf + g
    W_new = W - lr * buf_new
    m_new, v_new = adam_moments(m, v, g, beta1, beta2)
    return W_new, buf_new, m_new, v_new


def rmsprop_update(W, buf, sq, m, v, G, lr: float, alpha: float, eps: float, momentum: float,
                   weight_decay: float, beta1: float, beta2: float):
    """RMSProp with momentum, the update rule of the robustness study (Sec. IV-D:
    momentum 0.9), with the prediction's Adam moments advanced by the same
    gradient.  Tieleman and Hinton's running mean of the squared gradient with
    eps outside the root: g = G + wd * W, sq = alpha * sq + (1 - alpha) * g * g,
    buf = momentum * buf + g / (sqrt(sq) + eps), W = W - lr * buf.
    Returns (W, buf, sq, m, v) in fp64."""
    W = np.asarray(W, np.float64)
    buf = np.asarray(buf, np.float64)
    sq = np.asarray(sq, np.float64)
    g = np.asarray(G, np.float64) + weight_decay * W
    sq_new = alpha * sq + (1.0 - alpha) * g * g
    buf_new = momentum * buf + g / (np.sqrt(sq_new) + eps)
    W_new = W - lr * buf_new
    m_new, v_new = adam_moments(m, v, g, beta1, beta2)
    return W_new, buf_new, sq_new, m_new, v_new

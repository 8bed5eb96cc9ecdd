"""One pipeline stage's training step under XPipe, in fp64 numpy.

TEST INFRASTRUCTURE ONLY (the CPU oracle; see oracle/__init__.py).

The step per mini-batch follows Sec. III-A and III-B: the forward bellwether
predicts W_hat_f with its version difference (Eq. 1, Eq. 3), all T
micro-batches run the forward on the cached W_hat_f; the backward bellwether
predicts W_hat_b (Eq. 2, Eq. 3) and all T micro-batches run the backward on
it, each backward first recomputing its forward (Sec. IV-C, recomputation
during the backward pass); gradients are summed over the T micro-batches and
the weights are updated once, after the T-th backward (Sec. III-A).

Storage precision.  The oracle computes in fp64.  The GPU path stores
activations, activation gradients and the optimizer state in a narrower
format (fp32, or bf16 for activations in its bf16 variant).  Where a stored
value decides an integer (a max-pool argmax, a ReLU mask), both sides must
take the decision on values of the same precision, so the oracle can round
(to nearest, ties to even) at storage precision:
  storage="f32"   activations and gradients rounded to fp32;
  storage="bf16"  activations and gradients rounded to bf16, conv/linear
                  weights multiplied as bf16 (the fp32 prediction, rounded);
in both, the predicted weights, the master weights, both moments and the
gradient accumulator are rounded to fp32 each time they are written.
The rounding points are a property of the layer list alone: the output of
every layer is rounded (rounding is idempotent, so layers that only select
or copy stored values -- max pools, concatenations -- leave them unchanged,
and ReLU commutes with rounding).  In particular a BN output is rounded
before a residual add takes it in, and the sum is rounded again.  Every
activation gradient is rounded each time a contribution is added to it;
contributions arrive in reverse layer order.  storage="f64" rounds nothing.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

from . import layers as ly
from .method import (adam_update, momentum_sgd_update, predict, rmsprop_update, PRED_EQ3,
                     RULE_ADAM, RULE_MOMENTUM_SGD, RULE_RMSPROP)


def _rows(a):
    """A [n, 1, 1, C] activation (an NHWC map of one pixel, e.g. after the last
    pooling) as the [n, C] rows a linear layer reads; [n, C] stays."""
    if a.ndim == 4:
        assert a.shape[1] == 1 and a.shape[2] == 1, "linear input must have H = W = 1"
        return a.reshape(a.shape[0], a.shape[3])
    return a


def _round_f32(a):
    """Round to the nearest fp32 value, as fp64."""
    return np.asarray(a, np.float64).astype(np.float32).astype(np.float64)


def _round_bf16(a):
    """Round to the nearest bfloat16 value (ties to even) via fp32, as fp64."""
    f = np.ascontiguousarray(np.asarray(a, np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = (((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16).astype(np.uint32)
    return r.view(np.float32).astype(np.float64)


class Stage:
    """A stage given as a layer list (see the workloads module for the format)."""

    def __init__(self, layer_list: List[dict], storage: str = "f64"):
        self.layers = layer_list
        if storage not in ("f64", "f32", "bf16"):
            raise ValueError(storage)
        self.storage = storage
        # parameter tensor indices owned by each layer
        self.pidx = []
        k = 0
        for L in layer_list:
            n = 0
            if L["kind"] in ("linear", "conv"):
                n = 2 if L["bias"] else 1
            elif L["kind"] == "bn":
                n = 2
            self.pidx.append(list(range(k, k + n)))
            k += n
        self.n_params = k

    # storage rounding: activations / gradients (q), conv and linear weight
    # operands (qw), fp32 state (qs)
    def q(self, a):
        if self.storage == "bf16":
            return _round_bf16(a)
        if self.storage == "f32":
            return _round_f32(a)
        return a

    def qw(self, a):
        return self.q(a)

    def qs(self, a):
        return a if self.storage == "f64" else _round_f32(a)

    @property
    def has_loss(self):
        return self.layers[-1]["kind"] == "softmax_ce"

    # ------------------------------------------------------------ forward
    def forward(self, params, x, labels=None, N=None):
        """Returns (y, loss, saved): y is the stage output (the logits for a
        stage ending in a loss), loss the CE sum / N or None."""
        P = [np.asarray(p, np.float64) for p in params]
        outs = {-1: np.asarray(x, np.float64)}
        saved = {}
        loss = None
        for i, L in enumerate(self.layers):
            k = L["kind"]
            a = outs[L["inputs"][0]]
            pi = self.pidx[i]
            if k == "conv":
                b = P[pi[1]] if L["bias"] else None
                outs[i] = self.q(ly.conv2d(a, self.qw(P[pi[0]]), b, L.get("stride", 1),
                                           L.get("pad", "same") == "valid"))
            elif k == "linear":
                b = P[pi[1]] if L["bias"] else None
                outs[i] = self.q(ly.linear(_rows(a), self.qw(P[pi[0]]), b))
            elif k == "bn":
                y, xhat, rstd = ly.batchnorm(a, P[pi[0]], P[pi[1]])
                outs[i] = self.q(y)
                saved[i] = (xhat, rstd)
            elif k == "relu":
                outs[i] = self.q(ly.relu(a))
            elif k == "add":
                outs[i] = self.q(a + outs[L["inputs"][1]])
            elif k == "maxpool2":
                y, idx = ly.maxpool2(a)
                outs[i] = y
                saved[i] = idx
            elif k == "maxpool3s2":
                y, idx = ly.maxpool3s2(a, L.get("pad", "same") == "valid")
                outs[i] = y
                saved[i] = idx
            elif k == "avgpool3":
                outs[i] = self.q(ly.avgpool3(a))
            elif k == "gap":
                outs[i] = self.q(ly.gap(a))
            elif k == "concat":
                outs[i] = np.concatenate([outs[j] for j in L["inputs"]], axis=-1)
            elif k == "softmax_ce":
                loss, dz = ly.softmax_ce(a, labels, N)
                outs[i] = a
                saved[i] = dz
            else:
                raise ValueError(k)
        y = outs[len(self.layers) - 1]
        return y, loss, (outs, saved)

    # ------------------------------------------------------------ backward
    def backward(self, params, x, dy=None, labels=None, N=None, need_dx=True):
        """Recompute the forward at params, then the VJP.  Returns
        (dx or None, [grad per parameter tensor], loss)."""
        P = [np.asarray(p, np.float64) for p in params]
        _, loss, (outs, saved) = self.forward(P, x, labels, N)
        grads = [None] * self.n_params
        g = {}

        def acc(j, c):
            g[j] = self.q(c) if j not in g else self.q(g[j] + c)

        last = len(self.layers) - 1
        if self.has_loss:
            acc(self.layers[last]["inputs"][0], saved[last])
        else:
            g[last] = np.asarray(dy, np.float64)
        for i in range(last, -1, -1):
            L = self.layers[i]
            k = L["kind"]
            if k == "softmax_ce" or i not in g:
                continue
            gi = g[i]
            src = L["inputs"][0]
            a = outs[src]
            pi = self.pidx[i]
            want_dx = need_dx or src != -1
            if k == "conv":
                dx, dw, db = ly.conv2d_vjp(a, self.qw(P[pi[0]]), gi, want_dx, L["bias"],
                                           L.get("stride", 1), L.get("pad", "same") == "valid")
                grads[pi[0]] = dw
                if L["bias"]:
                    grads[pi[1]] = db
                if want_dx:
                    acc(src, dx)
            elif k == "linear":
                dx, dw, db = ly.linear_vjp(_rows(a), self.qw(P[pi[0]]), _rows(gi), want_dx, L["bias"])
                if dx is not None:
                    dx = dx.reshape(a.shape)
                grads[pi[0]] = dw
                if L["bias"]:
                    grads[pi[1]] = db
                if want_dx:
                    acc(src, dx)
            elif k == "bn":
                xhat, rstd = saved[i]
                dz, dgamma, dbeta = ly.batchnorm_vjp(xhat, rstd, P[pi[0]], gi)
                grads[pi[0]] = dgamma
                grads[pi[1]] = dbeta
                acc(src, dz)
            elif k == "relu":
                acc(src, ly.relu_vjp(outs[i], gi))
            elif k == "add":
                acc(src, gi)
                acc(L["inputs"][1], gi)
            elif k == "maxpool2":
                acc(src, ly.maxpool2_vjp(a.shape, saved[i], gi))
            elif k == "maxpool3s2":
                acc(src, ly.maxpool3s2_vjp(a.shape, saved[i], gi, L.get("pad", "same") == "valid"))
            elif k == "avgpool3":
                acc(src, ly.avgpool3_vjp(gi))
            elif k == "gap":
                acc(src, ly.gap_vjp(a.shape, gi))
            elif k == "concat":
                c0 = 0
                for j in L["inputs"]:
                    cj = outs[j].shape[-1]
                    acc(j, gi[..., c0:c0 + cj])
                    c0 += cj
            else:
                raise ValueError(k)
        dx = g.get(-1) if need_dx else None
        return dx, grads, loss


@dataclasses.dataclass
class Hyper:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    mode: str = PRED_EQ3
    # update rule at the mini-batch boundary (the prediction always uses the
    # Adam moments m, v): Adam, momentum SGD or RMSProp (both Sec. IV-D)
    rule: str = RULE_ADAM
    momentum: float = 0.9
    weight_decay: float = 0.0
    alpha: float = 0.99        # RMSProp's decay of the squared-gradient average
    rms_eps: float = 1e-8      # RMSProp's eps, outside the root


@dataclasses.dataclass
class MinibatchRecord:
    t_before: int
    w_pred_fwd: List[np.ndarray]
    w_pred_bwd: List[np.ndarray]
    ys: List[np.ndarray]
    losses: List[Optional[float]]
    dxs: List[Optional[np.ndarray]]
    grad: List[np.ndarray]          # accumulated over the T micro-batches
    W: List[np.ndarray]             # after the update
    m: List[np.ndarray]
    v: List[np.ndarray]
    buf: Optional[List[np.ndarray]] = None  # momentum buffer (momentum SGD, RMSProp)
    sq: Optional[List[np.ndarray]] = None   # RMSProp's squared-gradient average


def train_stage(stage: Stage, params, m, v, xs, s_fwd: int, s_bwd: int, hp: Hyper,
                labels=None, dys=None, need_dx=True, minibatches=None,
                t0: int = 0) -> List[MinibatchRecord]:
    """Run mini-batches through one stage.  xs[j][i] is micro-batch i of
    mini-batch j; labels or dys likewise.  params/m/v are per-tensor lists."""
    qs = stage.qs
    W = [qs(np.asarray(p, np.float64)) for p in params]
    m = [qs(np.asarray(a, np.float64)) for a in m]
    v = [qs(np.asarray(a, np.float64)) for a in v]
    t = t0
    buf = [np.zeros_like(a) for a in W]   # momentum buffer (momentum SGD, RMSProp)
    sq = [np.zeros_like(a) for a in W]    # RMSProp's squared-gradient average
    J = len(xs) if minibatches is None else minibatches
    T = len(xs[0])
    N = T * xs[0][0].shape[0]
    out = []
    for j in range(J):
        # forward bellwether: Eq. 1 version difference, Eq. 3 prediction, cached
        Wf = [qs(predict(W[k], m[k], v[k], t, s_fwd, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.mode))
              for k in range(len(W))]
        ys, losses = [], []
        for i in range(T):
            y, loss, _ = stage.forward(Wf, xs[j][i], None if labels is None else labels[j][i], N)
            ys.append(y)
            losses.append(loss)
        # backward bellwether: Eq. 2 version difference, Eq. 3 prediction, cached
        Wb = [qs(predict(W[k], m[k], v[k], t, s_bwd, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.mode))
              for k in range(len(W))]
        G = [np.zeros_like(a) for a in W]
        dxs = []
        for i in range(T):
            dx, gs, _ = stage.backward(Wb, xs[j][i], None if dys is None else dys[j][i],
                                       None if labels is None else labels[j][i], N, need_dx)
            for k in range(len(G)):
                G[k] = qs(G[k] + gs[k])
            dxs.append(dx)
        # update at the T-th backward (Sec. III-A): Adam with Eq. 4's moments,
        # or momentum SGD / RMSProp with the same moments kept for prediction
        t += 1
        if hp.rule == RULE_ADAM:
            new = [adam_update(W[k], m[k], v[k], G[k], t, hp.lr, hp.beta1, hp.beta2, hp.eps)
                   for k in range(len(W))]
            W = [qs(a[0]) for a in new]
            m = [qs(a[1]) for a in new]
            v = [qs(a[2]) for a in new]
        elif hp.rule == RULE_MOMENTUM_SGD:
            new = [momentum_sgd_update(W[k], buf[k], m[k], v[k], G[k], hp.lr, hp.momentum,
                                       hp.weight_decay, hp.beta1, hp.beta2)
                   for k in range(len(W))]
            W, buf, m, v = ([qs(a[q]) for a in new] for q in range(4))
        elif hp.rule == RULE_RMSPROP:
            new = [rmsprop_update(W[k], buf[k], sq[k], m[k], v[k], G[k], hp.lr, hp.alpha,
                                  hp.rms_eps, hp.momentum, hp.weight_decay, hp.beta1, hp.beta2)
                   for k in range(len(W))]
            W, buf, sq, m, v = ([qs(a[q]) for a in new] for q in range(5))
        else:
            raise ValueError(hp.rule)
        out.append(MinibatchRecord(t - 1, Wf, Wb, ys, losses, dxs, G, W, m, v,
                                   None if hp.rule == RULE_ADAM else list(buf),
                                   list(sq) if hp.rule == RULE_RMSPROP else None))
    return out


@dataclasses.dataclass
class ScheduleRecord:
    ys: List[np.ndarray]                 # forward output per micro-batch (index micro - 1)
    losses: List[Optional[float]]
    dxs: List[Optional[np.ndarray]]
    predictions: List[tuple]             # (kind, micro, s, t) of every prediction made
    W: List[np.ndarray]                  # after the last update
    m: List[np.ndarray]
    v: List[np.ndarray]


def train_schedule(stage: Stage, params, m, v, xs, events, hp: Hyper, labels=None, dys=None,
                   need_dx=True, t0: int = 0, draft: bool = False) -> ScheduleRecord:
    """One GPU's part of the interleaved schedule (oracle.schedule events) on
    one stage.  xs[k] / labels[k] / dys[k] belong to micro-batch k + 1; the
    mini-batch size N = T * micro-batch follows from the events.

    A bellwether predicts for its pass and caches the result (Eq. 3 with its
    event's s); the mini-batch's other micro-batches reuse the cache even when
    an update happened in between (Sec. III-B, final text).  draft=True takes
    the draft text's variant for the forward pass: a micro-batch that finds
    the cached prediction older than the latest update predicts again from the
    current weights with s reduced by the updates since the bellwether."""
    qs = stage.qs
    W = [qs(np.asarray(p, np.float64)) for p in params]
    m = [qs(np.asarray(a, np.float64)) for a in m]
    v = [qs(np.asarray(a, np.float64)) for a in v]
    buf = [np.zeros_like(a) for a in W]
    sq = [np.zeros_like(a) for a in W]
    n_micro = max(e.micro for e in events) if events else 0
    T = next((e.micro for e in events if e.update_after), n_micro)
    N = T * xs[0].shape[0]
    t = t0
    G = [np.zeros_like(a) for a in W]
    Wf = Wb = None
    bell_t = cache_t = -1
    bell_s = 0
    ys, losses, dxs = [None] * n_micro, [None] * n_micro, [None] * n_micro
    preds = []

    def pred(s):
        return [qs(predict(W[k], m[k], v[k], t, s, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.mode))
                for k in range(len(W))]

    for e in events:
        k = e.micro - 1
        lab = None if labels is None else labels[k]
        if e.kind == 0:
            if e.bellwether:
                Wf, bell_s, bell_t, cache_t = pred(e.s_eq), e.s_eq, t, t
                preds.append((0, e.micro, e.s_eq, t))
            elif draft and cache_t != t:
                s = max(bell_s - (t - bell_t), 0)
                Wf, cache_t = pred(s), t
                preds.append((0, e.micro, s, t))
            ys[k], losses[k], _ = stage.forward(Wf, xs[k], lab, N)
        else:
            if e.bellwether:
                Wb = pred(e.s_eq)
                preds.append((1, e.micro, e.s_eq, t))
            dx, gs, _ = stage.backward(Wb, xs[k], None if dys is None else dys[k], lab, N, need_dx)
            dxs[k] = dx
            for q in range(len(G)):
                G[q] = qs(G[q] + gs[q])
            if e.update_after:
                t += 1
                if hp.rule == RULE_ADAM:
                    new = [adam_update(W[q], m[q], v[q], G[q], t, hp.lr, hp.beta1, hp.beta2, hp.eps)
                           for q in range(len(W))]
                    W, m, v = ([qs(a[i]) for a in new] for i in range(3))
                elif hp.rule == RULE_MOMENTUM_SGD:
                    new = [momentum_sgd_update(W[q], buf[q], m[q], v[q], G[q], hp.lr, hp.momentum,
                                               hp.weight_decay, hp.beta1, hp.beta2) for q in range(len(W))]
                    W, buf, m, v = ([qs(a[i]) for a in new] for i in range(4))
                else:
                    new = [rmsprop_update(W[q], buf[q], sq[q], m[q], v[q], G[q], hp.lr, hp.alpha,
                                          hp.rms_eps, hp.momentum, hp.weight_decay, hp.beta1, hp.beta2)
                           for q in range(len(W))]
                    W, buf, sq, m, v = ([qs(a[i]) for a in new] for i in range(5))
                G = [np.zeros_like(a) for a in W]
    return ScheduleRecord(ys, losses, dxs, preds, W, m, v)

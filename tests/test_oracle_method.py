"""Pins for the oracle's method steps (Eq. 1-4 and the Adam update).

Each test checks the oracle against something other than its own formula: a
worked example the paper states, a brute-force schedule count, a closed form,
an invariant, or torch.optim.Adam as an independent library routine.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import method as om

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_worked_examples.json")))
HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)


# ------------------------------------------------------------------ Eq. 1 / Eq. 2
def test_worked_example_stale_forward():
    """Sec. III-A: at T=2 on 4 GPUs, GPU 0's forward bellwether sees 2 updates."""
    ex = GOLD["stale_forward_T2"]
    assert om.version_difference_fwd(ex["size"], ex["T"], ex["rank"]) == ex["updates_between"]
    # the updates land after micro-batches 2 and 4: the multiples of T
    assert [i for i in range(1, 6) if i % ex["T"] == 0] == ex["update_after_micro_batches"]


def test_no_pipeline_has_no_staleness():
    ex = GOLD["no_pipeline"]
    for rule in (om.HALF_UP, om.HALF_EVEN, om.HALF_DOWN):
        assert om.version_difference_fwd(ex["size"], ex["T"], ex["rank"], rule) == ex["s_fwd"]
        assert om.version_difference_bwd(ex["size"], ex["T"], ex["rank"], rule) == ex["s_bwd"]


def test_bellwether_indices():
    """Sec. III-B: the bellwether of mini-batch j is micro-batch (j-1)T+1."""
    for c in GOLD["bellwethers"]["cases"]:
        T, j = c["T"], c["mini_batch"]
        members = list(range((j - 1) * T + 1, j * T + 1))
        assert members[0] == c["bellwether"] and members[1:] == c["followers"]


def _schedule_counts(K, T, r, i):
    """Brute force over a unit-time 1F1B schedule: on GPU r the forward of
    micro-batch i runs in slot 2i+r and its backward in slot 2i+2K-1-r; each
    GPU updates at the end of the backward of every T-th micro-batch.
    Returns, for the forward and for the backward unit of micro-batch i, the
    number of updates on GPU r after that unit and up to the slot where GPU 0
    finishes the backward of the mini-batch's T-th micro-batch, not counting
    the mini-batch's own update."""
    j = (i - 1) // T + 1
    end = 2 * (j * T) + 2 * K - 1            # B_0 of the T-th micro-batch
    upd = [2 * (k * T) + 2 * K - 1 - r for k in range(1, j + K + 2) if k != j]
    f = 2 * i + r
    b = 2 * i + 2 * K - 1 - r
    return (sum(1 for u in upd if f < u <= end), sum(1 for u in upd if b < u <= end))


@pytest.mark.parametrize("K", [1, 2, 4, 8])
def test_eq1_eq2_against_schedule_at_T1(K):
    """At T=1 a brute-force 1F1B schedule count equals Eq. 2 for every rank and
    rounding rule, and equals Eq. 1 when rank/2 is read as ceil(rank/2) (the
    reading listed as an alternative; the literal rank/2 with round-half-up is
    the default and differs at odd ranks)."""
    i = 8 * K + 1  # a steady-phase micro-batch
    for r in range(K):
        f_cnt, b_cnt = _schedule_counts(K, 1, r, i)
        for rule in (om.HALF_UP, om.HALF_EVEN, om.HALF_DOWN):
            assert om.version_difference_bwd(K, 1, r, rule) == b_cnt
            assert om.version_difference_fwd(K, 1, r, rule, ceil_half_rank=True) == f_cnt


def test_schedule_reproduces_paper_example():
    """The brute-force schedule itself reproduces Sec. III-A's T=2 example."""
    f_cnt, _ = _schedule_counts(4, 2, 0, 5)
    assert f_cnt == GOLD["stale_forward_T2"]["updates_between"]


def test_eq2_independent_of_size():
    for T in (1, 2, 4):
        for r in range(8):
            vals = {om.version_difference_bwd(size, T, r) for size in (r + 1, 8, 16)}
            assert len(vals) == 1


def test_rounding_rules_on_ties():
    assert om._round(2.5, om.HALF_UP) == 3
    assert om._round(2.5, om.HALF_EVEN) == 2
    assert om._round(3.5, om.HALF_EVEN) == 4
    assert om._round(2.5, om.HALF_DOWN) == 2
    assert om._round(2.4999, om.HALF_UP) == 2 and om._round(2.5001, om.HALF_DOWN) == 3


# ------------------------------------------------------------------ prediction (Eq. 3)
def _state(n=4096, seed=7):
    rng = np.random.default_rng(seed)
    W = rng.normal(0, 0.02, n)
    m = rng.normal(0, 1e-3, n)
    v = np.abs(rng.normal(0, 1e-6, n))
    return W, m, v


@pytest.mark.parametrize("mode", [om.PRED_EQ3, om.PRED_ADAMDIR, om.PRED_LITERAL, om.PRED_SMOOTHED])
def test_predict_identities(mode):
    W, m, v = _state()
    assert np.array_equal(om.predict(W, m, v, 100, 0, mode=mode, **HP), W)          # s = 0
    z = np.zeros_like(W)
    assert np.array_equal(om.predict(W, z, v, 100, 3, mode=mode, **HP), W)          # m = 0
    if mode != om.PRED_LITERAL:
        assert np.array_equal(om.predict(W, m, v, 0, 3, mode=mode, **HP), W)        # t = 0


@pytest.mark.parametrize("mode", [om.PRED_EQ3, om.PRED_ADAMDIR, om.PRED_LITERAL, om.PRED_SMOOTHED])
def test_predict_linear_in_s(mode):
    """Eq. 3 extrapolates along a fixed direction: W_hat(s) - W = s (W_hat(1) - W)."""
    W, m, v = _state()
    d1 = om.predict(W, m, v, 100, 1, mode=mode, **HP) - W
    for s in (0, 1, 2, 3, 7):
        ds = om.predict(W, m, v, 100, s, mode=mode, **HP) - W
        np.testing.assert_allclose(ds, s * d1, rtol=1e-9, atol=1e-18)


@pytest.mark.parametrize("c", [0.3, -1e-3, 2.0, 3e-5, -4e-4])
@pytest.mark.parametrize("k", [1, 2, 5, 40])
def test_predict_constant_gradient_closed_form(c, k):
    """From zero moments, k Adam updates with a constant gradient c leave the
    bias-corrected moments at exactly c and c^2, so Eq. 3 (eps inside the
    root) predicts W_k - s lr c / sqrt(c^2 + eps)."""
    W = np.array([0.25, -0.5, 0.0])
    m = np.zeros(3)
    v = np.zeros(3)
    G = np.full(3, c)
    for t in range(1, k + 1):
        W, m, v = om.adam_update(W, m, v, G, t, **HP)
    for s in (1, 2, 7):
        got = om.predict(W, m, v, k, s, **HP)
        want = W - s * HP["lr"] * c / np.sqrt(c * c + HP["eps"])
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)


@pytest.mark.parametrize("c", [0.3, -1e-3, 2.0, 3e-5])
@pytest.mark.parametrize("k", [1, 2, 5, 40])
def test_predict_literal_constant_gradient_closed_form(c, k):
    """Eq. 4 as printed divides the moments by 1 - gamma and 1 - lambda with
    no power t.  From zero moments, k Adam updates with a constant gradient c
    leave m = c (1 - beta1^k) and v = c^2 (1 - beta2^k) (geometric sums of the
    recurrences), so the printed form predicts
        W_k - s lr [c (1 - beta1^k) / (1 - beta1)] / sqrt(c^2 (1 - beta2^k) / (1 - beta2) + eps).
    Swapping beta1 and beta2, or using 1 - beta^t, changes every case with
    k >= 2 (and the swap every case)."""
    W = np.array([0.25, -0.5, 0.0])
    m = np.zeros(3)
    v = np.zeros(3)
    G = np.full(3, c)
    for t in range(1, k + 1):
        W, m, v = om.adam_update(W, m, v, G, t, **HP)
    b1, b2, eps, lr = HP["beta1"], HP["beta2"], HP["eps"], HP["lr"]
    m_k = c * (1.0 - b1 ** k)
    v_k = c * c * (1.0 - b2 ** k)
    for s in (1, 2, 7):
        got = om.predict(W, m, v, k, s, mode=om.PRED_LITERAL, **HP)
        want = W - s * lr * (m_k / (1.0 - b1)) / np.sqrt(v_k / (1.0 - b2) + eps)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-17)


def test_predict_literal_hand_values():
    """Hand-computed values of Eq. 4 as printed (lr 1e-3, gamma 0.9, lambda
    0.999, eps 1e-8).  After two updates with gradient 1 from zero moments:
    m = 0.19, v = 0.001999, so the direction is (0.19 / 0.1) / sqrt(0.001999 /
    0.001 + 1e-8) = 1.9 / sqrt(1.99900001) = 1.3438389...; with m = 0.05,
    v = 0.0004 (t is not used): 0.5 / sqrt(0.4 + 1e-8) = 0.79056940...  With
    beta1 and beta2 swapped the first would be 190 / sqrt(0.01999) = 1343.8."""
    W = np.array([1.0, 1.0])
    m = np.array([0.19, 0.05])
    v = np.array([0.001999, 0.0004])
    got = om.predict(W, m, v, 2, 1, mode=om.PRED_LITERAL, **HP)
    want = 1.0 - 1e-3 * np.array([1.9 / np.sqrt(1.99900001), 0.5 / np.sqrt(0.40000001)])
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)
    np.testing.assert_allclose(1.0 - got, [1.3438389e-3, 7.905694e-4], rtol=1e-7)
    # s = 3 moves three times as far; t has no effect in this mode
    got3 = om.predict(W, m, v, 100, 3, mode=om.PRED_LITERAL, **HP)
    np.testing.assert_allclose(1.0 - got3, 3 * (1.0 - got), rtol=1e-12)


@pytest.mark.parametrize("wd", [0.0, 5e-4])
@pytest.mark.parametrize("k", [1, 2, 9])
def test_predict_smoothed_is_momentum_buffer(wd, k):
    """SpecTrain's predictor (Sec. II) moves W by s steps of momentum SGD's
    smoothed gradient.  The heavy-ball buffer is kept by its own recurrence in
    momentum_sgd_update (and matched to torch.optim.SGD above); with beta1
    equal to the momentum, the smoothed mode read from the first moment must
    give W - s lr buf for every s, with the same gradients and weight decay."""
    rng = np.random.default_rng(21)
    n = 300
    W = rng.normal(0, 0.05, n)
    buf, m, v = np.zeros(n), np.zeros(n), np.zeros(n)
    mu, lr = SGD["momentum"], SGD["lr"]
    for _ in range(k):
        g = rng.normal(0, 10 ** rng.uniform(-4, -1), n)
        W, buf, m, v = om.momentum_sgd_update(W, buf, m, v, g, lr, mu, wd, mu, HP["beta2"])
    for s in (1, 2, 7):
        got = om.predict(W, m, v, k, s, lr, mu, HP["beta2"], HP["eps"], mode=om.PRED_SMOOTHED)
        np.testing.assert_allclose(got, W - s * lr * buf, rtol=0, atol=1e-16)
        np.testing.assert_allclose(got - W, -s * lr * buf, rtol=1e-9, atol=1e-16)


@pytest.mark.parametrize("c", [0.3, -1e-3, 2.0])
@pytest.mark.parametrize("k", [1, 3, 40])
def test_predict_smoothed_constant_gradient_closed_form(c, k):
    """Constant gradient c from zero moments: m = c (1 - beta1^k), so the
    smoothed-gradient prediction is W - s lr c (1 - beta1^k) / (1 - beta1),
    with no bias correction and no second moment (v scaled by 100 changes
    nothing)."""
    W = np.array([0.25, -0.5, 0.0])
    m, v = np.zeros(3), np.zeros(3)
    G = np.full(3, c)
    for t in range(1, k + 1):
        W, m, v = om.adam_update(W, m, v, G, t, **HP)
    b1, lr = HP["beta1"], HP["lr"]
    for s in (1, 3):
        want = W - s * lr * c * (1.0 - b1 ** k) / (1.0 - b1)
        got = om.predict(W, m, v, k, s, mode=om.PRED_SMOOTHED, **HP)
        np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-17)
        got_v = om.predict(W, m, 100.0 * v, k, s, mode=om.PRED_SMOOTHED, **HP)
        assert np.array_equal(got_v, got)


def test_predict_adamdir_one_step_is_adam_step():
    """With Adam's own direction and s = 1, predicting from the moments that an
    update just produced reproduces that update's weights."""
    W, m, v = _state()
    G = np.random.default_rng(1).normal(0, 1e-3, W.size)
    for t in (1, 2, 50):
        W1, m1, v1 = om.adam_update(W, m, v, G, t, **HP)
        pred = om.predict(W, m1, v1, t, 1, mode=om.PRED_ADAMDIR, **HP)
        np.testing.assert_allclose(pred, W1, rtol=0, atol=1e-16)


# ------------------------------------------------------------------ Adam
def test_adam_matches_torch_optim():
    """torch.optim.Adam (float64, CPU) is an independent implementation of the
    same update (bias correction beta^t, eps outside the root)."""
    rng = np.random.default_rng(3)
    n = 1000
    W0 = rng.normal(0, 0.05, n)
    grads = [rng.normal(0, 10 ** rng.uniform(-6, -1), n) for _ in range(7)]
    p = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"])
    W, m, v = W0.copy(), np.zeros(n), np.zeros(n)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        W, m, v = om.adam_update(W, m, v, g, t, **HP)
        np.testing.assert_allclose(W, p.detach().numpy(), rtol=0, atol=1e-15)
        st = opt.state[p]
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-22)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-30)


@pytest.mark.parametrize("k", [1, 3, 5, 20])
def test_adam_constant_gradient_closed_form(k):
    c = np.array([0.3, -1e-3, 2.0, 1e-9, 0.0])
    W, m, v = np.zeros(5), np.zeros(5), np.zeros(5)
    for t in range(1, k + 1):
        W, m, v = om.adam_update(W, m, v, c, t, **HP)
    np.testing.assert_allclose(W, -k * HP["lr"] * c / (np.abs(c) + HP["eps"]), rtol=1e-12, atol=1e-20)


def test_adam_zero_gradient_keeps_zero_state():
    """Zero-padded tail elements (m = v = G = 0) never move."""
    z = np.zeros(8)
    W, m, v = om.adam_update(z, z, z, z, 5, **HP)
    assert not W.any() and not m.any() and not v.any()


# ------------------------------------------------------------------ momentum SGD / RMSProp
SGD = dict(lr=1e-2, momentum=0.9, weight_decay=5e-4)      # Sec. IV-D's settings
RMS = dict(lr=1e-4, alpha=0.99, eps=1e-8, momentum=0.9, weight_decay=0.0)  # Sec. IV-D


@pytest.mark.parametrize("wd", [0.0, 5e-4])
def test_momentum_sgd_matches_torch_optim(wd):
    """torch.optim.SGD (float64, CPU; momentum, no dampening, weight decay added
    to the gradient) is an independent implementation of the same rule."""
    rng = np.random.default_rng(11)
    n = 500
    W0 = rng.normal(0, 0.05, n)
    grads = [rng.normal(0, 10 ** rng.uniform(-4, -1), n) for _ in range(6)]
    p = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=SGD["lr"], momentum=SGD["momentum"], weight_decay=wd)
    W, buf, m, v = W0.copy(), np.zeros(n), np.zeros(n), np.zeros(n)
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        W, buf, m, v = om.momentum_sgd_update(W, buf, m, v, g, SGD["lr"], SGD["momentum"], wd,
                                             HP["beta1"], HP["beta2"])
        np.testing.assert_allclose(W, p.detach().numpy(), rtol=0, atol=1e-15)
        np.testing.assert_allclose(buf, opt.state[p]["momentum_buffer"].numpy(), rtol=1e-13, atol=1e-18)


@pytest.mark.parametrize("wd,mom", [(0.0, 0.9), (5e-4, 0.9), (0.0, 0.0)])
def test_rmsprop_matches_torch_optim(wd, mom):
    """torch.optim.RMSprop (float64, CPU; not centered, eps outside the root,
    momentum buffer of the normalised gradient) is an independent implementation."""
    rng = np.random.default_rng(12)
    n = 500
    W0 = rng.normal(0, 0.05, n)
    grads = [rng.normal(0, 10 ** rng.uniform(-4, -1), n) for _ in range(6)]
    p = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.RMSprop([p], lr=RMS["lr"], alpha=RMS["alpha"], eps=RMS["eps"],
                              momentum=mom, weight_decay=wd)
    W, buf, sq, m, v = W0.copy(), np.zeros(n), np.zeros(n), np.zeros(n), np.zeros(n)
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        W, buf, sq, m, v = om.rmsprop_update(W, buf, sq, m, v, g, RMS["lr"], RMS["alpha"], RMS["eps"],
                                             mom, wd, HP["beta1"], HP["beta2"])
        np.testing.assert_allclose(W, p.detach().numpy(), rtol=0, atol=1e-15)
        np.testing.assert_allclose(sq, opt.state[p]["square_avg"].numpy(), rtol=1e-13, atol=1e-30)


@pytest.mark.parametrize("k", [1, 2, 7])
def test_momentum_sgd_constant_gradient_closed_form(k):
    """Constant gradient c, no weight decay, from zero state: the buffer is the
    geometric sum c (1 - mu^j) / (1 - mu) after j steps, W moves by lr times
    the sum of the buffers, and the Adam moments are c (1 - beta1^k) and
    c^2 (1 - beta2^k)."""
    c = np.array([0.3, -1e-3, 2.0, 0.0])
    mu, lr = SGD["momentum"], SGD["lr"]
    W, buf, m, v = np.ones(4), np.zeros(4), np.zeros(4), np.zeros(4)
    for _ in range(k):
        W, buf, m, v = om.momentum_sgd_update(W, buf, m, v, c, lr, mu, 0.0, HP["beta1"], HP["beta2"])
    bufs = [c * (1 - mu ** j) / (1 - mu) for j in range(1, k + 1)]
    np.testing.assert_allclose(buf, bufs[-1], rtol=1e-13, atol=0)
    np.testing.assert_allclose(W, 1.0 - lr * sum(bufs), rtol=1e-13, atol=0)
    np.testing.assert_allclose(m, c * (1 - HP["beta1"] ** k), rtol=1e-13, atol=0)
    np.testing.assert_allclose(v, c * c * (1 - HP["beta2"] ** k), rtol=1e-12, atol=0)


@pytest.mark.parametrize("k", [1, 3])
def test_rmsprop_constant_gradient_closed_form(k):
    """Constant gradient c, no momentum, no weight decay: the squared average
    is c^2 (1 - alpha^j) after j steps and each step moves W by
    lr c / (|c| sqrt(1 - alpha^j) + eps)."""
    c = np.array([0.5, -2e-2, 3.0])
    a, e, lr = RMS["alpha"], RMS["eps"], RMS["lr"]
    W, buf, sq, m, v = np.zeros(3), np.zeros(3), np.zeros(3), np.zeros(3), np.zeros(3)
    for _ in range(k):
        W, buf, sq, m, v = om.rmsprop_update(W, buf, sq, m, v, c, lr, a, e, 0.0, 0.0,
                                             HP["beta1"], HP["beta2"])
    np.testing.assert_allclose(sq, c * c * (1 - a ** k), rtol=1e-12, atol=0)
    steps = [lr * c / (np.abs(c) * np.sqrt(1 - a ** j) + e) for j in range(1, k + 1)]
    np.testing.assert_allclose(W, -sum(steps), rtol=1e-12, atol=0)


def test_update_rules_weight_decay_reaches_the_moments():
    """The prediction's moments track the gradient the rule steps on: with
    G = 0 and weight decay wd they see wd * W."""
    W = np.array([0.5, -1.0])
    z = np.zeros(2)
    _, _, m, v = om.momentum_sgd_update(W, z, z, z, z, 1e-2, 0.9, 1e-3, HP["beta1"], HP["beta2"])
    np.testing.assert_allclose(m, (1 - HP["beta1"]) * 1e-3 * W, rtol=1e-15, atol=0)
    np.testing.assert_allclose(v, (1 - HP["beta2"]) * (1e-3 * W) ** 2, rtol=1e-14, atol=0)

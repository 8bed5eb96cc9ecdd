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


@pytest.mark.parametrize("mode", [om.PRED_EQ3, om.PRED_ADAMDIR, om.PRED_LITERAL])
def test_predict_identities(mode):
    W, m, v = _state()
    assert np.array_equal(om.predict(W, m, v, 100, 0, mode=mode, **HP), W)          # s = 0
    z = np.zeros_like(W)
    assert np.array_equal(om.predict(W, z, v, 100, 3, mode=mode, **HP), W)          # m = 0
    if mode != om.PRED_LITERAL:
        assert np.array_equal(om.predict(W, m, v, 0, 3, mode=mode, **HP), W)        # t = 0


@pytest.mark.parametrize("mode", [om.PRED_EQ3, om.PRED_ADAMDIR, om.PRED_LITERAL])
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

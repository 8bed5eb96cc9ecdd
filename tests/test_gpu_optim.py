"""GPU parity of the bandwidth-bound kernels (weight prediction, Eq. 3; Adam
with Eq. 4 moments, fused with zeroing the gradient and emitting the next
predictions) against the oracle, through the C ABI.

The kernels compute in fp64 and round once to fp32, so each result must be
the fp32 nearest to the oracle's fp64 value: at most 1 ulp apart, and only
where the exact value lies within fp64 rounding of an fp32 tie.  The
fp32 bar (relative L2 <= 2e-4) is asserted as well."""
import numpy as np
import pytest

import oracle
from oracle.stage import _round_bf16
import paper_1911_04610_amd as xp
import workloads as wl
from conftest import rel_l2

pytestmark = pytest.mark.gpu
TOL = 2e-4
MODES = {xp.PRED_EQ3: oracle.PRED_EQ3, xp.PRED_ADAMDIR: oracle.PRED_ADAMDIR,
         xp.PRED_LITERAL: oracle.PRED_LITERAL, xp.PRED_SMOOTHED: oracle.PRED_SMOOTHED}


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def _host(t):
    return t.cpu().numpy()


def _assert_rounded(a32, b64, what):
    """a32 must be the fp32 nearest to b64, except where b64 is (to fp64
    precision) exactly halfway between two fp32 values: there both are
    nearest and the kernel's fused multiply-adds may settle the tie either way."""
    a32 = np.asarray(a32, np.float32)
    b64 = np.asarray(b64, np.float64)
    b32 = b64.astype(np.float32)
    off = np.nonzero(a32 != b32)[0]                   # value compare: -0 == +0
    if off.size:
        ai = a32[off].view(np.int32).astype(np.int64)
        bi = b32[off].view(np.int32).astype(np.int64)
        assert np.abs(ai - bi).max() <= 1, f"{what}: more than 1 ulp"
        mid = (a32[off].astype(np.float64) + b32[off].astype(np.float64)) / 2
        ulp = np.abs(a32[off].astype(np.float64) - b32[off].astype(np.float64))
        tie = np.abs(b64[off] - mid) <= 1e-6 * ulp
        assert tie.all(), f"{what}: {np.count_nonzero(~tie)} elements not nearest and not ties"
    assert rel_l2(a32, b64) <= TOL


@pytest.mark.parametrize("n", [0, 1, 3, 4, 17, 1000003])
@pytest.mark.parametrize("mode", list(MODES))
def test_predict_flat_matches_oracle(n, mode):
    import torch
    st = wl.flat_state(n)
    hp = xp.Hyper(mode=mode)
    W, m, v = _dev(st.W), _dev(st.m), _dev(st.v)
    for s in (0, 1, 2, 3, 7):
        for t in (0, 1, 100):
            out = torch.empty_like(W)
            obf = torch.empty(max(n, 1), dtype=torch.int16, device="cuda")
            xp.xpipe_predict_flat(W, m, v, out, obf if n else None, s, hp, t)
            torch.cuda.synchronize()
            want = oracle.predict(st.W, st.m, st.v, t, s, hp.lr, hp.beta1, hp.beta2, hp.eps,
                                  MODES[mode])
            got = _host(out)
            if n == 0:
                continue
            _assert_rounded(got, want, f"predict s={s} t={t}")
            if s == 0 or (t == 0 and mode != xp.PRED_LITERAL):
                assert np.array_equal(got.view(np.int32), st.W.view(np.int32))  # bit for bit
            # bf16 shadow = nearest-even bf16 of the fp32 prediction
            bits = _host(obf).view(np.uint16)[:n].astype(np.uint32) << 16
            shadow = bits.view(np.float32)
            same = got == want.astype(np.float32)
            want_bf = _round_bf16(want.astype(np.float32))
            assert np.array_equal(shadow[same], want_bf[same].astype(np.float32))


@pytest.mark.parametrize("n", [5, 4096, 1000003])
def test_adam_flat_fused_matches_oracle(n):
    import torch
    st = wl.flat_state(n, seed=11)
    hp = xp.Hyper()
    for t in (0, 1, 99):
        W, m, v, G = _dev(st.W), _dev(st.m), _dev(st.v), _dev(st.G)
        pf, pb = torch.empty_like(W), torch.empty_like(W)
        xp.xpipe_adam_flat(W, m, v, G, hp, t, True, pf, 2, pb, 1)
        torch.cuda.synchronize()
        Wn, mn, vn = oracle.adam_update(st.W, st.m, st.v, st.G, t + 1, hp.lr, hp.beta1, hp.beta2,
                                        hp.eps)
        _assert_rounded(_host(W), Wn, "W")
        _assert_rounded(_host(m), mn, "m")
        _assert_rounded(_host(v), vn, "v")
        assert not _host(G).any()
        # predictions from the stored (fp32) state after update t+1
        W32, m32, v32 = (a.astype(np.float32) for a in (Wn, mn, vn))
        for out, s in ((pf, 2), (pb, 1)):
            want = oracle.predict(W32, m32, v32, t + 1, s, hp.lr, hp.beta1, hp.beta2, hp.eps)
            _assert_rounded(_host(out), want, f"pred s={s}")


def test_adam_flat_without_zeroing_or_predictions():
    import torch
    st = wl.flat_state(1024, seed=12)
    hp = xp.Hyper()
    W, m, v, G = _dev(st.W), _dev(st.m), _dev(st.v), _dev(st.G)
    xp.xpipe_adam_flat(W, m, v, G, hp, 5, False)
    torch.cuda.synchronize()
    assert np.array_equal(_host(G), st.G)
    Wn, _, _ = oracle.adam_update(st.W, st.m, st.v, st.G, 6, hp.lr, hp.beta1, hp.beta2, hp.eps)
    _assert_rounded(_host(W), Wn, "W")


def test_full_size_sweep_sampled():
    """1e8 parameters at t = 100, s in {0,1,2,3,7}: the launch the benchmark
    times; 200k sampled elements are checked against the oracle one by one."""
    import torch
    n = 100_000_000
    st = wl.flat_state(n)
    hp = xp.Hyper()
    W, m, v, G = _dev(st.W), _dev(st.m), _dev(st.v), _dev(st.G)
    out = torch.empty_like(W)
    idx = np.random.default_rng(0).choice(n, 200_000, replace=False)
    idx = np.concatenate([idx, [0, n - 1]])
    for s in (0, 1, 2, 3, 7):
        xp.xpipe_predict_flat(W, m, v, out, None, s, hp, 100)
        torch.cuda.synchronize()
        got = _host(out[torch.from_numpy(idx).cuda()])
        want = oracle.predict(st.W[idx], st.m[idx], st.v[idx], 100, s, hp.lr, hp.beta1, hp.beta2,
                              hp.eps)
        _assert_rounded(got, want, f"s={s}")
    pf, pb = torch.empty_like(W), torch.empty_like(W)
    xp.xpipe_adam_flat(W, m, v, G, hp, 100, True, pf, 2, pb, 1)
    torch.cuda.synchronize()
    ti = torch.from_numpy(idx).cuda()
    Wn, mn, vn = oracle.adam_update(st.W[idx], st.m[idx], st.v[idx], st.G[idx], 101, hp.lr,
                                    hp.beta1, hp.beta2, hp.eps)
    _assert_rounded(_host(W[ti]), Wn, "W")
    _assert_rounded(_host(m[ti]), mn, "m")
    _assert_rounded(_host(v[ti]), vn, "v")
    assert float(G.abs().max()) == 0.0


# ------------------------------------------------------------------ momentum SGD / RMSProp
RULES = [(xp.RULE_MOMENTUM_SGD, dict(lr=1e-2, momentum=0.9, weight_decay=5e-4)),
         (xp.RULE_RMSPROP, dict(lr=1e-4, momentum=0.9, weight_decay=5e-4, alpha=0.99, eps=1e-8))]


@pytest.mark.parametrize("n", [5, 4096, 1000003])
@pytest.mark.parametrize("rule,kw", RULES)
def test_rule_flat_fused_matches_oracle(n, rule, kw):
    """Momentum SGD / RMSProp with the prediction's Adam moments, fused with
    zeroing the gradient and the next two predictions."""
    import torch
    st = wl.flat_state(n, seed=13)
    b0, q0 = wl.rule_state(n)
    r = xp.Rule(rule=rule, **kw)
    hp = xp.Hyper(lr=r.lr)
    for t in (0, 7):
        W, m, v, G = _dev(st.W), _dev(st.m), _dev(st.v), _dev(st.G)
        buf, sq = _dev(b0), _dev(q0)
        pf, pb = torch.empty_like(W), torch.empty_like(W)
        xp.xpipe_rule_flat(W, buf, sq if rule == xp.RULE_RMSPROP else None, m, v, G, r, hp, t, True,
                           pf, 2, pb, 1)
        torch.cuda.synchronize()
        if rule == xp.RULE_MOMENTUM_SGD:
            Wn, bn, mn, vn = oracle.momentum_sgd_update(st.W, b0, st.m, st.v, st.G, r.lr, r.momentum,
                                                        r.weight_decay, hp.beta1, hp.beta2)
        else:
            Wn, bn, qn, mn, vn = oracle.rmsprop_update(st.W, b0, q0, st.m, st.v, st.G, r.lr, r.alpha,
                                                       r.eps, r.momentum, r.weight_decay, hp.beta1,
                                                       hp.beta2)
            _assert_rounded(_host(sq), qn, "sq")
        _assert_rounded(_host(W), Wn, "W")
        _assert_rounded(_host(buf), bn, "buf")
        _assert_rounded(_host(m), mn, "m")
        _assert_rounded(_host(v), vn, "v")
        assert not _host(G).any()
        W32, m32, v32 = (a.astype(np.float32) for a in (Wn, mn, vn))
        for out, s in ((pf, 2), (pb, 1)):
            want = oracle.predict(W32, m32, v32, t + 1, s, hp.lr, hp.beta1, hp.beta2, hp.eps)
            _assert_rounded(_host(out), want, f"pred s={s}")


@pytest.mark.parametrize("n", [5, 4096, 1000003])
def test_rule_flat_smoothed_prediction(n):
    """Momentum SGD predicting along its own smoothed gradient (SpecTrain's
    predictor, Sec. II): three fused updates from zero state with fresh
    gradients, beta1 = momentum.  The predictions of each pass must be the
    fp32 nearest to the oracle's from the stored state, and W_hat - W must
    track -s lr buf of the stored heavy-ball buffer."""
    import torch
    st = wl.flat_state(n, seed=14)
    r = xp.Rule(rule=xp.RULE_MOMENTUM_SGD, lr=1e-2, momentum=0.9, weight_decay=5e-4)
    hp = xp.Hyper(lr=r.lr, beta1=r.momentum, mode=xp.PRED_SMOOTHED)
    z = np.zeros(n, np.float32)
    W, buf, m, v = _dev(st.W), _dev(z), _dev(z), _dev(z)
    rng = np.random.default_rng(15)
    for t in range(3):
        g = rng.normal(0, 10 ** rng.uniform(-2, -1), n).astype(np.float32)
        G = _dev(g)
        pf, pb = torch.empty_like(W), torch.empty_like(W)
        xp.xpipe_rule_flat(W, buf, None, m, v, G, r, hp, t, True, pf, 2, pb, 1)
        torch.cuda.synchronize()
        W32, b32, m32, v32 = (_host(a) for a in (W, buf, m, v))
        for out, s in ((pf, 2), (pb, 1)):
            got = _host(out)
            want = oracle.predict(W32, m32, v32, t + 1, s, hp.lr, hp.beta1, hp.beta2, hp.eps,
                                  oracle.PRED_SMOOTHED)
            _assert_rounded(got, want, f"pred t={t} s={s}")
            d = got.astype(np.float64) - W32
            assert rel_l2(d, -s * r.lr * b32.astype(np.float64)) <= 1e-4


def test_rule_flat_rejects_bad_arguments():
    import torch
    W = torch.zeros(8, device="cuda")
    with pytest.raises(xp.XPipeError) as e:      # RMSProp needs its squared average
        xp.xpipe_rule_flat(W, W.clone(), None, W.clone(), W.clone(), W.clone(),
                           xp.Rule(rule=xp.RULE_RMSPROP), xp.Hyper(), 0)
    assert e.value.status == xp.EINVAL
    with pytest.raises(xp.XPipeError) as e:      # momentum must be below 1
        xp.xpipe_rule_flat(W, W.clone(), None, W.clone(), W.clone(), W.clone(),
                           xp.Rule(momentum=1.0), xp.Hyper(), 0)
    assert e.value.status == xp.EINVAL

"""GPU parity of the whole stage step (predict -> T x fwd -> predict -> T x
bwd with recomputation -> Adam) against the oracle, through the C ABI, on
every stage architecture at sizes that span several tiles with ragged
edges.

The fp32 variant stores fp32 and computes in fp64; it is compared with the
oracle in its fp32-storage mode, tensor by tensor, at relative L2 <= 2e-4.
The bf16 variant is compared with the oracle's bf16-storage mode at 2e-2.
Compared tensors per mini-batch: stage outputs, losses, input gradients, the
accumulated weight gradient, both predictions, and W, m, v after the update.
"""
import numpy as np
import pytest

import oracle
import paper_1911_04610_amd as xp
import workloads as wl
from conftest import rel_l2
from gpu_harness import run_stage

pytestmark = pytest.mark.gpu

TOL = {xp.F32: 2e-4, xp.BF16: 2e-2}
STORAGE = {xp.F32: "f32", xp.BF16: "bf16"}

CASES = {
    "tiny_mlp": lambda: wl.tiny_mlp(),
    "vgg16_stage0": lambda: wl.shrink(wl.vgg_stage(), micro_batch=4, spatial=(20, 20), T=2,
                                      minibatches=2),
    "resnet101_mid_stage": lambda: wl.shrink(
        wl.resnet_stage(), micro_batch=2, T=2, minibatches=2,
        layers=wl.resnet_stage_layers(blocks=2), in_shape=(9, 9, 512)),
    "inception_v3_stage": lambda: wl.shrink(
        wl.inception_stage(), micro_batch=2, T=2, minibatches=2,
        layers=wl.inception_stage_layers(modules=2), in_shape=(9, 9, 256)),
}


def _compare(gpu, ref, tol, what):
    errs = {}
    for j, (g, r) in enumerate(zip(gpu, ref)):
        for name in ("w_pred_fwd", "w_pred_bwd", "grad", "W", "m", "v"):
            for k, (a, b) in enumerate(zip(getattr(g, name), getattr(r, name))):
                errs[f"mb{j}.{name}[{k}]"] = rel_l2(a, b)
        for i, (a, b) in enumerate(zip(g.ys, r.ys)):
            errs[f"mb{j}.y[{i}]"] = rel_l2(a, b)
        for i, (a, b) in enumerate(zip(g.losses, r.losses)):
            if b is not None:
                errs[f"mb{j}.loss[{i}]"] = abs(a - b) / abs(b)
        for i, (a, b) in enumerate(zip(g.dxs, r.dxs)):
            if b is not None:
                errs[f"mb{j}.dx[{i}]"] = rel_l2(a, b)
    worst = max(errs, key=errs.get)
    print(f"{what}: worst {worst} = {errs[worst]:.3e} over {len(errs)} tensors")
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"{what}: {len(bad)} tensors above {tol}: " + ", ".join(
        f"{k}={v:.2e}" for k, v in sorted(bad.items(), key=lambda kv: -kv[1])[:12])


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("fwd_stream", [False, True])
def test_stage_step_fp32_matches_oracle(name, fwd_stream):
    """fp32 storage, fp64 arithmetic: every tensor of every mini-batch within
    2e-4 of the oracle's fp32-storage model (decisions taken on the same
    stored values on both sides) and of the exact fp64 oracle; with the
    forwards on one stream with the backwards, and on the stage's forward
    stream (chained passes) beside them."""
    w = CASES[name]()
    inp = wl.stage_inputs(w, act_dtype="f32")
    gpu, _ = run_stage(w, inp, xp.F32, xp.Hyper(), w.s_fwd, w.s_bwd, fwd_stream=fwd_stream)
    for storage in ("f32", "f64"):
        # the fp32-storage model, and the plain fp64 oracle that rounds nothing
        # (fp32 storage of fp64-computed values stays ~1e-6 from it here)
        ref = oracle.train_stage(oracle.Stage(w.layers, storage), inp.params, inp.m, inp.v, inp.xs,
                                 w.s_fwd, w.s_bwd, oracle.Hyper(), labels=inp.labels, dys=inp.dys)
        _compare(gpu, ref, TOL[xp.F32], f"{name}/f32 vs oracle-{storage}")


@pytest.mark.parametrize("name", ["tiny_mlp", "vgg16_stage0", "inception_v3_stage"])
@pytest.mark.parametrize("rule", [xp.RULE_MOMENTUM_SGD, xp.RULE_RMSPROP])
def test_stage_step_other_rules_fp32_match_oracle(name, rule):
    """The paper's other update rules (momentum SGD with weight decay, Sec.
    IV-D; RMSProp with momentum, Sec. IV-D) with Adam-moment prediction from
    the paper's moment initialisation: fp32 storage, every tensor within 2e-4
    of the oracle."""
    w = CASES[name]()
    inp = wl.stage_inputs(w, act_dtype="f32", moment_init="paper")
    if rule == xp.RULE_MOMENTUM_SGD:
        r = xp.Rule(rule=rule, lr=1e-2, momentum=0.9, weight_decay=5e-4)
        ohp = oracle.Hyper(lr=r.lr, rule=oracle.RULE_MOMENTUM_SGD, momentum=0.9, weight_decay=5e-4)
    else:
        r = xp.Rule(rule=rule, lr=1e-4, momentum=0.9, alpha=0.99, eps=1e-8)
        ohp = oracle.Hyper(lr=r.lr, rule=oracle.RULE_RMSPROP, momentum=0.9, alpha=0.99, rms_eps=1e-8)
    gpu, _ = run_stage(w, inp, xp.F32, xp.Hyper(lr=r.lr), w.s_fwd, w.s_bwd, rule=r)
    ref = oracle.train_stage(oracle.Stage(w.layers, "f32"), inp.params, inp.m, inp.v, inp.xs,
                             w.s_fwd, w.s_bwd, ohp, labels=inp.labels, dys=inp.dys)
    _compare(gpu, ref, TOL[xp.F32], f"{name}/f32/rule{rule}")


@pytest.mark.parametrize("name", ["tiny_mlp", "inception_v3_stage"])
def test_stage_step_smoothed_prediction_fp32_matches_oracle(name):
    """Momentum SGD predicting along its smoothed gradient (SpecTrain's
    predictor as Sec. II describes it; beta1 = momentum): both bellwether
    predictions and the fused update's predictions, every tensor within 2e-4
    of the oracle."""
    w = CASES[name]()
    inp = wl.stage_inputs(w, act_dtype="f32", moment_init="paper")
    r = xp.Rule(rule=xp.RULE_MOMENTUM_SGD, lr=1e-2, momentum=0.9, weight_decay=5e-4)
    ohp = oracle.Hyper(lr=r.lr, beta1=0.9, mode=oracle.PRED_SMOOTHED, rule=oracle.RULE_MOMENTUM_SGD,
                       momentum=0.9, weight_decay=5e-4)
    hp = xp.Hyper(lr=r.lr, beta1=0.9, mode=xp.PRED_SMOOTHED)
    gpu, _ = run_stage(w, inp, xp.F32, hp, w.s_fwd, w.s_bwd, rule=r)
    ref = oracle.train_stage(oracle.Stage(w.layers, "f32"), inp.params, inp.m, inp.v, inp.xs,
                             w.s_fwd, w.s_bwd, ohp, labels=inp.labels, dys=inp.dys)
    _compare(gpu, ref, TOL[xp.F32], f"{name}/f32/smoothed")


def _all_errs(recs, ref):
    e = {}
    for j, (g, r) in enumerate(zip(recs, ref)):
        for name in ("w_pred_fwd", "w_pred_bwd", "grad", "W", "m", "v"):
            for k, (a, b) in enumerate(zip(getattr(g, name), getattr(r, name))):
                e[f"mb{j}.{name}[{k}]"] = rel_l2(a, b)
        for i, (a, b) in enumerate(zip(g.ys, r.ys)):
            e[f"mb{j}.y[{i}]"] = rel_l2(a, b)
        for i, (a, b) in enumerate(zip(g.dxs, r.dxs)):
            if b is not None:
                e[f"mb{j}.dx[{i}]"] = rel_l2(a, b)
        for i, (a, b) in enumerate(zip(g.losses, r.losses)):
            if b is not None:
                e[f"mb{j}.loss[{i}]"] = abs(a - b) / abs(b)
    return e


@pytest.mark.parametrize("name", list(CASES))
def test_stage_step_bf16_matches_oracle(name):
    """bf16 storage with bf16 MFMA.  The first mini-batch's forward (outputs,
    loss) must be within 2e-2 of the oracle's bf16-storage model.  Gradients
    and everything downstream of them are not unique at bf16 precision: ReLU
    masks of pre-activations within bf16 noise of zero decide them, and two
    correct bf16 implementations differ by ~10% there.  For those tensors the
    GPU result must be no further from the exact (fp64) oracle than the
    oracle's own bf16 model is (x1.5, plus 2e-2)."""
    w = CASES[name]()
    inp = wl.stage_inputs(w, act_dtype="bf16")
    gpu, _ = run_stage(w, inp, xp.BF16, xp.Hyper(), w.s_fwd, w.s_bwd)
    args = (inp.params, inp.m, inp.v, inp.xs, w.s_fwd, w.s_bwd, oracle.Hyper())
    ref_bf = oracle.train_stage(oracle.Stage(w.layers, "bf16"), *args, labels=inp.labels, dys=inp.dys)
    ref_64 = oracle.train_stage(oracle.Stage(w.layers, "f64"), *args, labels=inp.labels, dys=inp.dys)
    fwd = {k: v for k, v in _all_errs(gpu, ref_bf).items() if k.startswith("mb0.y") or k.startswith("mb0.loss")}
    worst = max(fwd, key=fwd.get)
    print(f"{name}/bf16 forward vs oracle-bf16: worst {worst} = {fwd[worst]:.2e}")
    assert all(v <= 2e-2 for v in fwd.values()), {k: v for k, v in fwd.items() if v > 2e-2}
    e_gpu = _all_errs(gpu, ref_64)
    e_ref = _all_errs(ref_bf, ref_64)
    ratio = {k: e_gpu[k] / (1.5 * e_ref[k] + 2e-2) for k in e_gpu}
    worst = max(ratio, key=ratio.get)
    print(f"{name}/bf16 vs exact: worst {worst}: gpu {e_gpu[worst]:.2e}, bf16 model {e_ref[worst]:.2e}")
    bad = {k: (e_gpu[k], e_ref[k]) for k, r in ratio.items() if not r <= 1.0}
    assert not bad, ", ".join(f"{k}: gpu {a:.2e} model {b:.2e}" for k, (a, b) in list(bad.items())[:12])


EXACT_LR = 1e-5


def test_stage_step_bf16_exact_inputs_match_oracle():
    """The bf16 stage step where its results are unique: the VGG stage (no
    biases) on integer inputs with +-1 weights (workloads.exact_stage_inputs).
    Every forward product and partial sum is then an exact fp32 integer, so
    the GPU's fp32-accumulating MFMA GEMMs and the oracle's fp64 sums store the
    same bf16 values and take the same ReLU and (tie-heavy) max-pool decisions.
    The learning rate keeps |W_hat - W| below half a bf16 ulp of 1, so the
    second mini-batch multiplies the same bf16 operands while the fp32 master
    weights, moments and predictions move.  Every tensor of both mini-batches
    (outputs, input gradients, accumulated gradients, both predictions, W, m,
    v) is held to the bf16 bar of 2e-2; the forward outputs bit for bit."""
    w = wl.shrink(wl.vgg_stage(), micro_batch=4, spatial=(20, 20), T=2, minibatches=2,
                  layers=wl.vgg_stage_layers(bias=False))
    inp = wl.exact_stage_inputs(w)
    hp, ohp = xp.Hyper(lr=EXACT_LR), oracle.Hyper(lr=EXACT_LR)
    gpu, _ = run_stage(w, inp, xp.BF16, hp, w.s_fwd, w.s_bwd)
    ref = oracle.train_stage(oracle.Stage(w.layers, "bf16"), inp.params, inp.m, inp.v, inp.xs,
                             w.s_fwd, w.s_bwd, ohp, dys=inp.dys)
    from oracle.stage import _round_bf16
    for a, b in zip(ref[1].w_pred_fwd + ref[1].w_pred_bwd, inp.params):
        assert np.array_equal(_round_bf16(a), b)     # same bf16 operands in mini-batch 2
    assert not np.array_equal(ref[1].w_pred_fwd[0], inp.params[0])   # fp32 state moved
    for j in range(2):
        for a, b in zip(gpu[j].ys, ref[j].ys):
            np.testing.assert_array_equal(np.asarray(a, np.float64).reshape(b.shape), b)
    _compare(gpu, ref, TOL[xp.BF16], "vgg16_stage0/bf16/exact-inputs")


@pytest.mark.parametrize("name", ["tiny_mlp", "vgg16_stage0"])
def test_fused_update_emits_the_same_predictions(name):
    """Adam fused with the next mini-batch's predictions gives bit-identical
    predictions to separate predict calls."""
    w = CASES[name]()
    inp = wl.stage_inputs(w)
    hp = xp.Hyper()
    a, _ = run_stage(w, inp, xp.F32, hp, w.s_fwd, w.s_bwd, fused=True)
    b, _ = run_stage(w, inp, xp.F32, hp, w.s_fwd, w.s_bwd, fused=False)
    for ra, rb in zip(a, b):
        for x, y in zip(ra.w_pred_fwd + ra.w_pred_bwd + ra.W, rb.w_pred_fwd + rb.w_pred_bwd + rb.W):
            assert np.array_equal(x, y)


def test_zero_version_difference_predicts_master_weights():
    w = CASES["vgg16_stage0"]()
    inp = wl.stage_inputs(w)
    gpu, _ = run_stage(w, inp, xp.F32, xp.Hyper(), 0, 0)
    for j in range(1, len(gpu)):
        for a, b in zip(gpu[j].w_pred_fwd, gpu[j - 1].W):
            assert np.array_equal(a, b.astype(np.float32))


def test_repeat_runs_are_bitwise_identical():
    """No atomics or order-dependent reductions: two runs agree bit for bit."""
    w = CASES["inception_v3_stage"]()
    inp = wl.stage_inputs(w, act_dtype="bf16")
    a, _ = run_stage(w, inp, xp.BF16, xp.Hyper(), 1, 1, minibatches=1)
    b, _ = run_stage(w, inp, xp.BF16, xp.Hyper(), 1, 1, minibatches=1)
    for x, y in zip(a[0].grad + a[0].ys + a[0].dxs, b[0].grad + b[0].ys + b[0].dxs):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("name,dtype", [("inception_v3_stage", xp.BF16),
                                        ("inception_v3_stage", xp.F32),
                                        ("resnet101_mid_stage", xp.BF16)])
def test_concurrent_lanes_match_single_lane(name, dtype):
    """Independent branches run on several streams; with per-launch timing on
    everything runs on one stream.  Both orders give the same bits."""
    w = CASES[name]()
    inp = wl.stage_inputs(w, act_dtype="bf16" if dtype == xp.BF16 else "f32")
    one = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dtype)
    one.set_timing(True)
    a, _ = run_stage(w, inp, dtype, xp.Hyper(), 1, 1, minibatches=2, stage=one)
    b, _ = run_stage(w, inp, dtype, xp.Hyper(), 1, 1, minibatches=2)
    for ra, rb in zip(a, b):
        for x, y in zip(ra.grad + ra.ys + ra.dxs, rb.grad + rb.ys + rb.dxs):
            assert np.array_equal(x, y)


@pytest.mark.parametrize("name,dtype", [("inception_v3_stage", xp.BF16),
                                        ("resnet101_mid_stage", xp.BF16),
                                        ("vgg16_stage0", xp.F32)])
def test_recorded_passes_match_eager(name, dtype):
    """Passes replayed from their recorded HIP graphs (same pointers on every
    call, host reads and other eager work between replays) give the same bits
    as eager launches, on every replay."""
    w = CASES[name]()
    inp = wl.stage_inputs(w, act_dtype="bf16" if dtype == xp.BF16 else "f32")
    eager = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dtype)
    eager.set_graphs(False)
    a, _ = run_stage(w, inp, dtype, xp.Hyper(), 1, 1, minibatches=3, stage=eager, reuse_inputs=True)
    b, _ = run_stage(w, inp, dtype, xp.Hyper(), 1, 1, minibatches=3, reuse_inputs=True)
    for ra, rb in zip(a, b):
        for x, y in zip(ra.grad + ra.ys + ra.dxs + ra.W, rb.grad + rb.ys + rb.dxs + rb.W):
            assert np.array_equal(x, y)


def test_call_order_is_enforced():
    import torch
    w = wl.tiny_mlp()
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32)
    x = torch.zeros((32, 256), device="cuda")
    y = torch.zeros((32, 10), device="cuda")
    lab = torch.zeros(32, dtype=torch.int32, device="cuda")
    with pytest.raises(xp.XPipeError) as e:
        st.xpipe_stage_fwd(x, y, lab, None)
    assert e.value.status == xp.ESTATE
    with pytest.raises(xp.XPipeError) as e:
        st.xpipe_stage_bwd(x, None, lab, None)
    assert e.value.status == xp.ESTATE
    with pytest.raises(xp.XPipeError) as e:
        st.xpipe_adam_step(xp.Hyper(), 0)
    assert e.value.status == xp.ESTATE
    st.xpipe_predict_weights(xp.FWD, 1, xp.Hyper(), 0)
    st.xpipe_stage_fwd(x, y, lab, None)
    with pytest.raises(xp.XPipeError) as e:
        st.xpipe_stage_bwd(x, None, None, None)      # labels missing for a loss stage
    assert e.value.status == xp.EINVAL
    torch.cuda.synchronize()

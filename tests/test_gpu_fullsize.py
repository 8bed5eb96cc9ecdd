"""Parity at the full sizes the benchmark runs (micro-batch 32, full spatial
size, every layer at its real shape and therefore the same kernels, tiles and
grids), with T = 1 and one mini-batch so the fp64 oracle finishes in well
under a minute.

fp32 storage: every tensor (outputs, loss, input gradient, accumulated weight
gradient, predictions, W, m, v after the update) within 2e-4 of the oracle's
fp32-storage model; against the exact fp64 oracle, the forward within 2e-4 and
the rest within the bound stated in the test.  bf16 storage: the stage forward within 2e-2 of the
oracle's bf16-storage model, or no further from the exact (fp64) forward than
that bf16 model is (x1.25) where bf16 storage alone moves the output by more
than the bar (measured: 2.6e-2 for the 24-layer ResNet stage)."""
import numpy as np
import pytest

import oracle
import paper_1911_04610_amd as xp
import workloads as wl
from conftest import rel_l2
from gpu_harness import run_stage, to_device, to_host

pytestmark = pytest.mark.gpu
FULL = ["vgg16_stage0", "resnet101_mid_stage", "inception_v3_stage"]


@pytest.mark.parametrize("name", FULL)
def test_fullsize_fp32_step_matches_oracle(name):
    w = wl.shrink(wl.WORKLOADS[name](), T=1, minibatches=1)
    inp = wl.stage_inputs(w, act_dtype="f32", moment_init="paper")
    need_dx = w.rank > 0
    gpu, _ = run_stage(w, inp, xp.F32, xp.Hyper(), w.s_fwd, w.s_bwd, need_dx=need_dx)
    args = (inp.params, inp.m, inp.v, inp.xs, w.s_fwd, w.s_bwd, oracle.Hyper())
    kw = dict(labels=inp.labels, dys=inp.dys, need_dx=need_dx)
    r32 = oracle.train_stage(oracle.Stage(w.layers, "f32"), *args, **kw)[0]
    r64 = oracle.train_stage(oracle.Stage(w.layers, "f64"), *args, **kw)[0]
    e = _errs(gpu[0], r32, need_dx)
    worst = max(e, key=e.get)
    print(f"{name} full size fp32 vs oracle-f32: worst {worst} = {e[worst]:.2e} over {len(e)} tensors")
    bad = {k: v for k, v in e.items() if not v <= 2e-4}
    assert not bad, bad
    # Against the exact oracle: the forward within 2e-4; every other tensor
    # within 2e-4, or -- where fp32 storage alone moves it further (a ReLU mask
    # of a value within fp32 rounding of zero, whose effect the 24 BN layers
    # of the ResNet stage spread through every gradient) -- no further than
    # 1.25x the fp32-storage model's own distance, and never above 2e-2.
    e64, model = _errs(gpu[0], r64, need_dx), _errs(r32, r64, need_dx)
    worst = max(e64, key=e64.get)
    print(f"{name} full size fp32 vs oracle-f64: worst {worst} = {e64[worst]:.2e} "
          f"(fp32-storage model {model[worst]:.2e})")
    assert e64["y"] <= 2e-4
    bad = {k: (v, model[k]) for k, v in e64.items() if not (v <= 2e-4 or (v <= 1.25 * model[k] and v <= 2e-2))}
    assert not bad, bad


def _errs(g, r, need_dx):
    errs = {"y": rel_l2(g.ys[0], r.ys[0])}
    if need_dx:
        errs["dx"] = rel_l2(g.dxs[0], r.dxs[0])
    if r.losses[0] is not None:
        errs["loss"] = abs(g.losses[0] - r.losses[0]) / abs(r.losses[0])
    for field in ("grad", "w_pred_fwd", "w_pred_bwd", "W", "m", "v"):
        for k, (a, b) in enumerate(zip(getattr(g, field), getattr(r, field))):
            errs[f"{field}[{k}]"] = rel_l2(a, b)
    return errs


@pytest.mark.parametrize("name", FULL)
def test_fullsize_bf16_forward_matches_oracle(name):
    import torch
    w = wl.shrink(wl.WORKLOADS[name](), T=1, minibatches=1)
    inp = wl.stage_inputs(w, act_dtype="bf16", moment_init="paper")
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.BF16)
    st.set_flat(st.W, inp.params)
    st.set_flat(st.m, inp.m)
    st.set_flat(st.v, inp.v)
    st.xpipe_predict_weights(xp.FWD, w.s_fwd, xp.Hyper(), 3)
    n, H, W_, C = st.out_shape
    y = torch.empty((n, H, W_, C), dtype=torch.bfloat16, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    lab = None if inp.labels is None else torch.from_numpy(inp.labels[0][0]).cuda()
    st.xpipe_stage_fwd(to_device(inp.xs[0][0], xp.BF16), y, lab, loss if w.has_loss else None)
    torch.cuda.synchronize()
    Wf = st.get_tensors(st.w_pred_fwd)
    # the oracle's prediction of the same state (t = 3 completed updates)
    hp = oracle.Hyper()
    ref_w = [np.float32(oracle.predict(p, m, v, 3, w.s_fwd, hp.lr, hp.beta1, hp.beta2, hp.eps))
             for p, m, v in zip(inp.params, inp.m, inp.v)]
    for a, b in zip(Wf, ref_w):
        assert rel_l2(a, b) <= 2e-4
    N = w.T * w.micro_batch
    lab0 = None if inp.labels is None else inp.labels[0][0]
    yr, lr_, _ = oracle.Stage(w.layers, "bf16").forward(ref_w, inp.xs[0][0], lab0, N)
    y64, l64, _ = oracle.Stage(w.layers, "f64").forward(ref_w, inp.xs[0][0], lab0, N)
    gy = to_host(y).reshape(np.shape(yr))
    e, e_gpu, e_model = rel_l2(gy, yr), rel_l2(gy, y64), rel_l2(yr, y64)
    print(f"{name} full size bf16 forward: vs bf16 model {e:.2e}; vs exact {e_gpu:.2e} "
          f"(bf16 model vs exact {e_model:.2e})")
    # within the bf16 bar of the bf16 model, or -- where bf16 storage itself is
    # that far from exact (24 BN/ReLU layers of the ResNet stage) -- no further
    # from the exact result than the bf16 model is
    assert e <= 2e-2 or e_gpu <= 1.25 * e_model
    if lr_ is not None:
        el = abs(float(loss.item()) - lr_) / abs(lr_)
        print(f"   loss {el:.2e}")
        assert el <= 2e-2


def test_fullsize_bf16_exact_inputs_step_matches_oracle():
    """The benchmarked storage type through a whole step at full size, where
    its results are unique: the VGG stage (no biases) at micro-batch 32 and
    32 x 32 on integer inputs with +-1 weights (workloads.exact_stage_inputs),
    two accumulated micro-batches and two mini-batches, so the second
    mini-batch runs on non-trivial predictions (t = 1, s_f = 2, s_b = 1;
    Sec. III-B, Eq. 3).  Every forward partial sum is an exact fp32 integer
    (the largest stored activation is about 3e5), so both sides store the
    same bf16 values: the forward outputs bit for bit, every other tensor of
    both mini-batches (input gradients, accumulated gradients, both
    predictions, W, m, v) within the bf16 bar of 2e-2."""
    from test_gpu_stage import EXACT_LR, TOL, _compare
    from oracle.stage import _round_bf16
    w = wl.shrink(wl.WORKLOADS["vgg16_stage0"](), T=2, minibatches=2,
                  layers=wl.vgg_stage_layers(bias=False))
    assert w.micro_batch == 32 and tuple(w.in_shape) == (32, 32, 3)
    assert w.s_fwd > 0 and w.s_bwd > 0
    inp = wl.exact_stage_inputs(w)
    hp, ohp = xp.Hyper(lr=EXACT_LR), oracle.Hyper(lr=EXACT_LR)
    gpu, _ = run_stage(w, inp, xp.BF16, hp, w.s_fwd, w.s_bwd)
    ref = oracle.train_stage(oracle.Stage(w.layers, "bf16"), inp.params, inp.m, inp.v, inp.xs,
                             w.s_fwd, w.s_bwd, ohp, dys=inp.dys)
    for a, b in zip(ref[1].w_pred_fwd + ref[1].w_pred_bwd, inp.params):
        assert np.array_equal(_round_bf16(a), b)     # same bf16 operands in mini-batch 2
    assert not np.array_equal(ref[1].w_pred_fwd[0], inp.params[0])   # fp32 state moved
    for j in range(2):
        for a, b in zip(gpu[j].ys, ref[j].ys):
            np.testing.assert_array_equal(np.asarray(a, np.float64).reshape(b.shape), b)
    _compare(gpu, ref, TOL[xp.BF16], "vgg16_stage0/bf16/full-size/exact-inputs")

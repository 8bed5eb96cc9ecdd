"""Pins for the oracle's stage step: forward/VJP against torch float64
autograd on every stage architecture, gradient accumulation over
micro-batches, and the reduction to plain Adam training when there is no
pipeline (one stage, T = 1, s = 0)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from conftest import rel_l2
import torch_ref

SMALL = {
    "tiny_mlp": dict(micro_batch=6),
    "vgg16_stage0": dict(micro_batch=2, spatial=(12, 12)),
    "resnet101_mid_stage": dict(micro_batch=2, spatial=(5, 6),
                                layers=wl.resnet_stage_layers(blocks=2, c=24, mid=8),
                                in_shape=(5, 6, 24)),
    "inception_v3_stage": dict(micro_batch=2, spatial=(7, 7),
                               layers=wl.inception_stage_layers(modules=2, cin=256, classes=12),
                               in_shape=(7, 7, 256)),
}


def _small(name, **over):
    kw = dict(SMALL[name])
    kw.update(over)
    return wl.shrink(wl.WORKLOADS[name](), **kw)


@pytest.mark.parametrize("name", list(SMALL))
def test_stage_forward_backward_matches_torch(name):
    w = _small(name)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(w.layers)
    N = w.T * w.micro_batch
    lab = None if inp.labels is None else inp.labels[0][0]
    dy = None if inp.dys is None else inp.dys[0][0]
    y, loss, _ = st.forward(inp.params, inp.xs[0][0], lab, N)
    dx, grads, loss2 = st.backward(inp.params, inp.xs[0][0], dy, lab, N)
    yt, losst, dxt, gt = torch_ref.fwd_bwd(w.layers, inp.params, inp.xs[0][0], dy, lab, N)
    assert rel_l2(y, yt) < 1e-12
    if loss is not None:
        assert abs(loss - losst) < 1e-12 and loss2 == loss
    assert rel_l2(dx, dxt) < 1e-11
    for a, b in zip(grads, gt):
        assert rel_l2(a, b) < 1e-11


def test_full_vgg16_matches_torch():
    """The whole VGG-16 (thirteen convolutions, five pools, the classifier on a
    one-pixel map) against torch float64 autograd."""
    layers = wl.vgg16_layers()
    w = wl.StageWorkload("vgg16_full", layers, 2, 1, (32, 32, 3), 4, 0, 0, 0, minibatches=1)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(layers)
    x, lab = inp.xs[0][0], inp.labels[0][0]
    y, loss, _ = st.forward(inp.params, x, lab, 2)
    dx, grads, _ = st.backward(inp.params, x, None, lab, 2)
    yt, losst, dxt, gt = torch_ref.fwd_bwd(layers, inp.params, x, None, lab, 2)
    assert rel_l2(y.reshape(-1), np.asarray(yt).reshape(-1)) < 1e-12
    assert abs(loss - losst) < 1e-12
    assert rel_l2(dx, dxt) < 1e-11
    for a, b in zip(grads, gt):
        assert rel_l2(a, b) < 1e-11


def test_full_resnet101_matches_torch():
    """The whole ResNet-101 (strided stem, 3x3 stride-2 pool, 33 bottlenecks
    with strided first blocks and projection shortcuts, classifier) against
    torch float64 autograd, at a 64 x 64 input.  (At 32 x 32 the last group's
    BNs see two samples per channel and the 33 blocks amplify rounding-order
    differences to ~1e-3: a conditioning effect, not a disagreement; every
    shallower variant agrees to ~1e-12 at that size.)"""
    layers = wl.resnet101_layers()
    w = wl.StageWorkload("resnet101_full", layers, 2, 1, (64, 64, 3), 4, 0, 0, 0, minibatches=1)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(layers)
    x, lab = inp.xs[0][0], inp.labels[0][0]
    y, loss, _ = st.forward(inp.params, x, lab, 2)
    dx, grads, _ = st.backward(inp.params, x, None, lab, 2)
    yt, losst, dxt, gt = torch_ref.fwd_bwd(layers, inp.params, x, None, lab, 2)
    assert rel_l2(y.reshape(-1), np.asarray(yt).reshape(-1)) < 1e-10
    assert abs(loss - losst) < 1e-10
    assert rel_l2(dx, dxt) < 1e-10
    worst = max(rel_l2(a, b) for a, b in zip(grads, gt))
    assert worst < 1e-10, worst


def test_full_inception_v3_matches_torch():
    """The whole Inception-V3 (unpadded stem, three A modules, grid reductions B
    and D with their max-pool branches, four C modules with 1x7 / 7x1
    factorisations, two E modules with nested concats, classifier) against
    torch float64 autograd, at a 139 x 139 input (3 x 3 maps in the last modules)."""
    layers = wl.inception_v3_layers()
    w = wl.StageWorkload("inception_v3_full", layers, 2, 1, (139, 139, 3), 4, 0, 0, 0, minibatches=1)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(layers)
    x, lab = inp.xs[0][0], inp.labels[0][0]
    y, loss, _ = st.forward(inp.params, x, lab, 2)
    dx, grads, _ = st.backward(inp.params, x, None, lab, 2)
    yt, losst, dxt, gt = torch_ref.fwd_bwd(layers, inp.params, x, None, lab, 2)
    assert rel_l2(y.reshape(-1), np.asarray(yt).reshape(-1)) < 1e-10
    assert abs(loss - losst) < 1e-10
    assert rel_l2(dx, dxt) < 1e-10
    worst = max(rel_l2(a, b) for a, b in zip(grads, gt))
    assert worst < 1e-10, worst


@pytest.mark.parametrize("storage", ["f32", "bf16"])
def test_every_layer_output_is_rounded(storage):
    """The storage model rounds the output of every layer of the list,
    whatever kernels a GPU plan would fuse: a ResNet-101 block's BN outputs
    (those feeding a ReLU, the one feeding the residual add, and the
    projection shortcut's) and the residual sums are all storage values, and
    the add takes in the rounded BN output."""
    from oracle.stage import _round_bf16, _round_f32
    rnd = _round_bf16 if storage == "bf16" else _round_f32
    layers = wl.resnet101_layers(blocks=(1, 1, 1, 1))[:16]   # stem, pool, first block
    assert [L["kind"] for L in layers[-3:]] == ["bn", "add", "relu"]
    w = wl.StageWorkload("resnet_head", layers, 2, 1, (16, 16, 3), 4, 0, 0, 0, minibatches=1)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(layers, storage)
    _, _, (outs, _) = st.forward(inp.params, inp.xs[0][0])
    for i in range(len(layers)):
        assert np.array_equal(outs[i], rnd(outs[i])), (i, layers[i]["kind"])
    add = len(layers) - 2
    a, b = layers[add]["inputs"]
    # the sum is the rounding of the two stored operands' exact sum
    assert np.array_equal(outs[add], rnd(outs[a] + outs[b]))
    # and differs from rounding the unrounded BN output plus the shortcut
    ly_ = __import__("oracle.layers", fromlist=["batchnorm"])
    P = [np.asarray(p, np.float64) for p in inp.params]
    bn_raw, _, _ = ly_.batchnorm(outs[layers[a]["inputs"][0]], P[st.pidx[a][0]], P[st.pidx[a][1]])
    assert not np.array_equal(rnd(bn_raw + outs[b]), outs[add])


@pytest.mark.parametrize("name", ["tiny_mlp", "vgg16_stage0"])
def test_accumulated_gradient_equals_full_minibatch_gradient(name):
    """Sec. III-A: gradients accumulated over the T micro-batches of a mini-batch
    equal the gradient of the whole mini-batch (no BN here, so the micro-batch
    split does not change the function)."""
    w = _small(name, T=3)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(w.layers)
    N = w.T * w.micro_batch
    G = [np.zeros(p.shape) for p in inp.params]
    for i in range(w.T):
        lab = None if inp.labels is None else inp.labels[0][i]
        dy = None if inp.dys is None else inp.dys[0][i]
        _, g, _ = st.backward(inp.params, inp.xs[0][i], dy, lab, N)
        G = [a + b for a, b in zip(G, g)]
    x_all = np.concatenate(inp.xs[0])
    lab_all = None if inp.labels is None else np.concatenate(inp.labels[0])
    dy_all = None if inp.dys is None else np.concatenate(inp.dys[0])
    _, g_all, _ = st.backward(inp.params, x_all, dy_all, lab_all, N)
    for a, b in zip(G, g_all):
        assert rel_l2(a, b) < 1e-12


@pytest.mark.parametrize("name", ["tiny_mlp", "inception_v3_stage"])
def test_no_pipeline_reduces_to_plain_adam_training(name):
    """One stage, T = 1 and s = 0 (Eq. 1 and Eq. 2 both give 0 on one GPU):
    the step is ordinary Adam training of the stage.  Compared with a torch
    float64 model trained by torch.optim.Adam."""
    w = _small(name, T=1, minibatches=3)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(w.layers)
    s_f = oracle.version_difference_fwd(1, 1, 0)
    s_b = oracle.version_difference_bwd(1, 1, 0)
    assert s_f == 0 and s_b == 0
    hp = oracle.Hyper()
    recs = oracle.train_stage(st, inp.params, inp.m, inp.v, inp.xs, s_f, s_b, hp,
                              labels=inp.labels, dys=inp.dys)
    P = [torch.tensor(np.asarray(p, np.float64), requires_grad=True) for p in inp.params]
    opt = torch.optim.Adam(P, lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps)
    N = w.micro_batch
    for j in range(w.minibatches):
        opt.zero_grad()
        xt = torch.tensor(np.asarray(inp.xs[j][0], np.float64))
        y, loss = torch_ref.forward(w.layers, P, xt, inp.labels[j][0] if inp.labels else None, N)
        if loss is not None:
            loss.backward()
        else:
            y.backward(torch.tensor(np.asarray(inp.dys[j][0], np.float64)))
        opt.step()
        for a, b in zip(recs[j].W, P):
            np.testing.assert_allclose(a, b.detach().numpy(), rtol=0, atol=1e-13)


@pytest.mark.parametrize("rule", [oracle.RULE_MOMENTUM_SGD, oracle.RULE_RMSPROP])
def test_no_pipeline_reduces_to_plain_training_other_rules(rule):
    """One stage, T = 1, s = 0 with momentum SGD (weight decay 5e-4) or RMSProp
    (momentum 0.9) as the update rule: ordinary training with torch.optim.SGD
    or torch.optim.RMSprop of a torch float64 model."""
    w = _small("tiny_mlp", T=1, minibatches=3)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(w.layers)
    if rule == oracle.RULE_MOMENTUM_SGD:
        hp = oracle.Hyper(lr=1e-2, rule=rule, momentum=0.9, weight_decay=5e-4)
    else:
        hp = oracle.Hyper(lr=1e-4, rule=rule, momentum=0.9, alpha=0.99, rms_eps=1e-8)
    recs = oracle.train_stage(st, inp.params, inp.m, inp.v, inp.xs, 0, 0, hp,
                              labels=inp.labels, dys=inp.dys)
    P = [torch.tensor(np.asarray(p, np.float64), requires_grad=True) for p in inp.params]
    if rule == oracle.RULE_MOMENTUM_SGD:
        opt = torch.optim.SGD(P, lr=hp.lr, momentum=hp.momentum, weight_decay=hp.weight_decay)
    else:
        opt = torch.optim.RMSprop(P, lr=hp.lr, alpha=hp.alpha, eps=hp.rms_eps, momentum=hp.momentum)
    N = w.micro_batch
    for j in range(w.minibatches):
        opt.zero_grad()
        xt = torch.tensor(np.asarray(inp.xs[j][0], np.float64))
        y, loss = torch_ref.forward(w.layers, P, xt, inp.labels[j][0] if inp.labels else None, N)
        loss.backward()
        opt.step()
        for a, b in zip(recs[j].W, P):
            np.testing.assert_allclose(a, b.detach().numpy(), rtol=0, atol=1e-13)


def test_prediction_changes_the_step_once_moments_exist():
    """t = 0 makes both predictions equal W (no update has happened yet); from
    the second mini-batch on, s > 0 moves the predicted weights by s times the
    Adam direction."""
    w = _small("tiny_mlp", T=2, minibatches=2)
    inp = wl.stage_inputs(w)
    st = oracle.Stage(w.layers)
    hp = oracle.Hyper()
    recs = oracle.train_stage(st, inp.params, inp.m, inp.v, inp.xs, 2, 1, hp, labels=inp.labels)
    for a, b in zip(recs[0].w_pred_fwd, inp.params):
        assert np.array_equal(a, b)
    r1 = recs[1]
    for Wf, Wb, W, m, v in zip(r1.w_pred_fwd, r1.w_pred_bwd, recs[0].W, recs[0].m, recs[0].v):
        np.testing.assert_allclose(Wf - W, 2 * (Wb - W), rtol=1e-9, atol=1e-18)
        assert np.array_equal(Wf, oracle.predict(W, m, v, 1, 2, hp.lr, hp.beta1, hp.beta2, hp.eps))


def test_f32_storage_stays_close_to_exact():
    """Rounding activations, gradients and state to fp32 (values computed in
    fp64) perturbs the step by about fp32 precision: measured 3e-7 on the
    gradients here, held to 1e-5."""
    w = _small("vgg16_stage0", T=2, minibatches=2)
    inp = wl.stage_inputs(w)
    hp = oracle.Hyper()
    ref = oracle.train_stage(oracle.Stage(w.layers), inp.params, inp.m, inp.v, inp.xs, 2, 1, hp,
                             dys=inp.dys)
    got = oracle.train_stage(oracle.Stage(w.layers, "f32"), inp.params, inp.m, inp.v, inp.xs,
                             2, 1, hp, dys=inp.dys)
    for j in range(2):
        for a, b in zip(got[j].ys, ref[j].ys):
            assert rel_l2(a, b) < 1e-5
        for a, b in zip(got[j].grad, ref[j].grad):
            assert rel_l2(a, b) < 1e-5
    y = got[0].ys[0]
    assert np.array_equal(y, y.astype(np.float32).astype(np.float64))


def test_bf16_storage_forward_close_to_exact():
    """bf16 storage keeps the forward within bf16 precision of the exact one.
    (Its backward is not close to the exact one: max-pool windows whose top two
    values round to the same bf16 value route the gradient differently, which
    is why the bf16 variant is checked against this storage mode.)"""
    w = _small("vgg16_stage0", T=2, minibatches=1)
    inp = wl.stage_inputs(w, act_dtype="bf16")
    hp = oracle.Hyper()
    ref = oracle.train_stage(oracle.Stage(w.layers), inp.params, inp.m, inp.v, inp.xs, 2, 1, hp,
                             dys=inp.dys)
    got = oracle.train_stage(oracle.Stage(w.layers, "bf16"), inp.params, inp.m, inp.v, inp.xs,
                             2, 1, hp, dys=inp.dys)
    for a, b in zip(got[0].ys, ref[0].ys):
        assert rel_l2(a, b) < 1e-2
    y = got[0].ys[0]
    assert np.array_equal(y, ostage_round(y))


def ostage_round(a):
    from oracle.stage import _round_bf16
    return _round_bf16(a)


def test_bf16_whole_stage_gradients_are_not_unique():
    """Why the deep BN stages' bf16 gradients are held to a bar relative to the
    exact result rather than element by element to the bf16 model: two
    evaluations of the oracle's own bf16 model that differ only by a relative
    2^-24 sqrt(K) perturbation of each convolution before it is rounded (what
    fp32 accumulation in another order does) disagree on the ResNet stage's
    accumulated gradients by more than twice the 2e-2 bar, while their forward
    outputs stay within it.  Each rounding difference moves a BN channel's
    statistics, which moves the bf16 rounding of other elements, and so on
    through the layers.  No bf16 implementation can be held to 2e-2 on these
    gradients against any other."""
    from oracle import layers as ly
    w = wl.shrink(wl.resnet_stage(), micro_batch=2, T=2, minibatches=1,
                  layers=wl.resnet_stage_layers(blocks=2), in_shape=(9, 9, 512))
    inp = wl.stage_inputs(w, act_dtype="bf16", moment_init="paper")
    args = (inp.params, inp.m, inp.v, inp.xs, w.s_fwd, w.s_bwd, oracle.Hyper())
    ref = oracle.train_stage(oracle.Stage(w.layers, "bf16"), *args, dys=inp.dys)
    rng = np.random.default_rng(5)
    conv = ly.conv2d

    def noisy(x, wt, b=None, stride=1, valid=False):
        y = conv(x, wt, None, stride, valid)
        y = y * (1 + 2.0 ** -24 * np.sqrt(wt[0].size) * rng.standard_normal(y.shape))
        return y if b is None else y + b

    ly.conv2d = noisy
    try:
        alt = oracle.train_stage(oracle.Stage(w.layers, "bf16"), *args, dys=inp.dys)
    finally:
        ly.conv2d = conv
    assert max(rel_l2(a, b) for a, b in zip(alt[0].ys, ref[0].ys)) < 2e-2
    assert max(rel_l2(a, b) for a, b in zip(alt[0].grad, ref[0].grad)) > 4e-2

"""GPU parity of each layer kernel, through one-layer (or few-layer) stages
driven by the C ABI, in both storage formats.

Each case runs one mini-batch of T = 2 micro-batches (forward, then backward
with recomputation) and compares the stage output, the input gradient and
the accumulated weight gradient with the oracle on identical inputs.  These
stages have no chain of ReLU / max-pool decisions, so the bf16 variant is
held to the bf16 bar (relative L2 2e-2) against the oracle's bf16-storage
model, and, where the stage has no ReLU or max-pool at all, against the exact
(fp64) oracle too; the fp32
variant is held to 2e-4 against the oracle's fp32-storage model."""
import numpy as np
import pytest

import oracle
import paper_1911_04610_amd as xp
import workloads as wl
from conftest import rel_l2
from gpu_harness import run_stage

pytestmark = pytest.mark.gpu


def conv(x, cin, cout, k, bias=False, stride=1, kw=None, pad="same"):
    L = dict(kind="conv", inputs=[x], cin=cin, cout=cout, k=k, bias=bias, stride=stride)
    if kw is not None:
        L["kw"] = kw
    if pad != "same":
        L["pad"] = pad
    return L


def bn(x, c):
    return dict(kind="bn", inputs=[x], cin=c, cout=c)


def _module(kind):
    """Small Inception-V3 grid-reduction B or E module after a conv + BN + ReLU."""
    b = wl._Builder()
    x = b.conv_bn_relu(-1, 16, 32, 1)
    if kind == "B":
        b1 = b.conv_bn_relu(x, 32, 24, 3, stride=2, pad="valid")
        b2 = b.conv_bn_relu(b.conv_bn_relu(b.conv_bn_relu(x, 32, 16, 1), 16, 24, 3), 24, 24, 3,
                            stride=2, pad="valid")
        b3 = b.add(kind="maxpool3s2", inputs=[x], pad="valid")
        b.add(kind="concat", inputs=[b1, b2, b3])
    else:
        b1 = b.conv_bn_relu(x, 32, 16, 1)
        t = b.conv_bn_relu(x, 32, 24, 1)
        b2 = b.add(kind="concat", inputs=[b.conv_bn_relu(t, 24, 16, 1, kw=3), b.conv_bn_relu(t, 24, 16, 3, kw=1)])
        t = b.conv_bn_relu(b.conv_bn_relu(x, 32, 24, 1), 24, 16, 3)
        b3 = b.add(kind="concat", inputs=[b.conv_bn_relu(t, 16, 16, 1, kw=3), b.conv_bn_relu(t, 16, 16, 3, kw=1)])
        b4 = b.conv_bn_relu(b.add(kind="avgpool3", inputs=[x]), 32, 8, 1)
        b.add(kind="concat", inputs=[b1, b2, b3, b4])
    return b.layers


LAYER_CASES = {
    # name: (layers, per-sample input shape, micro-batch)
    "conv3x3_bias": ([conv(-1, 64, 128, 3, True)], (20, 20, 64), 3),
    "conv1x1_wide": ([conv(-1, 256, 64, 1)], (9, 9, 256), 2),
    "conv5x5_c48": ([conv(-1, 48, 64, 5)], (11, 11, 48), 2),
    "conv3x3_c3_flat": ([conv(-1, 3, 64, 3, True)], (18, 18, 3), 2),
    "conv_n96_c96": ([conv(-1, 96, 96, 3)], (7, 9, 96), 2),
    # 2 450 pixels per micro-batch: the 96 x 128 weight-gradient tile over
    # several pixel splits (K = 864: a ragged last K block)
    "conv_n96_c96_splits": ([conv(-1, 96, 96, 3)], (35, 35, 96), 2),
    # 65 884 rows (a ragged last tile): the 128-row tiles of large images,
    # 128 columns on eight waves (forward) and 64 (data gradient); then N = 160
    "conv3x3_many_rows_n128": ([conv(-1, 64, 128, 3)], (182, 181, 64), 2),
    "conv1x1_many_rows_n160": ([conv(-1, 64, 160, 1)], (182, 181, 64), 2),
    # the same for the unpadded and strided gathers (forward and data gradient):
    # 66 978 output / 68 450 input rows; 65 884 output / 263 536 input rows
    "conv3x3_valid_many_rows_n96": ([conv(-1, 80, 96, 3, pad="valid")], (185, 185, 80), 2),
    "conv3x3_valid_many_rows_n128": ([conv(-1, 64, 128, 3, pad="valid")], (185, 185, 64), 2),
    "conv3x3_s2_many_rows": ([conv(-1, 64, 64, 3, stride=2)], (364, 362, 64), 2),
    "conv_relu": ([conv(-1, 64, 64, 3, True), dict(kind="relu", inputs=[0])], (13, 13, 64), 2),
    "bn": ([dict(kind="bn", inputs=[-1], cin=96, cout=96)], (9, 9, 96), 3),
    "bn_add_relu": ([dict(kind="bn", inputs=[-1], cin=128, cout=128),
                     dict(kind="add", inputs=[0, -1]), dict(kind="relu", inputs=[1])], (9, 9, 128), 2),
    "maxpool_even": ([dict(kind="maxpool2", inputs=[-1])], (10, 12, 64), 2),
    "maxpool_odd": ([dict(kind="maxpool2", inputs=[-1])], (9, 11, 32), 2),
    "avgpool3": ([dict(kind="avgpool3", inputs=[-1])], (9, 9, 64), 2),
    # rows of 15 = two full sliding-window runs of 7 and a ragged run of 1
    "avgpool3_ragged_rows": ([dict(kind="avgpool3", inputs=[-1])], (5, 15, 32), 2),
    "avgpool3_single_pixel": ([dict(kind="avgpool3", inputs=[-1])], (1, 1, 16), 3),
    "avgpool3_after_concat": ([conv(-1, 32, 32, 1), conv(-1, 32, 16, 3),
                               dict(kind="concat", inputs=[0, 1]),
                               dict(kind="avgpool3", inputs=[2]), conv(3, 48, 32, 1)],
                              (6, 8, 32), 2),
    # 35 x 35 pixels: the average pool's partial sums split the pixels
    "head_gap_many_pixels": ([dict(kind="gap", inputs=[-1]),
                              dict(kind="linear", inputs=[0], cin=64, cout=10, bias=True),
                              dict(kind="softmax_ce", inputs=[1], classes=10)], (35, 35, 64), 2),
    "head_gap_linear_ce": ([dict(kind="gap", inputs=[-1]),
                            dict(kind="linear", inputs=[0], cin=256, cout=200, bias=True),
                            dict(kind="softmax_ce", inputs=[1], classes=200)], (7, 7, 256), 4),
    "mlp_head10": ([dict(kind="linear", inputs=[-1], cin=256, cout=10, bias=True),
                    dict(kind="softmax_ce", inputs=[0], classes=10)], (256,), 32),
    # more classes than the cross-entropy kernel keeps in registers (512)
    "mlp_head600": ([dict(kind="linear", inputs=[-1], cin=128, cout=600, bias=True),
                     dict(kind="softmax_ce", inputs=[0], classes=600)], (128,), 8),
    # the head's average-pool backward completes the BN output's gradient and
    # takes its backward partials (bf16)
    "bn_relu_gap_head": ([conv(-1, 32, 64, 3), bn(0, 64), dict(kind="relu", inputs=[1]),
                          dict(kind="gap", inputs=[2]),
                          dict(kind="linear", inputs=[3], cin=64, cout=10, bias=True),
                          dict(kind="softmax_ce", inputs=[4], classes=10)], (9, 9, 32), 4),
    "concat_views": ([conv(-1, 64, 64, 1), conv(-1, 64, 32, 3),
                      dict(kind="concat", inputs=[0, 1]), conv(2, 96, 48, 1)], (8, 8, 64), 2),
    # two wide 3x3 siblings (bf16: one 512 x 4608 launch of 576 tiles, whose
    # weight gradient takes one split and adds each sibling's rows straight into
    # its own accumulator)
    "siblings_merged_wide": ([conv(-1, 512, 256, 3), bn(0, 256), dict(kind="relu", inputs=[1]),
                              conv(-1, 512, 256, 3), bn(3, 256), dict(kind="relu", inputs=[4]),
                              dict(kind="add", inputs=[2, 5])], (4, 4, 512), 2),
    # two 1x1 siblings on one input share a launch in bf16 (channel-slice outputs)
    "siblings_merged_bn": ([conv(-1, 64, 32, 1), dict(kind="bn", inputs=[0], cin=32, cout=32),
                            dict(kind="relu", inputs=[1]),
                            conv(-1, 64, 16, 1), dict(kind="bn", inputs=[3], cin=16, cout=16),
                            dict(kind="relu", inputs=[4]), conv(5, 16, 24, 3),
                            dict(kind="relu", inputs=[6]),
                            dict(kind="avgpool3", inputs=[-1]), conv(8, 64, 8, 1),
                            dict(kind="bn", inputs=[9], cin=8, cout=8), dict(kind="relu", inputs=[10]),
                            dict(kind="concat", inputs=[2, 7, 11])], (7, 9, 64), 2),
    "add_relu_elementwise": ([conv(-1, 32, 32, 1), dict(kind="add", inputs=[0, -1]),
                              dict(kind="relu", inputs=[1])], (6, 7, 32), 2),
    "pool_then_relu": ([dict(kind="maxpool2", inputs=[-1]), dict(kind="relu", inputs=[0])],
                       (8, 8, 64), 2),
    # stride 2 (ResNet-101): odd and even sizes, ragged row tiles; the data
    # gradient gathers the output gradient tap by tap
    "conv3x3_s2": ([conv(-1, 64, 128, 3, stride=2)], (15, 14, 64), 2),
    "conv1x1_s2_projection": ([conv(-1, 64, 128, 1, stride=2)], (14, 13, 64), 2),
    "conv3x3_s2_narrow": ([conv(-1, 32, 32, 3, True, stride=2)], (9, 10, 32), 3),
    # 12 channels: element-gather forward and data gradient in bf16
    "conv3x3_s2_c12_flat": ([conv(-1, 12, 12, 3, stride=2)], (11, 7, 12), 2),
    "conv7x7_s2_stem": ([conv(-1, 3, 64, 7, stride=2)], (23, 22, 3), 2),
    "maxpool3s2_even": ([dict(kind="maxpool3s2", inputs=[-1])], (12, 10, 64), 2),
    "maxpool3s2_odd": ([dict(kind="maxpool3s2", inputs=[-1])], (11, 9, 24), 2),
    "maxpool3s2_c20": ([dict(kind="maxpool3s2", inputs=[-1])], (9, 8, 20), 2),
    # ResNet-101 stem: strided conv with BN statistics in its epilogue, ReLU,
    # the 3x3 stride-2 pool (its gradient masked by the ReLU)
    "resnet_stem": ([conv(-1, 3, 64, 7, stride=2), bn(0, 64), dict(kind="relu", inputs=[1]),
                     dict(kind="maxpool3s2", inputs=[2])], (30, 28, 3), 2),
    # Inception-V3: factorised 1 x n / n x 1 kernels (same grid, padding on one
    # axis), unpadded convolutions with and without stride, the unpadded pool
    "conv1x7": ([conv(-1, 32, 48, 1, kw=7)], (9, 10, 32), 2),
    "conv7x1": ([conv(-1, 48, 32, 7, kw=1)], (10, 9, 48), 2),
    "conv1x3_bias": ([conv(-1, 64, 40, 1, True, kw=3)], (7, 8, 64), 2),
    "conv3x3_valid": ([conv(-1, 32, 64, 3, pad="valid")], (11, 10, 32), 2),
    "conv3x3_s2_valid": ([conv(-1, 64, 96, 3, stride=2, pad="valid")], (13, 12, 64), 2),
    "conv3x3_s2_valid_c3_stem": ([conv(-1, 3, 32, 3, stride=2, pad="valid")], (23, 21, 3), 2),
    "maxpool3s2_valid": ([dict(kind="maxpool3s2", inputs=[-1], pad="valid")], (13, 12, 64), 2),
    "maxpool3s2_valid_c20": ([dict(kind="maxpool3s2", inputs=[-1], pad="valid")], (12, 11, 20), 2),
    # grid reduction B: strided unpadded branches and a max-pool branch in one concat
    "inception_b_module": (_module("B"), (11, 10, 16), 2),
    # Inception-E: parallel 1x3 / 3x1 convolutions concatenated inside the module concat
    "inception_e_module": (_module("E"), (6, 7, 16), 2),
    # degenerate cases: BN over one sample per channel (variance exactly 0,
    # x_hat = 0, zero input gradient), micro-batch 1, a 7x7 kernel on a 2x2
    # map (padding dominates), strided and unpadded layers down to 1x1 maps
    "bn_single_sample": ([conv(-1, 16, 16, 1), bn(0, 16), dict(kind="relu", inputs=[1])], (1, 1, 16), 1),
    "micro_batch_1": ([conv(-1, 32, 32, 3), bn(0, 32), dict(kind="relu", inputs=[1])], (5, 4, 32), 1),
    "conv7x7_on_2x2": ([conv(-1, 16, 24, 7, True)], (2, 2, 16), 2),
    "to_1x1_maps": ([conv(-1, 16, 32, 3, stride=2), conv(0, 32, 32, 3, pad="valid"),
                     dict(kind="maxpool3s2", inputs=[1])], (5, 6, 16), 2),
    # first bottleneck of a group: strided 3x3, projection shortcut with BN
    # (stored), the last BN taking in the shortcut with the ReLU
    "resnet_block_projection": ([conv(-1, 64, 32, 1), bn(0, 32), dict(kind="relu", inputs=[1]),
                                 conv(2, 32, 32, 3, stride=2), bn(3, 32), dict(kind="relu", inputs=[4]),
                                 conv(-1, 64, 128, 1, stride=2), bn(6, 128),
                                 conv(5, 32, 128, 1), bn(8, 128),
                                 dict(kind="add", inputs=[9, 7]), dict(kind="relu", inputs=[10])],
                                (10, 9, 64), 2),
}


def _workload(name):
    layers, shape, mb = LAYER_CASES[name]
    return wl.StageWorkload(name, layers, mb, 2, shape, 1, 0, 0, 0, minibatches=1, seed=97)


def _errs(g, r):
    e = {}
    for i, (a, b) in enumerate(zip(g.ys, r.ys)):
        e[f"y[{i}]"] = rel_l2(a, b)
    for i, (a, b) in enumerate(zip(g.dxs, r.dxs)):
        e[f"dx[{i}]"] = rel_l2(a, b)
    for k, (a, b) in enumerate(zip(g.grad, r.grad)):
        e[f"grad[{k}]"] = rel_l2(a, b)
    for i, (a, b) in enumerate(zip(g.losses, r.losses)):
        if b is not None:
            e[f"loss[{i}]"] = abs(a - b) / abs(b)
    return e


@pytest.mark.parametrize("dtype", [xp.F32, xp.BF16])
@pytest.mark.parametrize("name", list(LAYER_CASES))
def test_layer_kernels_match_oracle(name, dtype):
    w = _workload(name)
    act = "bf16" if dtype == xp.BF16 else "f32"
    inp = wl.stage_inputs(w, act_dtype=act)
    gpu, _ = run_stage(w, inp, dtype, xp.Hyper(), 0, 0, minibatches=1)
    decisions = any(L["kind"] in ("relu", "maxpool2", "maxpool3s2") for L in w.layers)
    refs = {act: oracle.train_stage(oracle.Stage(w.layers, act), inp.params, inp.m, inp.v, inp.xs,
                                    0, 0, oracle.Hyper(), labels=inp.labels, dys=inp.dys)[0]}
    if dtype == xp.BF16 and not decisions:
        # without ReLU / max-pool decisions the bf16 result is also within the bar
        # of the exact one (with them, bf16 rounding legitimately flips masks)
        refs["f64"] = oracle.train_stage(oracle.Stage(w.layers, "f64"), inp.params, inp.m, inp.v,
                                         inp.xs, 0, 0, oracle.Hyper(), labels=inp.labels,
                                         dys=inp.dys)[0]
    tol = 2e-4 if dtype == xp.F32 else 2e-2
    for mode, r in refs.items():
        e = _errs(gpu[0], r)
        worst = max(e, key=e.get)
        print(f"{name}/{act} vs oracle-{mode}: worst {worst} = {e[worst]:.2e}")
        bad = {k: v for k, v in e.items() if not v <= tol}
        assert not bad, f"vs oracle-{mode}: " + ", ".join(f"{k}={v:.2e}" for k, v in bad.items())


@pytest.mark.parametrize("dtype", [xp.F32, xp.BF16])
@pytest.mark.parametrize("kind,pad,shape", [("maxpool3s2", None, (13, 11, 16)),
                                            ("maxpool3s2", "valid", (12, 13, 16)),
                                            ("maxpool3s2", None, (9, 10, 20)),
                                            ("maxpool2", None, (12, 14, 16)),
                                            ("maxpool2", None, (13, 11, 16)),
                                            ("maxpool2", None, (10, 10, 20))])
def test_maxpool_ties_match_oracle_exactly(kind, pad, shape, dtype):
    """Inputs on five levels, so most windows hold their maximum more than once:
    the output is that maximum and each window's gradient goes to its first
    holder in row-major window order, as the oracle routes it.  Both are exact
    (the gradient sums at most four upstream values), so the comparison is bit
    for bit; C = 20 takes the element-wise kernels, odd sizes the floor of the
    2 x 2 pool."""
    L = dict(kind=kind, inputs=[-1])
    if pad:
        L["pad"] = pad
    w = wl.StageWorkload(kind + "_ties", [L], 2, 2, shape, 1, 0, 0, 0, minibatches=1, seed=23)
    act = "bf16" if dtype == xp.BF16 else "f32"
    inp = wl.stage_inputs(w, act_dtype=act, x_levels=5)
    gpu, _ = run_stage(w, inp, dtype, xp.Hyper(), 0, 0, minibatches=1)
    ref = oracle.train_stage(oracle.Stage(w.layers, act), inp.params, inp.m, inp.v, inp.xs, 0, 0,
                             oracle.Hyper(), labels=inp.labels, dys=inp.dys)[0]
    x = inp.xs[0][0]
    assert len(np.unique(x)) <= 5
    for i in range(w.T):
        np.testing.assert_array_equal(np.asarray(gpu[0].ys[i], np.float64).reshape(ref.ys[i].shape),
                                      np.asarray(ref.ys[i], np.float64))
        np.testing.assert_array_equal(np.asarray(gpu[0].dxs[i], np.float64).reshape(ref.dxs[i].shape),
                                      np.asarray(ref.dxs[i], np.float64))

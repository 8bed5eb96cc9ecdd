"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle.

This module holds data only: the layer lists of the stages measured here, the
parameter shapes they imply, and seeded random draws of parameters, inputs,
labels and upstream gradients.  It performs none of the method's arithmetic
(no prediction, no optimizer step, no layer math), so both the CPU oracle and
the GPU path may consume it without sharing any computation.

Stage layer lists follow the paper's setup (Sec. IV-C): VGG-16, ResNet-101 and
Inception-V3 stages, CIFAR-10 / Tiny-ImageNet-shaped tensors replaced by
synthetic normal data.  Seed 1 is the paper's shuffling seed (Sec. IV-C); the
i-th workload below uses seed 1 + i.

Layer spec (a plain dict, one per layer, in execution order):
  kind     one of linear, conv, bn, relu, add, maxpool2, avgpool3, gap, concat,
           softmax_ce
  inputs   list of producer layer indices; -1 is the stage input
  cin/cout channel counts (linear, conv); k = kernel size (conv, odd; padding
           k//2, stride 1); bias (linear, conv); classes (softmax_ce)
Parameters are ordered by layer, and within a layer weight then bias (conv,
linear) or gamma then beta (bn).  Conv weights are [cout, k, k, cin]; linear
weights are [cout, cin].  Activations are NHWC (or [n, C] once flattened).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

PAPER_SEED = 1  # the data-shuffling seed the paper states (Sec. IV-C)


# ----------------------------------------------------------------------------
# layer-list builders
# ----------------------------------------------------------------------------
class _Builder:
    def __init__(self):
        self.layers: List[dict] = []

    def add(self, **kw) -> int:
        self.layers.append(kw)
        return len(self.layers) - 1

    def linear(self, x, cin, cout, bias=True):
        return self.add(kind="linear", inputs=[x], cin=cin, cout=cout, bias=bias)

    def conv(self, x, cin, cout, k, bias=False, stride=1, kw=None, pad="same"):
        """k x kw kernel (kw defaults to k); pad "same" (k//2, kw//2) or "valid" (none)."""
        L = dict(kind="conv", inputs=[x], cin=cin, cout=cout, k=k, bias=bias, stride=stride)
        if kw is not None and kw != k:
            L["kw"] = kw
        if pad != "same":
            L["pad"] = pad
        return self.add(**L)

    def bn(self, x, c):
        return self.add(kind="bn", inputs=[x], cin=c, cout=c)

    def relu(self, x):
        return self.add(kind="relu", inputs=[x])

    def conv_bn_relu(self, x, cin, cout, k, stride=1, kw=None, pad="same"):
        return self.relu(self.bn(self.conv(x, cin, cout, k, stride=stride, kw=kw, pad=pad), cout))


def mlp_stage_layers(d_in=256, d_hidden=256, classes=10) -> List[dict]:
    b = _Builder()
    h = b.relu(b.linear(-1, d_in, d_hidden))
    z = b.linear(h, d_hidden, classes)
    b.add(kind="softmax_ce", inputs=[z], classes=classes)
    return b.layers


def vgg_stage_layers(bias=True) -> List[dict]:
    """First of four VGG-16 stages: two conv blocks of (conv3x3+ReLU)x2 + maxpool."""
    b = _Builder()
    x = b.relu(b.conv(-1, 3, 64, 3, bias=bias))
    x = b.relu(b.conv(x, 64, 64, 3, bias=bias))
    x = b.add(kind="maxpool2", inputs=[x])
    x = b.relu(b.conv(x, 64, 128, 3, bias=bias))
    x = b.relu(b.conv(x, 128, 128, 3, bias=bias))
    b.add(kind="maxpool2", inputs=[x])
    return b.layers


def vgg16_layers(classes=10) -> List[dict]:
    """VGG-16 for 32x32 inputs (Sec. IV-C's CIFAR-10 model): thirteen 3x3
    convolutions with bias and ReLU in five blocks, each closed by a 2x2 max
    pool (32 -> 1), then a linear classifier and the cross-entropy loss."""
    b = _Builder()
    x, cin = -1, 3
    for widths in ((64, 64), (128, 128), (256, 256, 256), (512, 512, 512), (512, 512, 512)):
        for c in widths:
            x = b.relu(b.conv(x, cin, c, 3, bias=True))
            cin = c
        x = b.add(kind="maxpool2", inputs=[x])
    z = b.linear(x, 512, classes)
    b.add(kind="softmax_ce", inputs=[z], classes=classes)
    return b.layers


def split_layers(layers: List[dict], first: List[int]) -> List[List[dict]]:
    """Per-stage layer lists for stage boundaries `first` (first[k] = stage k's
    first layer, last entry = len(layers)): inputs re-indexed within the stage,
    the previous stage's last layer becoming the stage input -1.

    A stage whose max pool reads the stage input, when the previous stage ends
    in ReLU outputs (a ReLU or a concat of them), starts with a ReLU on its
    input: the identity on those values, it marks the input as a ReLU output so
    that a concat of the pool with ReLU branches (Inception-V3's grid
    reductions) is masked as one tensor.  It changes no value and no weight
    gradient; only the stage-input gradient at the input's zeros, which the
    previous stage's ReLU zeroes anyway."""
    def relu_out(j):
        L = layers[j]
        return L["kind"] == "relu" or (L["kind"] == "concat" and all(relu_out(q) for q in L["inputs"]))

    out = []
    for k in range(len(first) - 1):
        a, b = first[k], first[k + 1]
        stage = []
        for L in layers[a:b]:
            L = dict(L)
            L["inputs"] = [-1 if (j == a - 1 or j == -1) else j - a for j in L["inputs"]]
            stage.append(L)
        pools_input = any(L["kind"] in ("maxpool2", "maxpool3s2") and L["inputs"] == [-1] for L in stage)
        if a > 0 and pools_input and relu_out(a - 1):
            shifted = [dict(kind="relu", inputs=[-1])]
            for L in stage:
                L = dict(L)
                L["inputs"] = [j + 1 for j in L["inputs"]]  # -1 -> 0: the ReLU
                shifted.append(L)
            stage = shifted
        out.append(stage)
    return out


def resnet101_layers(classes=200, blocks=(3, 4, 23, 3)) -> List[dict]:
    """ResNet-101 (Sec. IV-C's Tiny ImageNet model, inputs scaled to 224 x 224):
    a 7x7 stride-2 stem convolution with BN and ReLU, a 3x3 stride-2 max pool,
    four groups of bottleneck blocks (1x1, 3x3, 1x1 with 4x expansion; BN after
    each convolution) whose first block strides by 2 on its 3x3 convolution
    (groups 2-4) and adds a 1x1 projection with BN on the shortcut, then global
    average pooling, the linear classifier and the cross-entropy loss.  Within
    a block the projection comes before the third convolution, so that the
    third BN takes in the shortcut (BN + add + ReLU)."""
    b = _Builder()
    x = b.conv_bn_relu(-1, 3, 64, 7, stride=2)
    x = b.add(kind="maxpool3s2", inputs=[x])
    cin = 64
    for g, nblk in enumerate(blocks):
        mid = 64 << g
        for j in range(nblk):
            stride = 2 if (j == 0 and g > 0) else 1
            y = b.conv_bn_relu(x, cin, mid, 1)
            y = b.conv_bn_relu(y, mid, mid, 3, stride=stride)
            sc = x
            if j == 0:
                sc = b.bn(b.conv(x, cin, 4 * mid, 1, stride=stride), 4 * mid)
            y = b.bn(b.conv(y, mid, 4 * mid, 1), 4 * mid)
            x = b.relu(b.add(kind="add", inputs=[y, sc]))
            cin = 4 * mid
    g_ = b.add(kind="gap", inputs=[x])
    z = b.linear(g_, cin, classes)
    b.add(kind="softmax_ce", inputs=[z], classes=classes)
    return b.layers


def inception_v3_layers(classes=200) -> List[dict]:
    """Inception-V3 (Sec. IV-C's Tiny ImageNet model, inputs scaled to 224 x
    224), as defined by its authors: every convolution followed by BN and ReLU;
    an unpadded stem (3x3 stride 2, 3x3, padded 3x3, 3x3 stride-2 max pool,
    1x1, 3x3, 3x3 stride-2 max pool); three Inception-A modules (1x1 | 1x1 ->
    5x5 | 1x1 -> 3x3 -> 3x3 | 3x3 average pool -> 1x1); the grid reduction B;
    four Inception-C modules with factorised 1x7 / 7x1 convolutions; the grid
    reduction D; two Inception-E modules whose 3x3 branches end in parallel
    1x3 and 3x1 convolutions; global average pooling, the classifier and the
    cross-entropy loss (no auxiliary head)."""
    b = _Builder()
    cbr = b.conv_bn_relu
    x = cbr(-1, 3, 32, 3, stride=2, pad="valid")
    x = cbr(x, 32, 32, 3, pad="valid")
    x = cbr(x, 32, 64, 3)
    x = b.add(kind="maxpool3s2", inputs=[x], pad="valid")
    x = cbr(x, 64, 80, 1)
    x = cbr(x, 80, 192, 3, pad="valid")
    x = b.add(kind="maxpool3s2", inputs=[x], pad="valid")
    cin = 192
    for pool_f in (32, 64, 64):                       # Inception-A
        b1 = cbr(x, cin, 64, 1)
        b2 = cbr(cbr(x, cin, 48, 1), 48, 64, 5)
        b3 = cbr(cbr(cbr(x, cin, 64, 1), 64, 96, 3), 96, 96, 3)
        b4 = cbr(b.add(kind="avgpool3", inputs=[x]), cin, pool_f, 1)
        x = b.add(kind="concat", inputs=[b1, b2, b3, b4])
        cin = 64 + 64 + 96 + pool_f
    b1 = cbr(x, cin, 384, 3, stride=2, pad="valid")   # grid reduction B
    b2 = cbr(cbr(cbr(x, cin, 64, 1), 64, 96, 3), 96, 96, 3, stride=2, pad="valid")
    b3 = b.add(kind="maxpool3s2", inputs=[x], pad="valid")
    x = b.add(kind="concat", inputs=[b1, b2, b3])
    cin = 384 + 96 + cin
    for c7 in (128, 160, 160, 192):                   # Inception-C
        b1 = cbr(x, cin, 192, 1)
        b2 = cbr(cbr(cbr(x, cin, c7, 1), c7, c7, 1, kw=7), c7, 192, 7, kw=1)
        b3 = cbr(x, cin, c7, 1)
        b3 = cbr(b3, c7, c7, 7, kw=1)
        b3 = cbr(b3, c7, c7, 1, kw=7)
        b3 = cbr(b3, c7, c7, 7, kw=1)
        b3 = cbr(b3, c7, 192, 1, kw=7)
        b4 = cbr(b.add(kind="avgpool3", inputs=[x]), cin, 192, 1)
        x = b.add(kind="concat", inputs=[b1, b2, b3, b4])
        cin = 768
    b1 = cbr(cbr(x, cin, 192, 1), 192, 320, 3, stride=2, pad="valid")   # grid reduction D
    b2 = cbr(cbr(cbr(cbr(x, cin, 192, 1), 192, 192, 1, kw=7), 192, 192, 7, kw=1),
             192, 192, 3, stride=2, pad="valid")
    b3 = b.add(kind="maxpool3s2", inputs=[x], pad="valid")
    x = b.add(kind="concat", inputs=[b1, b2, b3])
    cin = 320 + 192 + cin
    for _ in range(2):                                # Inception-E
        b1 = cbr(x, cin, 320, 1)
        t = cbr(x, cin, 384, 1)
        b2 = b.add(kind="concat", inputs=[cbr(t, 384, 384, 1, kw=3), cbr(t, 384, 384, 3, kw=1)])
        t = cbr(cbr(x, cin, 448, 1), 448, 384, 3)
        b3 = b.add(kind="concat", inputs=[cbr(t, 384, 384, 1, kw=3), cbr(t, 384, 384, 3, kw=1)])
        b4 = cbr(b.add(kind="avgpool3", inputs=[x]), cin, 192, 1)
        x = b.add(kind="concat", inputs=[b1, b2, b3, b4])
        cin = 2048
    g_ = b.add(kind="gap", inputs=[x])
    z = b.linear(g_, cin, classes)
    b.add(kind="softmax_ce", inputs=[z], classes=classes)
    return b.layers


def resnet_stage_layers(blocks=8, c=512, mid=128) -> List[dict]:
    """Middle ResNet-101 stage: bottlenecks with identity shortcut."""
    b = _Builder()
    x = -1
    for _ in range(blocks):
        y = b.conv_bn_relu(x, c, mid, 1)
        y = b.conv_bn_relu(y, mid, mid, 3)
        y = b.bn(b.conv(y, mid, c, 1), c)
        x = b.relu(b.add(kind="add", inputs=[y, x]))
    return b.layers


def inception_stage_layers(modules=3, cin=256, classes=200) -> List[dict]:
    """Inception-V3-style stage: Inception-A modules, then GAP, linear head, CE."""
    b = _Builder()
    x = -1
    for _ in range(modules):
        b1 = b.conv_bn_relu(x, cin, 64, 1)
        b2 = b.conv_bn_relu(b.conv_bn_relu(x, cin, 48, 1), 48, 64, 5)
        b3 = b.conv_bn_relu(x, cin, 64, 1)
        b3 = b.conv_bn_relu(b3, 64, 96, 3)
        b3 = b.conv_bn_relu(b3, 96, 96, 3)
        p = b.add(kind="avgpool3", inputs=[x])
        b4 = b.conv_bn_relu(p, cin, 32, 1)
        x = b.add(kind="concat", inputs=[b1, b2, b3, b4])
        cin = 64 + 64 + 96 + 32
    g = b.add(kind="gap", inputs=[x])
    z = b.linear(g, cin, classes)
    b.add(kind="softmax_ce", inputs=[z], classes=classes)
    return b.layers


def param_shapes(layers: List[dict]) -> List[tuple]:
    """Shapes of the parameter tensors, in buffer order."""
    shapes = []
    for L in layers:
        if L["kind"] == "linear":
            shapes.append((L["cout"], L["cin"]))
            if L["bias"]:
                shapes.append((L["cout"],))
        elif L["kind"] == "conv":
            shapes.append((L["cout"], L["k"], L.get("kw", L["k"]), L["cin"]))
            if L["bias"]:
                shapes.append((L["cout"],))
        elif L["kind"] == "bn":
            shapes.append((L["cout"],))
            shapes.append((L["cout"],))
    return shapes


def param_roles(layers: List[dict]) -> List[tuple]:
    """(layer index, role) per parameter tensor; role in weight/bias/gamma/beta."""
    roles = []
    for i, L in enumerate(layers):
        if L["kind"] in ("linear", "conv"):
            roles.append((i, "weight"))
            if L["bias"]:
                roles.append((i, "bias"))
        elif L["kind"] == "bn":
            roles.append((i, "gamma"))
            roles.append((i, "beta"))
    return roles


# ----------------------------------------------------------------------------
# workload descriptions
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class StageWorkload:
    name: str
    layers: List[dict]
    micro_batch: int
    T: int                      # micro-batches per mini-batch
    in_shape: tuple             # per-sample input shape (H, W, C) or (C,)
    size: int                   # pipeline stages (GPUs) in the paper's setting
    rank: int                   # this stage's rank
    s_fwd: int                  # version difference for the forward bellwether
    s_bwd: int                  # version difference for the backward bellwether
    minibatches: int = 3
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    dy_std: float = 1e-2        # upstream gradient N(0, dy_std) for stages without a loss
    seed: int = PAPER_SEED

    @property
    def has_loss(self) -> bool:
        return self.layers[-1]["kind"] == "softmax_ce"

    @property
    def classes(self) -> Optional[int]:
        return self.layers[-1]["classes"] if self.has_loss else None

    @property
    def spatial(self) -> bool:
        return len(self.in_shape) == 3


def tiny_mlp() -> StageWorkload:
    return StageWorkload("tiny_mlp", mlp_stage_layers(), 32, 4, (256,), 1, 0, 2, 2,
                         seed=PAPER_SEED + 0)


def vgg_stage() -> StageWorkload:
    # rank 0 of 4 stages, T=4: Eq.1 gives 2 (round half up), Eq.2 gives 1.
    return StageWorkload("vgg16_stage0", vgg_stage_layers(), 32, 4, (32, 32, 3), 4, 0, 2, 1,
                         seed=PAPER_SEED + 2)


def resnet_stage() -> StageWorkload:
    return StageWorkload("resnet101_mid_stage", resnet_stage_layers(), 32, 4, (16, 16, 512),
                         4, 1, 1, 1, seed=PAPER_SEED + 3)


def inception_stage() -> StageWorkload:
    return StageWorkload("inception_v3_stage", inception_stage_layers(), 32, 4, (35, 35, 256),
                         4, 3, 1, 1, seed=PAPER_SEED + 4)


WORKLOADS = {
    "tiny_mlp": tiny_mlp,
    "vgg16_stage0": vgg_stage,
    "resnet101_mid_stage": resnet_stage,
    "inception_v3_stage": inception_stage,
}


def shrink(w: StageWorkload, micro_batch=None, spatial=None, T=None, minibatches=None,
           layers=None, in_shape=None) -> StageWorkload:
    """A smaller copy of a workload (test sizes); layers/in_shape may be replaced."""
    w = dataclasses.replace(w)
    if micro_batch is not None:
        w.micro_batch = micro_batch
    if T is not None:
        w.T = T
    if minibatches is not None:
        w.minibatches = minibatches
    if layers is not None:
        w.layers = layers
    if in_shape is not None:
        w.in_shape = in_shape
    elif spatial is not None and w.spatial:
        w.in_shape = (spatial[0], spatial[1], w.in_shape[2])
    return w


# ----------------------------------------------------------------------------
# seeded draws
# ----------------------------------------------------------------------------
def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 values -> nearest bfloat16 values (ties to even), returned as fp32.

    A storage-format conversion used to hand both sides identical bf16 inputs.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), a, out)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """bf16-representable fp32 values -> their 16-bit patterns (uint16)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def init_params(layers: List[dict], rng: np.random.Generator) -> List[np.ndarray]:
    """Kaiming-uniform weights U(-sqrt(6/fan_in), +sqrt(6/fan_in)), zero biases,
    BN gamma 1 and beta 0.  fp32 values."""
    out = []
    for shape, (li, role) in zip(param_shapes(layers), param_roles(layers)):
        if role == "weight":
            fan_in = int(np.prod(shape[1:]))
            bound = math.sqrt(6.0 / fan_in)
            out.append(rng.uniform(-bound, bound, size=shape).astype(np.float32))
        elif role == "gamma":
            out.append(np.ones(shape, np.float32))
        else:
            out.append(np.zeros(shape, np.float32))
    return out


@dataclasses.dataclass
class StageInputs:
    params: List[np.ndarray]          # fp32 master weights, one array per tensor
    m: List[np.ndarray]               # first moments (fp32)
    v: List[np.ndarray]               # second moments (fp32)
    xs: List[List[np.ndarray]]        # [minibatch][micro-batch] stage inputs (fp32 values)
    labels: Optional[List[List[np.ndarray]]]  # int32 labels for stages with a loss
    dys: Optional[List[List[np.ndarray]]]     # upstream gradients for stages without one


def stage_inputs(w: StageWorkload, act_dtype: str = "f32", moment_init: str = "zeros",
                 seed: Optional[int] = None, x_levels: Optional[int] = None) -> StageInputs:
    """Draw params, moments, inputs, labels/dy in that fixed order from PCG64(seed).

    act_dtype "bf16" rounds inputs and upstream gradients to bf16 values (the
    storage format of that variant); parameters stay fp32 masters.
    moment_init "paper" draws both moments as 1e-4 * U(0, 1) (Sec. IV-C).
    x_levels = L draws the inputs as integers uniform in [-(L // 2), L // 2]
    instead of N(0, 1) (exact in either format; equal values are common).
    """
    rng = np.random.default_rng(w.seed if seed is None else seed)
    params = init_params(w.layers, rng)
    if moment_init == "zeros":
        m = [np.zeros_like(p) for p in params]
        v = [np.zeros_like(p) for p in params]
    elif moment_init == "paper":
        m = [(1e-4 * rng.uniform(0.0, 1.0, size=p.shape)).astype(np.float32) for p in params]
        v = [(1e-4 * rng.uniform(0.0, 1.0, size=p.shape)).astype(np.float32) for p in params]
    else:
        raise ValueError(moment_init)
    conv = (lambda a: round_to_bf16(a)) if act_dtype == "bf16" else (lambda a: a)
    shape = (w.micro_batch,) + tuple(w.in_shape)
    if x_levels:
        draw = lambda: rng.integers(-(x_levels // 2), x_levels // 2 + 1, size=shape).astype(np.float32)
    else:
        draw = lambda: rng.standard_normal(shape).astype(np.float32)
    xs = [[conv(draw()) for _ in range(w.T)] for _ in range(w.minibatches)]
    labels = dys = None
    if w.has_loss:
        labels = [[rng.integers(0, w.classes, size=w.micro_batch).astype(np.int32)
                   for _ in range(w.T)] for _ in range(w.minibatches)]
    else:
        out_shape = stage_output_shape(w)
        dys = [[conv((w.dy_std * rng.standard_normal(out_shape)).astype(np.float32))
                for _ in range(w.T)] for _ in range(w.minibatches)]
    return StageInputs(params, m, v, xs, labels, dys)


def exact_stage_inputs(w: StageWorkload, seed: Optional[int] = None, two_point: bool = False,
                       x_levels: int = 5, dy_levels: int = 7, dy_scale: float = 2.0 ** -8) -> StageInputs:
    """Inputs on which the bf16 variant's stored values are unique: every
    product and partial sum of a forward contraction is an exact fp32 value,
    so an fp32-accumulating kernel and an fp64 reference store the same bits,
    and equal values (max-pool ties) are compared exactly on both sides.

      weights     conv / linear weights +-1 (random signs), no biases (a bias
                  update is an fp32 value that no grid keeps exact); BN gamma 1,
                  beta 0;
      moments     the paper's initialisation 1e-4 * U(0, 1) (Sec. IV-C);
      inputs      integers uniform in [-(x_levels // 2), x_levels // 2];
                  with two_point, each micro-batch holds two such input
                  vectors, alternating over its samples (even micro-batch), so
                  that every BN channel sees exactly two values, equally often:
                  its normalised outputs are +-d / sqrt(d^2 + eps), which bf16
                  stores as +-1 (or 0 when d = 0), keeping the next contraction
                  on integers (use with 1 x 1 maps, where a padded k x k
                  convolution reduces to its centre tap);
      upstream    integers in [-(dy_levels // 2), dy_levels // 2] times dy_scale;
      labels      uniform.

    Integer activations stay exact in fp32 while every partial sum is below
    2^24.  A learning rate small enough that |W_hat - W| stays under half a
    bf16 ulp of 1 keeps the bf16 weight operands at +-1 in later mini-batches
    (the fp32 master weights, moments and predictions still move)."""
    rng = np.random.default_rng(w.seed if seed is None else seed)
    params = []
    for shape, (li, role) in zip(param_shapes(w.layers), param_roles(w.layers)):
        if role == "weight":
            params.append(np.where(rng.integers(0, 2, size=shape) == 1, 1.0, -1.0).astype(np.float32))
        elif role == "gamma":
            params.append(np.ones(shape, np.float32))
        else:
            params.append(np.zeros(shape, np.float32))
    m = [(1e-4 * rng.uniform(0.0, 1.0, size=p.shape)).astype(np.float32) for p in params]
    v = [(1e-4 * rng.uniform(0.0, 1.0, size=p.shape)).astype(np.float32) for p in params]
    shape = (w.micro_batch,) + tuple(w.in_shape)
    half = x_levels // 2

    def draw():
        if not two_point:
            return rng.integers(-half, half + 1, size=shape).astype(np.float32)
        assert w.micro_batch % 2 == 0, "two-point inputs need an even micro-batch"
        uv = rng.integers(-half, half + 1, size=(2,) + tuple(w.in_shape)).astype(np.float32)
        return np.stack([uv[i % 2] for i in range(w.micro_batch)])

    xs = [[draw() for _ in range(w.T)] for _ in range(w.minibatches)]
    labels = dys = None
    if w.has_loss:
        labels = [[rng.integers(0, w.classes, size=w.micro_batch).astype(np.int32)
                   for _ in range(w.T)] for _ in range(w.minibatches)]
    else:
        out_shape = stage_output_shape(w)
        dh = dy_levels // 2
        dys = [[(dy_scale * rng.integers(-dh, dh + 1, size=out_shape)).astype(np.float32)
                for _ in range(w.T)] for _ in range(w.minibatches)]
    return StageInputs(params, m, v, xs, labels, dys)


def stage_output_shape(w: StageWorkload) -> tuple:
    """Shape of the stage output for one micro-batch (shape bookkeeping only)."""
    shapes: Dict[int, tuple] = {-1: (w.micro_batch,) + tuple(w.in_shape)}
    for i, L in enumerate(w.layers):
        s = shapes[L["inputs"][0]]
        k = L["kind"]
        if k in ("linear",):
            shapes[i] = s[:-1] + (L["cout"],)
        elif k == "conv":
            st, kh, kw = L.get("stride", 1), L["k"], L.get("kw", L["k"])
            ph, pw = (0, 0) if L.get("pad", "same") == "valid" else (kh // 2, kw // 2)
            shapes[i] = (s[0], (s[1] + 2 * ph - kh) // st + 1, (s[2] + 2 * pw - kw) // st + 1, L["cout"])
        elif k == "maxpool2":
            shapes[i] = (s[0], s[1] // 2, s[2] // 2, s[3])
        elif k == "maxpool3s2":
            p = 0 if L.get("pad", "same") == "valid" else 1
            shapes[i] = (s[0], (s[1] + 2 * p - 3) // 2 + 1, (s[2] + 2 * p - 3) // 2 + 1, s[3])
        elif k == "gap":
            shapes[i] = (s[0], s[3])
        elif k == "concat":
            shapes[i] = s[:-1] + (sum(shapes[j][-1] for j in L["inputs"]),)
        elif k == "softmax_ce":
            shapes[i] = ()
        else:
            shapes[i] = s
    return shapes[len(w.layers) - 1]


@dataclasses.dataclass
class FlatState:
    W: np.ndarray
    m: np.ndarray
    v: np.ndarray
    G: np.ndarray


def flat_state(n: int, seed: int = PAPER_SEED + 1) -> FlatState:
    """Flat fp32 buffers for the prediction/Adam sweep: W~N(0,0.02), m~N(0,1e-3),
    v=|N(0,1e-6)|, G~N(0,1e-3) (standard deviations), drawn in that order."""
    rng = np.random.default_rng(seed)
    W = rng.standard_normal(n, dtype=np.float32); W *= np.float32(0.02)
    m = rng.standard_normal(n, dtype=np.float32); m *= np.float32(1e-3)
    v = rng.standard_normal(n, dtype=np.float32); np.abs(v, out=v); v *= np.float32(1e-6)
    G = rng.standard_normal(n, dtype=np.float32); G *= np.float32(1e-3)
    return FlatState(W, m, v, G)


def rule_state(n: int, seed: int = PAPER_SEED + 6):
    """Optimizer buffers of the momentum-SGD / RMSProp rules, continuing a run:
    momentum buffer ~N(0,1e-3), squared-gradient average |N(0,1e-6)| (standard
    deviations), drawn in that order.  Returns (buf, sq) fp32."""
    rng = np.random.default_rng(seed)
    buf = rng.standard_normal(n, dtype=np.float32); buf *= np.float32(1e-3)
    sq = rng.standard_normal(n, dtype=np.float32); np.abs(sq, out=sq); sq *= np.float32(1e-6)
    return buf, sq

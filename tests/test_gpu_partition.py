"""Whole networks partitioned into four stages by Sec. IV-B's rule, run
stage by stage on the GPU library (the activation of stage k is the input of
stage k + 1, the input gradient of stage k + 1 the upstream gradient of stage
k) against the oracle's forward and backward of the unpartitioned network.
fp32 storage, s = 0: logits, loss and every weight gradient within 2e-4.
VGG-16 at 32 x 32 (CIFAR-10); ResNet-101 at 64 x 64 (its strided stem, pool,
projections and 33 bottlenecks; 2 x 2 maps in the last group keep the
micro-batch BNs well conditioned); Inception-V3 at 139 x 139 (3 x 3 maps in the
last modules)."""
import numpy as np
import pytest

import oracle
import paper_1911_04610_amd as xp
import workloads as wl
from conftest import rel_l2
from gpu_harness import to_device, to_host

pytestmark = pytest.mark.gpu


NETS = {"vgg16": (wl.vgg16_layers, (32, 32, 3)), "resnet101": (wl.resnet101_layers, (64, 64, 3)),
        "inception_v3": (wl.inception_v3_layers, (139, 139, 3))}


@pytest.mark.parametrize("net", list(NETS))
def test_partitioned_network_matches_unpartitioned_oracle(net):
    import torch
    build, in_shape = NETS[net]
    layers = build()
    w = wl.StageWorkload(net + "_full", layers, 2, 1, in_shape, 4, 0, 0, 0, minibatches=1)
    inp = wl.stage_inputs(w, act_dtype="f32")
    x, labels = inp.xs[0][0], inp.labels[0][0]
    first = xp.xpipe_partition(layers, 4)
    parts = wl.split_layers(layers, first)
    counts = [len(wl.param_shapes(p)) for p in parts]
    offs = np.cumsum([0] + counts)
    hp = xp.Hyper()
    stages, ins, outs = [], [to_device(x, xp.F32)], []
    lab = torch.from_numpy(labels).cuda()
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    for k, p in enumerate(parts):
        st = xp.Stage(p, w.micro_batch, 1, in_shape, xp.F32)
        st.set_flat(st.W, inp.params[offs[k]:offs[k + 1]])
        st.xpipe_predict_weights(xp.FWD, 0, hp, 0)
        st.xpipe_predict_weights(xp.BWD, 0, hp, 0)
        n, H, W_, C = st.out_shape
        y = torch.empty((n, H, W_, C), dtype=torch.float32, device="cuda")
        last = k == len(parts) - 1
        st.xpipe_stage_fwd(ins[-1], y, lab if last else None, loss if last else None)
        stages.append(st)
        outs.append(y)
        ins.append(y)
        in_shape = (H, W_, C)
    dy = None
    for k in reversed(range(len(parts))):
        st = stages[k]
        dx = torch.empty_like(ins[k]) if k > 0 else None
        st.xpipe_stage_bwd(ins[k], dy, lab if k == len(parts) - 1 else None, dx)
        dy = dx
    torch.cuda.synchronize()
    grads = [g for st in stages for g in st.get_tensors(st.grad)]

    ref = oracle.Stage(layers, "f32")
    z, ref_loss, _ = ref.forward(inp.params, x, labels, w.micro_batch)
    _, ref_grads, _ = ref.backward(inp.params, x, None, labels, w.micro_batch, False)
    errs = {"logits": rel_l2(to_host(outs[-1]).reshape(z.shape), z),
            "loss": abs(float(loss[0]) - ref_loss) / abs(ref_loss)}
    for q, (a, b) in enumerate(zip(grads, ref_grads)):
        errs[f"grad[{q}]"] = rel_l2(a, b)
    worst = max(errs, key=errs.get)
    print(f"partitioned {net} {first}: worst {worst} = {errs[worst]:.2e}")
    assert all(v <= 2e-4 for v in errs.values()), {k: v for k, v in errs.items() if v > 2e-4}

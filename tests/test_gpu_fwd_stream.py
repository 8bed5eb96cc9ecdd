"""Forward passes on a stream of their own (xpipe_stage_set_fwd_stream).

In the pipeline's steady state a stage alternates the forward of one
micro-batch with the backward of another (Sec. III-A); with the forwards on a
second stream and a workspace of their own the two run concurrently.  The
results must be bit-identical to the same calls on one stream: every forward
output and loss, every input gradient, and W, m, v and both predictions after
each update.  The calls are issued both as forward/backward pairs (the
steady-state order of the last stage) and as all forwards then all
backwards, with recorded passes and eagerly."""
import pytest

import paper_1911_04610_amd as xp
import workloads as wl
from gpu_harness import to_device

pytestmark = pytest.mark.gpu

SMALL = {
    "tiny_mlp": lambda: wl.tiny_mlp(),
    "vgg16_stage0": lambda: wl.shrink(wl.vgg_stage(), micro_batch=4, spatial=(20, 20), T=2,
                                      minibatches=2),
    "resnet101_mid_stage": lambda: wl.shrink(
        wl.resnet_stage(), micro_batch=2, T=2, minibatches=2,
        layers=wl.resnet_stage_layers(blocks=2), in_shape=(9, 9, 512)),
    "inception_v3_stage": lambda: wl.shrink(
        wl.inception_stage(), micro_batch=2, T=3, minibatches=2,
        layers=wl.inception_stage_layers(modules=2), in_shape=(9, 9, 256)),
}


def _run(w, inp, dtype, overlap, order, graphs=True):
    import torch
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dtype)
    st.set_graphs(graphs)
    st.set_flat(st.W, inp.params)
    st.set_flat(st.m, inp.m)
    st.set_flat(st.v, inp.v)
    if overlap:
        assert st.xpipe_stage_set_fwd_stream(True) is not None
    J, T = len(inp.xs), w.T
    xs = [[to_device(x, dtype) for x in row] for row in inp.xs]
    labels = None if inp.labels is None else [[torch.from_numpy(l).cuda() for l in row]
                                              for row in inp.labels]
    dys = None if inp.dys is None else [[to_device(d, dtype) for d in row] for row in inp.dys]
    tdt = torch.bfloat16 if dtype == xp.BF16 else torch.float32
    ys = [[torch.empty(st.out_shape, dtype=tdt, device="cuda") for _ in range(T)] for _ in range(J)]
    loss = torch.zeros((J, T), dtype=torch.float32, device="cuda")
    dxs = [[torch.empty((w.micro_batch,) + tuple(w.in_shape), dtype=tdt, device="cuda")
            for _ in range(T)] for _ in range(J)]
    torch.cuda.synchronize()
    hp = xp.Hyper()
    snaps = []

    def fwd(j, i):
        st.xpipe_stage_fwd(xs[j][i], ys[j][i], None if labels is None else labels[j][i],
                           loss[j, i:i + 1] if w.has_loss else None)

    def bwd(j, i):
        st.xpipe_stage_bwd(xs[j][i], None if dys is None else dys[j][i],
                           None if labels is None else labels[j][i], dxs[j][i])

    for j in range(J):
        if j == 0:
            st.xpipe_predict_weights(xp.FWD, w.s_fwd, hp, 0)
            st.xpipe_predict_weights(xp.BWD, w.s_bwd, hp, 0)
        if order == "pairs":
            for i in range(T):
                fwd(j, i)
                bwd(j, i)
        else:
            for i in range(T):
                fwd(j, i)
            for i in range(T):
                bwd(j, i)
        st.xpipe_adam_step(hp, j, w.s_fwd, w.s_bwd, emit_pred=True)
        # on the stage's stream, after the update (which waited for the forwards)
        snaps.append([t.clone() for t in (st.W, st.m, st.v, st.w_pred_fwd, st.w_pred_bwd)])
    torch.cuda.synchronize()
    return ys, loss, dxs, snaps


def _assert_same(a, b):
    import torch
    ya, la, da, sa = a
    yb, lb, db, sb = b
    for j in range(len(ya)):
        for i in range(len(ya[j])):
            assert torch.equal(ya[j][i], yb[j][i]), f"y[{j}][{i}]"
            assert torch.equal(da[j][i], db[j][i]), f"dx[{j}][{i}]"
        for k, name in enumerate(("W", "m", "v", "w_pred_fwd", "w_pred_bwd")):
            assert torch.equal(sa[j][k], sb[j][k]), f"{name} after update {j}"
    assert torch.equal(la, lb), "loss"


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("dtype", [xp.F32, xp.BF16])
def test_forward_stream_matches_one_stream(name, dtype):
    w = SMALL[name]()
    inp = wl.stage_inputs(w, act_dtype="bf16" if dtype == xp.BF16 else "f32", moment_init="paper")
    ref = _run(w, inp, dtype, overlap=False, order="pairs")
    _assert_same(_run(w, inp, dtype, overlap=True, order="pairs"), ref)
    _assert_same(_run(w, inp, dtype, overlap=True, order="all"), ref)


def test_forward_stream_eager_matches_one_stream():
    w = SMALL["inception_v3_stage"]()
    inp = wl.stage_inputs(w, act_dtype="bf16", moment_init="paper")
    ref = _run(w, inp, xp.BF16, overlap=False, order="pairs", graphs=False)
    _assert_same(_run(w, inp, xp.BF16, overlap=True, order="pairs", graphs=False), ref)


def test_forward_stream_full_size_inception_a():
    """The benchmarked stage (three Inception-A modules and the head at
    32 x 35 x 35, T = 4, bf16), two mini-batches in forward/backward pairs:
    the configuration the benchmark times."""
    w = wl.shrink(wl.inception_stage(), minibatches=2)
    inp = wl.stage_inputs(w, act_dtype="bf16", moment_init="paper")
    ref = _run(w, inp, xp.BF16, overlap=False, order="pairs")
    _assert_same(_run(w, inp, xp.BF16, overlap=True, order="pairs"), ref)


def test_forward_stream_arguments():
    import torch
    import ctypes
    w = SMALL["tiny_mlp"]()
    s0 = torch.cuda.Stream()
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32, stream=s0)
    L = xp.lib()
    buf = torch.empty(st.ws_bytes + 512, dtype=torch.uint8, device="cuda")
    base = (buf.data_ptr() + 255) // 256 * 256
    fs = ctypes.c_void_p(1)
    assert L.xpipe_stage_set_fwd_stream(st._h, base, st.ws_bytes - 1, ctypes.byref(fs)) == xp.EINVAL
    assert fs.value is None
    assert L.xpipe_stage_set_fwd_stream(st._h, base + 16, st.ws_bytes, None) == xp.EINVAL
    assert L.xpipe_stage_set_fwd_stream(st._h, base, st.ws_bytes, ctypes.byref(fs)) == xp.OK
    assert fs.value not in (None, s0.cuda_stream)          # a stream of the stage's own
    assert L.xpipe_stage_set_fwd_stream(st._h, None, 0, ctypes.byref(fs)) == xp.OK
    assert fs.value is None
    one = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32, static_workspace=True)
    try:
        assert L.xpipe_stage_set_fwd_stream(one._h, base, st.ws_bytes, None) == xp.EUNSUPPORTED
        assert L.xpipe_stage_set_fwd_stream(one._h, None, 0, None) == xp.OK
    finally:
        one.destroy()
    torch.cuda.synchronize()


def test_forward_stream_many_recorded_passes():
    """More distinct pointer sets than the stage keeps recorded passes (64):
    the least recently used graphs are dropped while passes still run on both
    streams.  Outputs and the accumulated gradient must equal an eager run on
    one stream, bit for bit."""
    import torch
    w = SMALL["tiny_mlp"]()
    inp = wl.stage_inputs(w, act_dtype="f32", moment_init="paper")
    n = 80
    g = torch.Generator().manual_seed(5)
    xs = [torch.randn((w.micro_batch,) + tuple(w.in_shape), generator=g).cuda() for _ in range(n)]
    labels = [torch.randint(0, 10, (w.micro_batch,), generator=g, dtype=torch.int32).cuda()
              for _ in range(n)] if w.has_loss else None
    hp = xp.Hyper()
    outs = []
    for overlap in (False, True):
        st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32)
        st.set_graphs(overlap)
        st.set_flat(st.W, inp.params)
        st.set_flat(st.m, inp.m)
        st.set_flat(st.v, inp.v)
        if overlap:
            st.xpipe_stage_set_fwd_stream(True)
        st.xpipe_predict_weights(xp.FWD, 1, hp, 3)
        st.xpipe_predict_weights(xp.BWD, 1, hp, 3)
        ys = [torch.empty(st.out_shape, dtype=torch.float32, device="cuda") for _ in range(n)]
        dys = None if w.has_loss else [torch.randn(st.out_shape, generator=g).cuda() for _ in range(n)]
        torch.cuda.synchronize()
        for k in range(n):
            st.xpipe_stage_fwd(xs[k], ys[k], None if labels is None else labels[k], None)
            st.xpipe_stage_bwd(xs[k], None if dys is None else dys[k],
                               None if labels is None else labels[k], None)
        torch.cuda.synchronize()
        outs.append((ys, st.grad.clone()))
        st.destroy()
    for k in range(n):
        assert torch.equal(outs[0][0][k], outs[1][0][k]), f"y[{k}]"
    assert torch.equal(outs[0][1], outs[1][1]), "grad"

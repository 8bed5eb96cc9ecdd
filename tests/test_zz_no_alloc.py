"""The stage that allocates nothing (xpipe_stage_create_static: the library's
static device workspace, one launch lane, no recorded passes) against the
ordinary stage (xpipe_stage_create with a caller workspace), through the C
ABI: the whole step (predictions, forward, backward with recomputation, fused
Adam) bit for bit, on two stages in a row, the second with a smaller input,
which finds the first one's leftovers in the shared array."""
import numpy as np
import pytest

import paper_1911_04610_amd as xp
import workloads as wl
from gpu_harness import run_stage

pytestmark = pytest.mark.gpu


def _same_bits(a, b):
    for ra, rb in zip(a, b):
        for f in ("w_pred_fwd", "w_pred_bwd", "grad", "W", "m", "v"):
            for x, y in zip(getattr(ra, f), getattr(rb, f)):
                assert np.array_equal(x, y), f
        for x, y in zip(ra.ys + ra.dxs, rb.ys + rb.dxs):
            assert np.array_equal(x, y)
        assert ra.losses == rb.losses


CASES = {
    xp.BF16: [
        lambda: wl.shrink(wl.inception_stage(), micro_batch=2, T=2, minibatches=2,
                          layers=wl.inception_stage_layers(modules=2), in_shape=(9, 9, 256)),
        lambda: wl.shrink(wl.inception_stage(), micro_batch=2, T=2, minibatches=2,
                          layers=wl.inception_stage_layers(modules=1, classes=10), in_shape=(7, 7, 256)),
    ],
    xp.F32: [
        lambda: wl.shrink(wl.vgg_stage(), micro_batch=4, spatial=(20, 20), T=2, minibatches=2),
        lambda: wl.shrink(wl.vgg_stage(), micro_batch=2, spatial=(12, 12), T=2, minibatches=2),
    ],
}


@pytest.mark.parametrize("dtype", [xp.BF16, xp.F32])
def test_static_workspace_stage_matches_ordinary_stage(dtype):
    act = "bf16" if dtype == xp.BF16 else "f32"
    sizes = []
    for make in CASES[dtype]:
        w = make()
        sizes.append(xp.xpipe_stage_query(w.layers, w.micro_batch, w.in_shape, dtype)[1])
        inp = wl.stage_inputs(w, act_dtype=act)
        st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dtype, static_workspace=True)
        assert st.workspace is None
        try:
            a, _ = run_stage(w, inp, dtype, xp.Hyper(), w.s_fwd, w.s_bwd, stage=st)
        finally:
            st.destroy()
        b, _ = run_stage(w, inp, dtype, xp.Hyper(), w.s_fwd, w.s_bwd)
        _same_bits(a, b)
    assert sizes[1] < sizes[0] <= 64 << 20


def test_static_workspace_stage_refusals():
    """One such stage per device at a time; stages whose workspace exceeds the
    array are refused on the host; recorded passes are not offered."""
    w = wl.shrink(wl.vgg_stage(), micro_batch=2, spatial=(12, 12), T=2)
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32, static_workspace=True)
    try:
        with pytest.raises(xp.XPipeError) as e:
            xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32, static_workspace=True)
        assert e.value.status == xp.ESTATE
        with pytest.raises(xp.XPipeError) as e:
            st.set_graphs(True)
        assert e.value.status == xp.EUNSUPPORTED
    finally:
        st.destroy()
    big = wl.vgg_stage()                          # micro-batch 32 at 32 x 32: ~200 MiB in fp32
    assert xp.xpipe_stage_query(big.layers, big.micro_batch, big.in_shape, xp.F32)[1] > 64 << 20
    with pytest.raises(xp.XPipeError) as e:
        xp.Stage(big.layers, big.micro_batch, big.T, big.in_shape, xp.F32, static_workspace=True)
    assert e.value.status == xp.EINVAL and "static workspace" in str(e.value)
    # the slot is free again
    xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, xp.F32, static_workspace=True).destroy()

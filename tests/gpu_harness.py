"""Runs a stage workload through the GPU library (via the C ABI binding) and
returns records shaped like the oracle's, for the parity tests and bench."""
import numpy as np

import paper_1911_04610_amd as xp


def to_device(a, dtype, device="cuda"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device)
    return t.to(torch.bfloat16) if dtype == xp.BF16 else t


def to_host(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


class GpuRecord:
    def __init__(self):
        self.w_pred_fwd = self.w_pred_bwd = self.grad = self.W = self.m = self.v = None
        self.ys, self.losses, self.dxs = [], [], []


def run_stage(w, inp, dtype, hp, s_fwd, s_bwd, minibatches=None, fused=True, need_dx=True,
              stage=None, reuse_inputs=False, rule=None, fwd_stream=False):
    """Mini-batch loop of the XPipe stage step on the GPU.  With fused=True the
    Adam step also emits the next mini-batch's predictions (no separate
    predict calls after the first mini-batch).  reuse_inputs feeds mini-batch
    0's buffers to every mini-batch (same pointers on every call).  rule (an
    xp.Rule) updates with momentum SGD / RMSProp instead of Adam.  fwd_stream
    runs the forwards on the stage's forward stream (each output is read after
    that stream)."""
    import torch
    J = len(inp.xs) if minibatches is None else minibatches
    st = stage or xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dtype)
    fs = st.xpipe_stage_set_fwd_stream(True) if fwd_stream else None
    st.set_flat(st.W, inp.params)
    st.set_flat(st.m, inp.m)
    st.set_flat(st.v, inp.v)
    xs = [[to_device(x, dtype) for x in row] for row in inp.xs[:J]]
    labels = None if inp.labels is None else [
        [torch.from_numpy(l).to("cuda") for l in row] for row in inp.labels[:J]]
    dys = None if inp.dys is None else [[to_device(d, dtype) for d in row] for row in inp.dys[:J]]
    tdt = torch.bfloat16 if dtype == xp.BF16 else torch.float32
    n, H, W_, C = st.out_shape
    y = torch.empty((n, H, W_, C), dtype=tdt, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dx = torch.empty((w.micro_batch,) + tuple(w.in_shape), dtype=tdt, device="cuda") if need_dx else None
    out_shape_oracle = (n, C) if (H == 1 and W_ == 1 and len(w.in_shape) == 1) or w.has_loss else (n, H, W_, C)
    buf = torch.zeros(st.P, dtype=torch.float32, device="cuda") if rule is not None else None
    sq = torch.zeros(st.P, dtype=torch.float32, device="cuda") if rule is not None else None
    recs = []
    t = 0
    for jj in range(J):
        j = 0 if reuse_inputs else jj
        r = GpuRecord()
        if jj == 0 or not fused:
            st.xpipe_predict_weights(xp.FWD, s_fwd, hp, t)
        for i in range(w.T):
            st.xpipe_stage_fwd(xs[j][i], y, None if labels is None else labels[j][i],
                               loss if w.has_loss else None)
            if fs is not None:
                torch.cuda.current_stream().wait_stream(fs)
            r.ys.append(to_host(y).reshape(out_shape_oracle))
            r.losses.append(float(loss.item()) if w.has_loss else None)
        r.w_pred_fwd = st.get_tensors(st.w_pred_fwd)
        if jj == 0 or not fused:
            st.xpipe_predict_weights(xp.BWD, s_bwd, hp, t)
        r.w_pred_bwd = st.get_tensors(st.w_pred_bwd)
        for i in range(w.T):
            st.xpipe_stage_bwd(xs[j][i], None if dys is None else dys[j][i],
                               None if labels is None else labels[j][i], dx)
            r.dxs.append(to_host(dx).reshape(inp.xs[0][0].shape) if need_dx else None)
        r.grad = st.get_tensors(st.grad)
        if rule is None:
            st.xpipe_adam_step(hp, t, s_fwd, s_bwd, emit_pred=fused)
        else:
            st.xpipe_rule_step(rule, hp, t, buf, sq, s_fwd, s_bwd, emit_pred=fused)
        t += 1
        r.W = st.get_tensors(st.W)
        r.m = st.get_tensors(st.m)
        r.v = st.get_tensors(st.v)
        recs.append(r)
    torch.cuda.synchronize()
    return recs, st

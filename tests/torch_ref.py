"""A torch CPU float64 autograd implementation of a stage layer list.

Used only by the oracle's pin tests, as an independent library routine that
the oracle's forward and VJP are compared with."""
import numpy as np
import torch
import torch.nn.functional as F


def param_owner(layers):
    out, k = [], 0
    for L in layers:
        n = 0
        if L["kind"] in ("linear", "conv"):
            n = 2 if L["bias"] else 1
        elif L["kind"] == "bn":
            n = 2
        out.append(list(range(k, k + n)))
        k += n
    return out


def forward(layers, P, x, labels=None, N=None):
    """P: list of torch tensors (parameters).  Returns (y, loss)."""
    own = param_owner(layers)
    outs = {-1: x}
    loss = None
    for i, L in enumerate(layers):
        k = L["kind"]
        a = outs[L["inputs"][0]]
        pi = own[i]
        if k == "conv":
            b = P[pi[1]] if L["bias"] else None
            wk = P[pi[0]]
            pad = (0, 0) if L.get("pad", "same") == "valid" else (wk.shape[1] // 2, wk.shape[2] // 2)
            outs[i] = F.conv2d(a.permute(0, 3, 1, 2), wk.permute(0, 3, 1, 2), b,
                               stride=L.get("stride", 1), padding=pad).permute(0, 2, 3, 1)
        elif k == "linear":
            a2 = a.reshape(a.shape[0], a.shape[-1]) if a.dim() == 4 else a   # [n,1,1,C] -> [n,C]
            outs[i] = F.linear(a2, P[pi[0]], P[pi[1]] if L["bias"] else None)
        elif k == "bn":
            outs[i] = F.batch_norm(a.permute(0, 3, 1, 2), None, None, P[pi[0]], P[pi[1]],
                                   training=True, eps=1e-5).permute(0, 2, 3, 1)
        elif k == "relu":
            outs[i] = F.relu(a)
        elif k == "add":
            outs[i] = a + outs[L["inputs"][1]]
        elif k == "maxpool2":
            outs[i] = F.max_pool2d(a.permute(0, 3, 1, 2), 2).permute(0, 2, 3, 1)
        elif k == "maxpool3s2":
            outs[i] = F.max_pool2d(a.permute(0, 3, 1, 2), 3, stride=2,
                                   padding=0 if L.get("pad", "same") == "valid" else 1).permute(0, 2, 3, 1)
        elif k == "avgpool3":
            outs[i] = F.avg_pool2d(a.permute(0, 3, 1, 2), 3, 1, 1,
                                   count_include_pad=True).permute(0, 2, 3, 1)
        elif k == "gap":
            outs[i] = a.mean((1, 2))
        elif k == "concat":
            outs[i] = torch.cat([outs[j] for j in L["inputs"]], -1)
        elif k == "softmax_ce":
            outs[i] = a
            loss = F.cross_entropy(a, torch.as_tensor(labels, dtype=torch.long), reduction="sum") / N
    return outs[len(layers) - 1], loss


def fwd_bwd(layers, params, x, dy=None, labels=None, N=None):
    P = [torch.tensor(np.asarray(p, np.float64), requires_grad=True) for p in params]
    xt = torch.tensor(np.asarray(x, np.float64), requires_grad=True)
    y, loss = forward(layers, P, xt, labels, N)
    if loss is not None:
        loss.backward()
    else:
        y.backward(torch.tensor(np.asarray(dy, np.float64)))
    return (y.detach().numpy(), None if loss is None else loss.item(), xt.grad.numpy(),
            [p.grad.numpy() for p in P])

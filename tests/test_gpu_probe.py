"""The measurement probes that bench.py reports next to the stage step run
on the GPU and return sane figures (they are not part of the method)."""
import math

import pytest

import paper_1911_04610_amd as xp

pytestmark = pytest.mark.gpu


def test_graph_probe_times_both_layouts():
    import torch
    scratch = torch.zeros(2048, dtype=torch.float32, device="cuda")
    for width, length, spin in ((1, 1, 0), (3, 2, 200)):
        par, ser = xp.xpipe_probe_graph(scratch, width, length, 8, spin)
        assert math.isfinite(par) and math.isfinite(ser) and par > 0 and ser > 0
    torch.cuda.synchronize()
    # the spin launches wrote their results (one float per launch slot)
    assert torch.isfinite(scratch).all() and (scratch[1024:1024 + 8] > 0).all()
    with pytest.raises(xp.XPipeError):
        xp.xpipe_probe_graph(scratch, 4, 1, 8, 0)

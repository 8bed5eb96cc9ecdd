"""XPipe's pipeline schedule as a unit-time model, for counting staleness.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. III-A describes the workflow on a K-GPU pipeline: micro-batches are the
processing unit, the T micro-batches of a mini-batch share weights, gradients
accumulate and the update happens when the T-th micro-batch finishes its
backward pass on that GPU, and micro-batches of different mini-batches are
interleaved after a warm-up.  Modelled here as one forward or backward pass
per time unit per GPU, one-forward-one-backward in the steady phase:
forward of micro-batch i (1-based) on GPU r at time 2i + r, its backward at
2i + 2K - 1 - r.  This reproduces the orders the text describes (GPU 0 with
K = 4 runs F1..F4, then B1 F5 B2 F6 ...; with T = 2 micro-batch 5's forward
uses the initial weights and two updates, after B2 and B4, precede B5).

For a bellwether (the first micro-batch of its mini-batch, Sec. III-B) the
version difference it should predict over is counted as the number of updates
on its GPU after its pass, up to the unit in which the T-th micro-batch of its
mini-batch completes its backward pass on GPU 0; "incl" also counts the
mini-batch's own update on that GPU, "excl" does not.
"""
from __future__ import annotations

import dataclasses
from typing import List

from .method import HALF_UP, version_difference_bwd, version_difference_fwd

FWD, BWD = 0, 1


@dataclasses.dataclass
class Event:
    time: int          # pipeline unit
    kind: int          # FWD or BWD
    micro: int         # 1-based micro-batch index
    mini: int          # 1-based mini-batch index
    bellwether: bool   # first micro-batch of its mini-batch
    update_after: bool  # the weights are updated right after this backward
    version: int       # updates applied on this GPU before the pass
    s_eq: int = 0      # bellwether: Eq. 1 (forward) / Eq. 2 (backward)
    s_excl: int = 0    # bellwether: counted updates, without its own mini-batch's
    s_incl: int = 0    # bellwether: counted updates, with its own mini-batch's


def fwd_time(K: int, r: int, i: int) -> int:
    return 2 * i + r


def bwd_time(K: int, r: int, i: int) -> int:
    return 2 * i + 2 * K - 1 - r


def schedule(size: int, T: int, rank: int, minibatches: int, rule: str = HALF_UP,
             ceil_half_rank: bool = False) -> List[Event]:
    """Events of GPU `rank` for `minibatches` mini-batches, in time order."""
    K = size
    n = T * minibatches
    raw = []
    for i in range(1, n + 1):
        raw.append((fwd_time(K, rank, i), FWD, i))
        raw.append((bwd_time(K, rank, i), BWD, i))
    raw.sort()
    # times of this GPU's updates (after the backward of each T-th micro-batch)
    upd = [bwd_time(K, rank, T * j) for j in range(1, minibatches + 1)]
    events = []
    for time, kind, i in raw:
        j = (i - 1) // T + 1
        bell = (i - 1) % T == 0
        version = sum(1 for u in upd if u < time)
        e = Event(time, kind, i, j, bell, kind == BWD and i % T == 0, version)
        if bell:
            e.s_eq = (version_difference_fwd(size, T, rank, rule, ceil_half_rank) if kind == FWD
                      else version_difference_bwd(size, T, rank, rule))
            end = bwd_time(K, 0, T * j)          # the round trip ends on GPU 0
            own = bwd_time(K, rank, T * j)       # this mini-batch's update here
            # updates strictly after the pass (an update that follows the
            # bellwether's own backward pass, T = 1, does not change the weights
            # that pass used) up to the unit in which the round trip ends
            between = [u for u in upd if time < u <= end]
            e.s_incl = len(between)
            e.s_excl = len([u for u in between if u != own])
        events.append(e)
    return events

"""The oracle's pipeline schedule (unit-time model of Sec. III-A) pinned to
the orders and weight versions the paper's text walks through, and to
properties the text states."""
import pytest

from oracle import schedule as sc
from oracle import method as om


def _order(ev, n):
    return " ".join(("F" if e.kind == sc.FWD else "B") + str(e.micro) for e in ev[:n])


def test_gpu0_order_with_four_gpus():
    """GPU 0 of four: a warm-up of four forwards, then one forward and one
    backward in turn (Fig. 1)."""
    ev = sc.schedule(4, 1, 0, 8)
    assert _order(ev, 13) == "F1 F2 F3 F4 B1 F5 B2 F6 B3 F7 B4 F8 B5"


def test_fifth_micro_batch_example_T2():
    """Sec. III-A, T = 2 on four GPUs: GPU 0 runs micro-batch 5's forward on
    the initial weights and, by its backward, the weights were updated twice,
    after the backward passes of micro-batches 2 and 4."""
    ev = sc.schedule(4, 2, 0, 4)
    f5 = next(e for e in ev if e.kind == sc.FWD and e.micro == 5)
    b5 = next(e for e in ev if e.kind == sc.BWD and e.micro == 5)
    assert f5.version == 0 and b5.version == 2
    ups = [e.micro for e in ev if e.update_after and e.time < b5.time]
    assert ups == [2, 4]


def test_update_between_bellwether_and_followers_T4():
    """The draft text's example, T = 4 on four GPUs: on GPU 2 the update for
    mini-batch 1 lands after micro-batch 5's forward (the bellwether of
    mini-batch 2) and before micro-batch 6's."""
    ev = sc.schedule(4, 4, 2, 3)
    i5 = next(q for q, e in enumerate(ev) if e.kind == sc.FWD and e.micro == 5)
    i6 = next(q for q, e in enumerate(ev) if e.kind == sc.FWD and e.micro == 6)
    between = [e for e in ev[i5 + 1:i6] if e.update_after]
    assert [e.micro for e in between] == [4]
    assert ev[i5].version == 0 and ev[i6].version == 1


@pytest.mark.parametrize("T", [1, 2, 4])
def test_lower_ranks_see_staler_weights(T):
    """Sec. III-A: the number of updates between a micro-batch's forward and
    backward varies with the GPU, and smaller indices are staler."""
    K = 4
    stale = []
    for r in range(K):
        ev = sc.schedule(K, T, r, 6)
        f = {e.micro: e.version for e in ev if e.kind == sc.FWD}
        b = {e.micro: e.version for e in ev if e.kind == sc.BWD}
        stale.append(max(b[i] - f[i] for i in f))
    assert stale == sorted(stale, reverse=True) and stale[0] > stale[-1]


@pytest.mark.parametrize("K,T", [(1, 1), (1, 4), (2, 2), (4, 4), (8, 1)])
def test_schedule_invariants(K, T):
    """Every micro-batch runs forward then backward on every GPU; the weights
    are updated once per mini-batch, after its T-th backward; a mini-batch's
    backward passes are consecutive; bellwethers carry Eq. 1 / Eq. 2."""
    for r in range(K):
        ev = sc.schedule(K, T, r, 5)
        assert len(ev) == 2 * T * 5
        assert all(a.time < b.time for a, b in zip(ev, ev[1:]))
        for i in range(1, T * 5 + 1):
            f = next(e for e in ev if e.kind == sc.FWD and e.micro == i)
            b = next(e for e in ev if e.kind == sc.BWD and e.micro == i)
            assert f.time < b.time and f.version <= b.version
        bw = [e.micro for e in ev if e.kind == sc.BWD]
        assert bw == sorted(bw)
        assert [e.micro for e in ev if e.update_after] == [T * j for j in range(1, 6)]
        for e in ev:
            if e.bellwether:
                want = (om.version_difference_fwd(K, T, r) if e.kind == sc.FWD
                        else om.version_difference_bwd(K, T, r))
                assert e.s_eq == want and 0 <= e.s_excl <= e.s_incl


def test_no_pipeline_has_no_staleness_in_the_schedule():
    """One GPU: each forward is followed by its own backward, so every pass
    sees the weights the previous mini-batch left, and no update falls
    between a bellwether's pass and the end of its round trip."""
    ev = sc.schedule(1, 1, 0, 6)
    assert _order(ev, 6) == "F1 B1 F2 B2 F3 B3"
    assert all(e.s_excl == 0 for e in ev)

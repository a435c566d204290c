"""Pins of the resharding oracle (CPU only).

The input generator draws every weight per (tensor, expert, row chunk), so it
produces a rank's EP slice and a rank's TP slice independently, without the
reshard code.  The oracle's EP->TP result must equal the generator's TP slice
of every rank and vice versa; a round trip is the identity.
"""
import numpy as np
import pytest

import moe_inputs as mi
from oracle import reshard

BASE = mi.MoeConfig("reshard-small", T=4, H=64, E=8, k=2, I=256, P=4, seed=321)


def slices(layout):
    out = [mi.make_inputs(BASE.with_(layout=layout, rank=r)) for r in range(BASE.P)]
    return [o.w13 for o in out], [o.w2 for o in out]


@pytest.fixture(scope="module")
def views():
    return slices("ep"), slices("tp")


def test_ep_to_tp_matches_generated_tp_slices(views):
    (ew13, ew2), (tw13, tw2) = views
    for r in range(BASE.P):
        w13, w2 = reshard.ep_to_tp(ew13, ew2, r, BASE.E, BASE.H, BASE.I)
        np.testing.assert_array_equal(w13, tw13[r])
        np.testing.assert_array_equal(w2, tw2[r])


def test_tp_to_ep_matches_generated_ep_slices(views):
    (ew13, ew2), (tw13, tw2) = views
    for r in range(BASE.P):
        w13, w2 = reshard.tp_to_ep(tw13, tw2, r, BASE.E, BASE.H, BASE.I)
        np.testing.assert_array_equal(w13, ew13[r])
        np.testing.assert_array_equal(w2, ew2[r])


def test_round_trip_is_identity():
    g = np.random.default_rng(5)
    E, H, I, P = 16, 24, 96, 8
    ew13 = [g.integers(0, 65536, (E // P, 2 * I, H), dtype=np.uint16) for _ in range(P)]
    ew2 = [g.integers(0, 65536, (E // P, H, I), dtype=np.uint16) for _ in range(P)]
    tp = [reshard.ep_to_tp(ew13, ew2, r, E, H, I) for r in range(P)]
    back = [reshard.tp_to_ep([t[0] for t in tp], [t[1] for t in tp], r, E, H, I) for r in range(P)]
    for r in range(P):
        np.testing.assert_array_equal(back[r][0], ew13[r])
        np.testing.assert_array_equal(back[r][1], ew2[r])


def test_a_planted_mistake_is_caught(views):
    """Up rows taken from the gate block, or W2 columns from the wrong rank's
    range (plausible slips), fail the pin."""
    (ew13, ew2), (tw13, tw2) = views
    w13, w2 = reshard.ep_to_tp(ew13, ew2, 1, BASE.E, BASE.H, BASE.I)
    Is = BASE.I // BASE.P
    bad13 = w13.copy()
    bad13[:, Is:] = w13[:, :Is]
    assert not np.array_equal(bad13, tw13[1])
    w13_0, w2_0 = reshard.ep_to_tp(ew13, ew2, 0, BASE.E, BASE.H, BASE.I)
    assert not np.array_equal(w2_0, tw2[1])

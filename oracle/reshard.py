"""Expert-weight resharding between the EP and TP layouts, written out from
the layout definitions (Sec. 3.1): a plain, slow CPU reference.

TEST INFRASTRUCTURE ONLY: imported by tests/ and never by the product path.

With E experts, P ranks, hidden size H and expert intermediate size I:

- EP view of rank q: W13 [E/P, 2I, H] (the full gate rows [0, I) then the
  full up rows [I, 2I) of experts q*E/P .. q*E/P + E/P - 1) and
  W2 [E/P, H, I].
- TP view of rank r: W13 [E, 2I/P, H] (for every expert, gate rows
  [r*I/P, (r+1)*I/P) followed by the matching up rows) and W2 [E, H, I/P]
  (columns [r*I/P, (r+1)*I/P) of every expert's W2).

Both views hold the same global weights; a switch only changes which rank
owns which slice.  Arrays are numpy arrays of bf16 bit patterns (uint16), so
every comparison is bit-exact.
"""
from __future__ import annotations

import numpy as np


def ep_to_tp(ep_w13: list, ep_w2: list, r: int, E: int, H: int, I: int) -> tuple:
    """Rank r's TP view from every rank's EP view (lists indexed by rank)."""
    P = len(ep_w13)
    El, Is = E // P, I // P
    w13 = np.zeros((E, 2 * Is, H), np.uint16)
    w2 = np.zeros((E, H, Is), np.uint16)
    for e in range(E):
        q, l = divmod(e, El)                 # owner rank and local index under EP
        for j in range(Is):
            w13[e, j] = ep_w13[q][l, r * Is + j]             # gate row
            w13[e, Is + j] = ep_w13[q][l, I + r * Is + j]    # matching up row
        for h in range(H):
            w2[e, h] = ep_w2[q][l, h, r * Is:(r + 1) * Is]
    return w13, w2


def tp_to_ep(tp_w13: list, tp_w2: list, r: int, E: int, H: int, I: int) -> tuple:
    """Rank r's EP view from every rank's TP view (lists indexed by rank)."""
    P = len(tp_w13)
    El, Is = E // P, I // P
    w13 = np.zeros((El, 2 * I, H), np.uint16)
    w2 = np.zeros((El, H, I), np.uint16)
    for l in range(El):
        e = r * El + l
        for q in range(P):                   # shard q of expert e lives on TP rank q
            for j in range(Is):
                w13[l, q * Is + j] = tp_w13[q][e, j]
                w13[l, I + q * Is + j] = tp_w13[q][e, Is + j]
            for h in range(H):
                w2[l, h, q * Is:(q + 1) * Is] = tp_w2[q][e, h]
    return w13, w2

"""Pins of the switch-policy and request-partition oracle (CPU only).

The partition is greedy longest-first list scheduling on an additive load, so
it must meet the longest-processing-time bound (max load <= (4/3 - 1/(3P))
times the optimum) against a brute-force optimum on small inputs, and the
list-scheduling bound (max load <= mean load + largest item).  The other
values below are worked by hand from the rules of Sec. 3.2 and Sec. 4.5 and
the readings in the oracle's header.
"""
import itertools
import math
import random
from fractions import Fraction

import pytest

from oracle import policy as pol


def loads(tokens, owner, P):
    """Per-rank load tokens_r / T + requests_r / N as exact rationals."""
    N, T = len(tokens), sum(tokens)
    out = [Fraction(0)] * P
    for i, r in enumerate(owner):
        out[r] += Fraction(tokens[i], T) + Fraction(1, N)
    return out


def brute_opt(tokens, P):
    best = None
    for assign in itertools.product(range(P), repeat=len(tokens)):
        m = max(loads(tokens, assign, P))
        best = m if best is None or m < best else best
    return best


@pytest.mark.parametrize("P", [2, 3])
def test_partition_meets_lpt_bound_against_brute_force(P):
    rng = random.Random(P)
    for _ in range(60):
        n = rng.randint(1, 7)
        tokens = [rng.randint(1, 40) for _ in range(n)]
        owner = pol.partition(tokens, P)
        got = max(loads(tokens, owner, P))
        opt = brute_opt(tokens, P)
        assert got <= (Fraction(4, 3) - Fraction(1, 3 * P)) * opt, (tokens, owner)
        item = max(Fraction(t, sum(tokens)) + Fraction(1, n) for t in tokens)
        assert got <= sum(loads(tokens, owner, P)) / P + item


def test_partition_by_hand():
    # tokens [5, 2, 2, 1] on 2 ranks, N = 4, T = 10: 5 -> r0 (0.75); 2 -> r1
    # (0.45); 2 -> r1 (0.90 after); 1 -> r0 (0.75 < 0.90).  A token-only
    # balance would put the last request on r1 (4 < 5).
    assert pol.partition([5, 2, 2, 1], 2) == [0, 1, 1, 0]
    # equal lengths: ties to the lower rank, so round robin in input order
    assert pol.partition([7] * 6, 3) == [0, 1, 2, 0, 1, 2]
    # more ranks than requests: the longest first, each on a fresh rank
    assert pol.partition([1, 9, 4], 5) == [2, 0, 1]


def test_partition_follows_requests_not_positions():
    rng = random.Random(3)
    tokens = rng.sample(range(1, 1000), 40)           # distinct lengths
    owner = pol.partition(tokens, 8)
    perm = list(range(40))
    rng.shuffle(perm)
    owner2 = pol.partition([tokens[i] for i in perm], 8)
    assert [owner[i] for i in perm] == owner2


def test_kv_fits_by_hand():
    # 16-token pages: 32, 16, 17 tokens -> 2, 1, 2 pages (5 in all)
    toks = [32, 16, 17]
    # Qwen3: 4 KV heads on 8 ranks -> TP keeps one head of every request per rank
    assert pol.kv_fits(pol.TP, toks, 8, 4, 16, 5)
    assert not pol.kv_fits(pol.TP, toks, 8, 4, 16, 4)
    # 16 KV heads on 8 ranks -> two per rank
    assert pol.kv_fits(pol.TP, toks, 8, 16, 16, 10)
    assert not pol.kv_fits(pol.TP, toks, 8, 16, 16, 9)
    # EP: rank 0 holds requests 0 and 1 with all 4 heads: (2 + 1) * 4 = 12
    assert pol.kv_fits(pol.EP, toks, 8, 4, 16, 12, owner=[0, 0, 1])
    assert not pol.kv_fits(pol.EP, toks, 8, 4, 16, 11, owner=[0, 0, 1])


def test_tp_needs_more_capacity_when_heads_are_replicated():
    # With n_kv < P and an even EP spread, TP needs P / n_kv times the per-rank capacity of EP.
    toks = [64] * 16                                  # 4 pages each, 2 requests per rank
    owner = [i % 8 for i in range(16)]
    tp_need = 16 * 4 * 1
    ep_need = 2 * 4 * 4
    assert tp_need == ep_need * 8 // 4
    assert pol.kv_fits(pol.TP, toks, 8, 4, 16, tp_need) and not pol.kv_fits(pol.TP, toks, 8, 4, 16, tp_need - 1)
    assert pol.kv_fits(pol.EP, toks, 8, 4, 16, ep_need, owner) and not pol.kv_fits(pol.EP, toks, 8, 4, 16,
                                                                                   ep_need - 1, owner)


def run(policy, trace):
    return [policy.step(c, t, fits) for t, c, fits in trace]


def test_interactive_policy_by_hand():
    # T_h 256, T_l 0.8 * 256, W 8, cooldown 5 s; one iteration per second
    p = pol.Policy(256, 0.8 * 256, 8, 5.0)
    S, W_, C = pol.STAY, pol.SWITCH, pol.CANCELLED
    trace = [(0, 100, True), (1, 200, True), (2, 256, True),   # 256 does not exceed T_h
             (3, 300, True),                                   # exceeds: TP -> EP
             (4, 100, True), (5, 100, True), (6, 100, True), (7, 100, True),  # cooldown until t = 8
             (8, 300, True),  # window t1..t8 = 200 256 300 100 100 100 100 300: mean 182 < 204.8 -> EP -> TP
             (9, 900, True),                                   # cooldown again
             (13, 900, False),                                 # t - 8 = 5: exceeds, EP cannot hold the KV
             (14, 900, True), (17, 900, True),                 # cooldown from the cancel
             (18, 900, True)]                                  # TP -> EP
    assert run(p, trace) == [S, S, S, W_, S, S, S, S, W_, S, C, S, S, W_]
    assert p.mode == pol.EP
    # EP is sticky through a short dip: the window is 900 x 7 then 50 -> mean 793.75
    q = pol.Policy(256, 0.8 * 256, 8, 5.0, mode=pol.EP)
    assert run(q, [(t, 900, True) for t in range(7)] + [(7, 50, True)]) == [S] * 8
    # a sustained dip: after 50 x 7 the mean is (900 + 7*50) / 8 = 156.25 < 204.8
    assert run(q, [(8 + t, 50, True) for t in range(6)]) == [S] * 5 + [W_]


def test_rollout_policy_by_hand():
    # T_l = T_h = 256, W = 1, no cooldown: one threshold, both directions
    p = pol.Policy(256, 256, 1, 0.0)
    S, W_ = pol.STAY, pol.SWITCH
    counts = [300, 256, 255, 256, 257, 10]
    assert run(p, [(t, c, True) for t, c in enumerate(counts)]) == [W_, S, W_, S, W_, W_]


def test_crossover_by_hand():
    assert pol.crossover([8, 16, 32, 64], [1, 1, 2, 3], [2, 1.5, 1.9, 2.5]) == 32
    # EP wins at 16 but not at 32: the threshold is where it wins from then on
    assert pol.crossover([64, 8, 32, 16], [3, 1, 1, 1], [2, 2, 2, 0.5]) == 64
    assert pol.crossover([8, 16], [1, 1], [2, 2]) == math.inf
    assert pol.crossover([8, 16], [2, 2], [1, 2]) == 8                # equal cost counts as a win

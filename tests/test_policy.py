"""The layout-switch control in libmoe (host-only C++ behind the C ABI)
against the policy oracle: request partitions, KV-capacity checks, policy
decision traces and threshold calibration, on seeded random inputs, plus the
error paths.  No GPU is used."""
import math
import random

import numpy as np
import pytest

import paper_2606_26607_amd as moe
from oracle import policy as pol


def test_constants_match_oracle():
    assert (moe.MODE_TP, moe.MODE_EP) == (pol.TP, pol.EP)
    assert (moe.STAY, moe.SWITCH, moe.SWITCH_CANCELLED) == (pol.STAY, pol.SWITCH, pol.CANCELLED)


@pytest.mark.parametrize("seed", range(12))
def test_partition_matches_oracle(seed):
    rng = random.Random(seed)
    for _ in range(10):
        P = rng.choice([1, 2, 3, 4, 8, 16])
        n = rng.choice([0, 1, 2, 7, 40, 257])
        hi = rng.choice([1, 5, 4000, 200000])
        tokens = [rng.randint(0, hi) for _ in range(n)]
        if n and rng.random() < 0.3:
            tokens = [rng.choice(tokens[:3]) for _ in range(n)]          # many equal lengths
        owner, rt, rr = moe.partition_requests(tokens, P)
        ref = pol.partition(tokens, P)
        assert list(owner) == ref, (P, tokens)
        for r in range(P):
            assert rt[r] == sum(t for t, o in zip(tokens, ref) if o == r)
            assert rr[r] == ref.count(r)


def test_partition_all_zero_and_large():
    owner, _, rr = moe.partition_requests([0] * 10, 4)
    assert list(owner) == pol.partition([0] * 10, 4) == [0, 1, 2, 3, 0, 1, 2, 3, 0, 1]
    big = [2 ** 40 + i for i in range(9)]
    assert list(moe.partition_requests(big, 3)[0]) == pol.partition(big, 3)


@pytest.mark.parametrize("seed", range(6))
def test_kv_fits_matches_oracle(seed):
    rng = random.Random(100 + seed)
    for _ in range(40):
        P = rng.choice([1, 2, 4, 8])
        n_kv = rng.choice([1, 2, 4, 8, 16])
        if n_kv % P and P % n_kv:
            continue
        ps = rng.choice([1, 16, 64])
        tokens = [rng.randint(0, 5000) for _ in range(rng.randint(0, 60))]
        owner = [rng.randrange(P) for _ in tokens]
        for mode in (pol.TP, pol.EP):
            for cap in (0, rng.randint(0, 4000), rng.randint(0, 40000)):
                got = moe.kv_fits(mode, tokens, P, n_kv, ps, cap, owner if mode == pol.EP else None)
                assert got == pol.kv_fits(mode, tokens, P, n_kv, ps, cap, owner)


@pytest.mark.parametrize("seed", range(10))
def test_policy_traces_match_oracle(seed):
    rng = random.Random(200 + seed)
    t_high = rng.choice([64, 256, 1000])
    t_low = rng.choice([t_high, 0.8 * t_high, 0.5 * t_high])
    window = rng.choice([1, 2, 8, 33])
    cooldown = rng.choice([0.0, 0.5, 5.0])
    mode = rng.choice([pol.TP, pol.EP])
    a = moe.SwitchPolicy(t_high, t_low, window, cooldown, mode)
    b = pol.Policy(t_high, t_low, window, cooldown, mode)
    now, count = 0.0, rng.randint(0, 2 * t_high)
    for _ in range(600):
        now += rng.choice([0.01, 0.1, 0.3, 1.0])
        count = max(0, count + rng.randint(-t_high // 4, t_high // 4))
        if rng.random() < 0.05:
            count = rng.randint(0, 3 * t_high)                               # bursts and drops
        fits = rng.random() < 0.85
        assert a.step(count, now, fits) == b.step(count, now, fits)
        assert a.mode == b.mode


def test_crossover_matches_oracle():
    rng = random.Random(7)
    for _ in range(200):
        n = rng.randint(1, 10)
        batch = rng.sample(range(1, 5000), n)
        tp = [rng.uniform(0, 10) for _ in range(n)]
        ep = [rng.choice([t, rng.uniform(0, 10)]) for t in tp]
        assert moe.policy_crossover(batch, tp, ep) == pol.crossover(batch, tp, ep)


def test_calibrated_threshold_drives_the_policy():
    # the threshold from a probe where EP wins from B = 64 on; TP -> EP past it
    th = moe.policy_crossover([8, 16, 32, 64, 128], [1.0, 1.1, 1.3, 1.8, 2.9], [1.5, 1.4, 1.35, 1.5, 1.9])
    assert th == 64
    p = moe.SwitchPolicy(th, th, 1, 0.0)
    assert [p.step(c, i) for i, c in enumerate([40, 64, 65, 63])] == [moe.STAY, moe.STAY, moe.SWITCH, moe.SWITCH]


def test_rejects():
    with pytest.raises(moe.MoeError):
        moe.SwitchPolicy(100, 200, 8, 5.0)                                    # t_low > t_high
    with pytest.raises(moe.MoeError):
        moe.SwitchPolicy(200, 100, 0, 5.0)
    with pytest.raises(moe.MoeError):
        moe.SwitchPolicy(200, 100, moe.binding.POLICY_MAX_WINDOW + 1, 5.0)
    with pytest.raises(moe.MoeError):
        moe.SwitchPolicy(200, 100, 8, -1.0)
    with pytest.raises(moe.MoeError):
        moe.SwitchPolicy(200, 100, 8, 1.0, mode=2)
    with pytest.raises(moe.MoeError):
        moe.SwitchPolicy(float("nan"), 100, 8, 1.0)
    p = moe.SwitchPolicy(200, 100, 8, 1.0)
    with pytest.raises(moe.MoeError):
        p.step(-1, 0.0)
    with pytest.raises(moe.MoeError):
        moe.partition_requests([1, 2], 0)
    with pytest.raises(moe.MoeError):
        moe.partition_requests([1, -2], 2)
    with pytest.raises(moe.MoeError):
        moe.partition_requests([2 ** 61, 2 ** 61], 2)                          # total past 2^62
    with pytest.raises(moe.MoeError) as e:
        moe.kv_fits(moe.MODE_TP, [5], 8, 3, 16, 10)                           # 3 heads over 8 ranks
    assert e.value.status == 2
    with pytest.raises(moe.MoeError):
        moe.kv_fits(moe.MODE_EP, [5, 6], 2, 2, 16, 10, owner=[0, 2])
    with pytest.raises(moe.MoeError):
        moe.kv_fits(moe.MODE_EP, [5, 6], 2, 2, 16, 10)                        # EP without owners
    with pytest.raises(moe.MoeError):
        moe.kv_fits(moe.MODE_TP, [5], 2, 2, 0, 10)
    with pytest.raises(moe.MoeError):
        moe.policy_crossover([8, 8], [1, 1], [1, 1])
    with pytest.raises(moe.MoeError):
        moe.policy_crossover([8], [math.nan], [1])
    assert moe.partition_requests([], 3)[0].size == 0
    assert moe.kv_fits(moe.MODE_EP, np.zeros(0), 4, 4, 16, 0, owner=np.zeros(0))

"""Paged KV head moves on the GPU through the C ABI, bit-exact against the
KV move oracle."""
import numpy as np
import pytest
import torch

import paper_2606_26607_amd as moe
from oracle import kvmove

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def host(t):
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def tables(rng, lengths, page_size, n_pages, width):
    perm = rng.permutation(n_pages)
    tab = np.zeros((len(lengths), width), np.int32)
    k = 0
    for q, n in enumerate(lengths):
        m = -(-n // page_size)
        tab[q, :m] = perm[k:k + m]
        k += m
    return tab


def gpu_slots(tab, lengths, page_size, capacity=None):
    first = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    cap = int(first[-1]) if capacity is None else capacity
    out = torch.full((max(cap, 1),), -7, dtype=torch.int32, device="cuda")
    moe.kv_slots(torch.from_numpy(tab).cuda(), torch.from_numpy(first).cuda(), page_size, out=out, capacity=cap)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("page_size", [1, 16, 7])
def test_kv_slots(page_size):
    rng = np.random.default_rng(page_size)
    lengths = [5, 0, 33, 1, 70]
    tab = tables(rng, lengths, page_size, 400, 80)
    got = gpu_slots(tab, lengths, page_size)
    ref = kvmove.token_slots([list(r) for r in tab], lengths, page_size)
    np.testing.assert_array_equal(got[:len(ref)], ref)
    part = gpu_slots(tab, lengths, page_size, capacity=10)   # capacity below the total
    np.testing.assert_array_equal(part[:10], ref[:10])


@pytest.mark.parametrize("with_v", [True, False])
def test_kv_move_matches_oracle(with_v):
    rng = np.random.default_rng(4)
    S1, S2, H1, H2, D, n = 300, 200, 8, 4, 128, 150
    sk = rng.integers(0, 65536, (S1, H1, D), dtype=np.uint16)
    sv = rng.integers(0, 65536, (S1, H1, D), dtype=np.uint16)
    dk = rng.integers(0, 65536, (S2, H2, D), dtype=np.uint16)
    dv = rng.integers(0, 65536, (S2, H2, D), dtype=np.uint16)
    src = rng.integers(0, S1, n).astype(np.int32)
    dst = rng.permutation(S2)[:n].astype(np.int32)
    src[3], dst[5], src[7], dst[9] = -1, -1, S1, S2    # out-of-pool entries are skipped
    valid = (src >= 0) & (src < S1) & (dst >= 0) & (dst < S2)
    Dk, Dv = dev(dk), dev(dv)
    moe.kv_move(dev(sk), dev(sv) if with_v else None, Dk, Dv if with_v else None,
                torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(), 5, 1, 3)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(Dk), kvmove.kv_move(sk, dk, src[valid], dst[valid], 5, 1, 3))
    ref_v = kvmove.kv_move(sv, dv, src[valid], dst[valid], 5, 1, 3) if with_v else dv
    np.testing.assert_array_equal(host(Dv), ref_v)


def test_ep_to_tp_and_back_with_shared_heads():
    """4 KV heads over 8 ranks (two ranks per head under TP): EP pools ->
    TP pools -> fresh EP pools, checked through the page tables."""
    rng = np.random.default_rng(8)
    P, Hkv, D, ps, n_pages = 8, 4, 64, 16, 256
    owners = [[0], [1, 2], [], [3], [4], [5, 6], [7], [8]]
    lengths = rng.integers(1, 120, 9)
    dense = [rng.integers(0, 65536, (n, Hkv, D), dtype=np.uint16) for n in lengths]
    head = lambda r: r * Hkv // P                                   # noqa: E731
    ep_k, ep_tab = [], []
    for q in range(P):
        ls = [int(lengths[i]) for i in owners[q]]
        tab = tables(rng, ls, ps, n_pages, 16)
        pool = np.zeros((n_pages * ps, Hkv, D), np.uint16)
        if ls:
            pool[kvmove.token_slots([list(t) for t in tab], ls, ps)] = np.concatenate([dense[i] for i in owners[q]])
        ep_k.append(dev(pool))
        ep_tab.append(tab)
    tp_tab = [tables(rng, [int(n) for n in lengths], ps, n_pages, 16) for _ in range(P)]
    tp_k = [torch.zeros((n_pages * ps, 1, D), dtype=torch.bfloat16, device="cuda") for _ in range(P)]
    for r in range(P):
        for q in range(P):
            reqs = owners[q]
            if not reqs:
                continue
            ls = [int(lengths[i]) for i in reqs]
            src = gpu_slots(ep_tab[q], ls, ps)
            dst = gpu_slots(tp_tab[r][reqs], ls, ps)
            moe.kv_move(ep_k[q], None, tp_k[r], None, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                        head(r), 0, 1)
    torch.cuda.synchronize()
    for r in range(P):
        pool = host(tp_k[r])
        for i, n in enumerate(lengths):
            sl = kvmove.token_slots([list(tp_tab[r][i])], [int(n)], ps)
            np.testing.assert_array_equal(pool[sl, 0], dense[i][:, head(r)])
    for q in range(P):
        reqs = owners[q]
        if not reqs:
            continue
        ls = [int(lengths[i]) for i in reqs]
        back = torch.zeros_like(ep_k[q])
        dst = gpu_slots(ep_tab[q], ls, ps)
        for r in range(0, P, P // Hkv):                             # one rank per head suffices
            src = gpu_slots(tp_tab[r][reqs], ls, ps)
            moe.kv_move(tp_k[r], None, back, None, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(),
                        0, head(r), 1)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(back)[dst], host(ep_k[q])[dst])


def test_all_sources_in_one_launch():
    """A TP rank's whole pool from every EP pool in one kv_move call: the
    slot vectors come from one kv_slots call per side (the EP owners' page
    tables stacked in owner order, each row indexing its owner's pool), and
    an owner without requests supplies zero tokens.  Checked against the
    oracle moving source by source."""
    rng = np.random.default_rng(15)
    P, Hkv, D, ps, n_pages = 8, 8, 128, 16, 128
    owners = [[0, 1], [2], [], [3, 4, 5], [6], [7], [8, 9], [10]]
    lengths = [int(n) for n in rng.integers(1, 200, 11)]
    ep_k, ep_v, ep_tab = [], [], []
    for q in range(P):
        ls = [lengths[i] for i in owners[q]]
        ep_k.append(rng.integers(0, 65536, (n_pages * ps, Hkv, D), dtype=np.uint16))
        ep_v.append(rng.integers(0, 65536, (n_pages * ps, Hkv, D), dtype=np.uint16))
        ep_tab.append(tables(rng, ls, ps, n_pages, 16))
    order = [i for q in range(P) for i in owners[q]]
    ls_all = [lengths[i] for i in order]
    src_tab = np.concatenate([ep_tab[q][:len(owners[q])] for q in range(P)])
    tp_tab = tables(rng, ls_all, ps, n_pages * 2, 16)
    src = gpu_slots(src_tab, ls_all, ps)
    dst = gpu_slots(tp_tab, ls_all, ps)
    counts = [sum(lengths[i] for i in owners[q]) for q in range(P)]
    dk = rng.integers(0, 65536, (n_pages * 2 * ps, 2, D), dtype=np.uint16)
    dv = rng.integers(0, 65536, (n_pages * 2 * ps, 2, D), dtype=np.uint16)
    Dk, Dv = dev(dk), dev(dv)
    moe.kv_move([dev(t) for t in ep_k], [dev(t) for t in ep_v], Dk, Dv, torch.from_numpy(src).cuda(),
                torch.from_numpy(dst).cuda(), 3, 0, 2, src_tokens=counts)
    torch.cuda.synchronize()
    rk, rv, t0 = dk, dv, 0
    for q in range(P):
        s, d = src[t0:t0 + counts[q]], dst[t0:t0 + counts[q]]
        rk = kvmove.kv_move(ep_k[q], rk, s, d, 3, 0, 2)
        rv = kvmove.kv_move(ep_v[q], rv, s, d, 3, 0, 2)
        t0 += counts[q]
    np.testing.assert_array_equal(host(Dk), rk)
    np.testing.assert_array_equal(host(Dv), rv)


def test_sixteen_sources_and_degenerate_tables():
    """The maximum of 16 source pools in one launch (some supplying no
    tokens), a slot expansion with capacity 0 (writes nothing), and a page
    table narrower than a request (its tokens past the last listed page get
    slot -1 and are not moved)."""
    rng = np.random.default_rng(21)
    S, Hs, D = 96, 2, 64
    counts = [int(c) for c in rng.integers(0, 9, 16)]
    counts[3] = counts[11] = 0
    n = sum(counts)
    pools_k = [rng.integers(0, 65536, (S, Hs, D), dtype=np.uint16) for _ in range(16)]
    src = np.concatenate([rng.integers(0, S, c) for c in counts]).astype(np.int32)
    dst = rng.permutation(4 * S)[:n].astype(np.int32)
    dk = rng.integers(0, 65536, (4 * S, 1, D), dtype=np.uint16)
    Dk = dev(dk)
    moe.kv_move([dev(t) for t in pools_k], None, Dk, None, torch.from_numpy(src).cuda(),
                torch.from_numpy(dst).cuda(), 1, 0, 1, src_tokens=counts)
    torch.cuda.synchronize()
    ref, t0 = dk, 0
    for q in range(16):
        ref = kvmove.kv_move(pools_k[q], ref, src[t0:t0 + counts[q]], dst[t0:t0 + counts[q]], 1, 0, 1)
        t0 += counts[q]
    np.testing.assert_array_equal(host(Dk), ref)
    # capacity 0: nothing written
    out = torch.full((4,), -7, dtype=torch.int32, device="cuda")
    tab = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    moe.kv_slots(tab, torch.tensor([0, 5], dtype=torch.int32, device="cuda"), 4, out=out, capacity=0)
    torch.cuda.synchronize()
    assert torch.all(out == -7)
    # a 2-page table for a 13-token request with 4-token pages: tokens 8..12 have no page
    tab = torch.tensor([[3, 1]], dtype=torch.int32, device="cuda")
    got = gpu_slots(tab.cpu().numpy(), [13], 4)
    np.testing.assert_array_equal(got[:8], kvmove.token_slots([[3, 1]], [8], 4))
    assert np.all(got[8:13] == -1)

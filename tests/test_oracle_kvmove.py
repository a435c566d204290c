"""Pins of the paged KV move oracle (CPU only): a dense per-request cache is
laid into paged EP pools, moved to TP pools by head shard (every rank pair),
and read back through the TP page tables; it must equal the dense cache's
head slices.  Moving back to EP reproduces the original pools' contents."""
import numpy as np

from oracle import kvmove


def paged(rng, lengths, page_size, n_pages):
    """A random page table (distinct pages, shuffled) for each request."""
    perm = rng.permutation(n_pages)
    tables, k = [], 0
    for n in lengths:
        m = -(-n // page_size)
        tables.append(list(perm[k:k + m]))
        k += m
    return tables


def test_ep_to_tp_and_back_through_page_tables():
    rng = np.random.default_rng(11)
    P, Hkv, D, ps = 4, 8, 16, 4          # 2 heads per TP rank
    hr = Hkv // P
    owners = [[0, 1], [2], [3, 4, 5], [6]]            # EP: requests of each rank
    lengths = rng.integers(1, 23, 7)
    dense = [rng.integers(0, 65536, (n, Hkv, D), dtype=np.uint16) for n in lengths]
    n_pages = 64
    # EP pools: rank q holds all heads of its requests
    ep_pool, ep_tab = [], []
    for q in range(P):
        tab = paged(rng, [lengths[i] for i in owners[q]], ps, n_pages)
        pool = np.zeros((n_pages * ps, Hkv, D), np.uint16)
        slots = kvmove.token_slots(tab, [lengths[i] for i in owners[q]], ps)
        pool[slots] = np.concatenate([dense[i] for i in owners[q]])
        ep_pool.append(pool)
        ep_tab.append(tab)
    # TP pools: rank r holds heads [r*hr, (r+1)*hr) of every request
    tp_tab = [paged(rng, lengths, ps, n_pages) for _ in range(P)]
    tp_pool = [np.zeros((n_pages * ps, hr, D), np.uint16) for _ in range(P)]
    for r in range(P):
        for q in range(P):
            reqs = owners[q]
            src = kvmove.token_slots(ep_tab[q], [lengths[i] for i in reqs], ps)
            dst = kvmove.token_slots([tp_tab[r][i] for i in reqs], [lengths[i] for i in reqs], ps)
            tp_pool[r] = kvmove.kv_move(ep_pool[q], tp_pool[r], src, dst, r * hr, 0, hr)
    for r in range(P):
        for i, n in enumerate(lengths):
            slots = kvmove.token_slots([tp_tab[r][i]], [n], ps)
            np.testing.assert_array_equal(tp_pool[r][slots], dense[i][:, r * hr:(r + 1) * hr])
    # and back to fresh EP pools
    for q in range(P):
        reqs = owners[q]
        back = np.zeros_like(ep_pool[q])
        dst = kvmove.token_slots(ep_tab[q], [lengths[i] for i in reqs], ps)
        for r in range(P):
            src = kvmove.token_slots([tp_tab[r][i] for i in reqs], [lengths[i] for i in reqs], ps)
            back = kvmove.kv_move(tp_pool[r], back, src, dst, 0, r * hr, hr)
        np.testing.assert_array_equal(back[dst], ep_pool[q][dst])


def test_token_slots_by_hand():
    # page size 4: request 0 on pages [5, 2] with 6 tokens, request 1 on page [0] with 3
    s = kvmove.token_slots([[5, 2], [0]], [6, 3], 4)
    np.testing.assert_array_equal(s, [20, 21, 22, 23, 8, 9, 0, 1, 2])

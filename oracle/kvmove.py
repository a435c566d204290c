"""Paged KV-cache head moves for a layout switch (Sec. 3.2), written out from
the definition: a plain, slow CPU reference.

TEST INFRASTRUCTURE ONLY: imported by tests/ and never by the product path.

A KV pool of one layer is [slots, heads, head_dim] (a paged pool
[pages, page_size, heads, head_dim] is the same memory, slot = page *
page_size + offset).  A request's tokens sit in the slots its page table
lists.  Under EP a rank holds every KV head of its own requests; under TP it
holds its head shard of every request.  A move copies, for every listed
token i, heads [h_src0, h_src0 + n) of slot src_slot[i] of the source pool
into heads [h_dst0, h_dst0 + n) of slot dst_slot[i] of the destination pool.
"""
from __future__ import annotations

import numpy as np


def token_slots(page_table: list, lengths: list, page_size: int) -> np.ndarray:
    """Slots of every token of the listed requests, in request order: token t
    of request q is at page page_table[q][t // page_size], offset
    t % page_size."""
    out = []
    for pages, n in zip(page_table, lengths):
        for t in range(n):
            out.append(pages[t // page_size] * page_size + t % page_size)
    return np.array(out, dtype=np.int32)


def kv_move(src: np.ndarray, dst: np.ndarray, src_slot, dst_slot, h_src0: int, h_dst0: int,
            n_heads: int) -> np.ndarray:
    """dst with the listed tokens' heads copied in (a new array)."""
    out = dst.copy()
    for s, d in zip(src_slot, dst_slot):
        out[d, h_dst0:h_dst0 + n_heads] = src[s, h_src0:h_src0 + n_heads]
    return out

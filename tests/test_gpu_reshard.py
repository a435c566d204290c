"""Expert-weight resharding on the GPU through the C ABI, bit-exact against
the resharding oracle."""
import numpy as np
import pytest
import torch

import moe_inputs as mi
import paper_2606_26607_amd as moe
from oracle import reshard

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def host(t):
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def random_ep(E, H, I, P, seed):
    g = np.random.default_rng(seed)
    return ([g.integers(0, 65536, (E // P, 2 * I, H), dtype=np.uint16) for _ in range(P)],
            [g.integers(0, 65536, (E // P, H, I), dtype=np.uint16) for _ in range(P)])


@pytest.mark.parametrize("E,H,I,P", [(16, 64, 256, 4), (8, 136, 64, 8), (4, 8, 8, 1), (32, 256, 384, 16)])
def test_reshard_both_directions(E, H, I, P):
    ew13, ew2 = random_ep(E, H, I, P, seed=E + H + I)
    d13 = [dev(a) for a in ew13]
    d2 = [dev(a) for a in ew2]
    tp_ref = [reshard.ep_to_tp(ew13, ew2, r, E, H, I) for r in range(P)]
    tp_dev = []
    for r in range(P):
        t13 = torch.empty((E, 2 * I // P, H), dtype=torch.bfloat16, device="cuda")
        t2 = torch.empty((E, H, I // P), dtype=torch.bfloat16, device="cuda")
        moe.reshard_experts(moe.EP_TO_TP, r, E, H, I, d13, d2, t13, t2)
        tp_dev.append((t13, t2))
    torch.cuda.synchronize()
    for r in range(P):
        np.testing.assert_array_equal(host(tp_dev[r][0]), tp_ref[r][0])
        np.testing.assert_array_equal(host(tp_dev[r][1]), tp_ref[r][1])
    # and back
    for r in range(P):
        b13 = torch.empty_like(d13[r])
        b2 = torch.empty_like(d2[r])
        moe.reshard_experts(moe.TP_TO_EP, r, E, H, I, [t[0] for t in tp_dev], [t[1] for t in tp_dev], b13, b2)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(b13), ew13[r])
        np.testing.assert_array_equal(host(b2), ew2[r])


def test_reshard_own_part_only_leaves_the_rest():
    """With only the destination rank's own source, exactly its 1/P is
    written; the parts other ranks supply keep their previous contents."""
    E, H, I, P, r = 16, 64, 256, 4, 2
    ew13, ew2 = random_ep(E, H, I, P, seed=3)
    ref13, ref2 = reshard.ep_to_tp(ew13, ew2, r, E, H, I)
    t13 = torch.full((E, 2 * I // P, H), 7.0, dtype=torch.bfloat16, device="cuda")
    t2 = torch.full((E, H, I // P), 7.0, dtype=torch.bfloat16, device="cuda")
    sentinel13, sentinel2 = host(t13).copy(), host(t2).copy()
    srcs13 = [dev(ew13[q]) if q == r else None for q in range(P)]
    srcs2 = [dev(ew2[q]) if q == r else None for q in range(P)]
    moe.reshard_experts(moe.EP_TO_TP, r, E, H, I, srcs13, srcs2, t13, t2)
    torch.cuda.synchronize()
    got13, got2 = host(t13), host(t2)
    own = slice(r * E // P, (r + 1) * E // P)   # experts owned by rank r under EP
    np.testing.assert_array_equal(got13[own], ref13[own])
    np.testing.assert_array_equal(got2[own], ref2[own])
    rest = np.ones(E, bool)
    rest[own] = False
    np.testing.assert_array_equal(got13[rest], sentinel13[rest])
    np.testing.assert_array_equal(got2[rest], sentinel2[rest])


def test_slot_buffer_switch_in_place():
    """N layers in N+1 slots per rank, P ranks on one GPU: EP->TP in place
    (layers walked upward), then TP->EP back (downward)."""
    E, H, I, P, N = 16, 64, 256, 4, 3
    ranks = [moe.ExpertSlots(N, E, H, I, P, r, "cuda") for r in range(P)]
    layers = [random_ep(E, H, I, P, seed=100 + i) for i in range(N)]
    for i, (ew13, ew2) in enumerate(layers):
        for r in range(P):
            v13, v2 = ranks[r].ep(i)
            v13.copy_(dev(ew13[r]))
            v2.copy_(dev(ew2[r]))
    moe.ExpertSlots.switch(ranks, moe.EP_TO_TP)
    torch.cuda.synchronize()
    for i, (ew13, ew2) in enumerate(layers):
        for r in range(P):
            ref13, ref2 = reshard.ep_to_tp(ew13, ew2, r, E, H, I)
            t13, t2 = ranks[r].tp(i)
            np.testing.assert_array_equal(host(t13), ref13)
            np.testing.assert_array_equal(host(t2), ref2)
    moe.ExpertSlots.switch(ranks, moe.TP_TO_EP)
    torch.cuda.synchronize()
    for i, (ew13, ew2) in enumerate(layers):
        for r in range(P):
            e13, e2 = ranks[r].ep(i)
            np.testing.assert_array_equal(host(e13), ew13[r])
            np.testing.assert_array_equal(host(e2), ew2[r])


def test_reshard_qwen3_shaped_layer_matches_generated_slices():
    """Full size (128 experts, H 4096, I 1536, P 8): rank 3's TP view built
    on the GPU from the eight EP slices equals the generator's TP slice."""
    base = mi.qwen3_layer(8, "ep")
    ep = [mi.make_inputs(base.with_(rank=q)) for q in range(base.P)]
    tp3 = mi.make_inputs(mi.qwen3_layer(8, "tp", rank=3))
    t13 = torch.empty(tp3.w13.shape, dtype=torch.bfloat16, device="cuda")
    t2 = torch.empty(tp3.w2.shape, dtype=torch.bfloat16, device="cuda")
    moe.reshard_experts(moe.EP_TO_TP, 3, base.E, base.H, base.I, [dev(e.w13) for e in ep],
                        [dev(e.w2) for e in ep], t13, t2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(t13), tp3.w13)
    np.testing.assert_array_equal(host(t2), tp3.w2)

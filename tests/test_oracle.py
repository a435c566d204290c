"""Pins for the CPU oracle (no GPU).

Each check compares the oracle with something other than itself: library
sorts and softmax, a dense all-experts evaluation, a torch SwiGLU MLP,
closed forms, and the identity that the P partial outputs of either layout
sum to the unsliced layer (the paper's claim that EP and TP compute the same
function over the same weights, Sec. 1 and Sec. 3).
"""
import json
import os

import numpy as np
import pytest
import torch

import moe_inputs as mi
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny(**kw):
    base = dict(name="t", T=13, H=32, E=4, k=2, I=24, P=1, layout="replicated", seed=7)
    base.update(kw)
    return mi.MoeConfig(**base)


# ----------------------------------------------------------------- routing
@pytest.mark.parametrize("E,k", [(1, 1), (4, 2), (8, 2), (8, 8), (64, 8), (65, 3), (128, 8),
                                 (256, 8), (1000, 16), (1024, 16)])
@pytest.mark.parametrize("kind", ["normal", "ties"])
def test_route_ids_match_lexsort(oracle, E, k, kind):
    g = np.random.default_rng(E * 31 + k)
    T = 97
    if kind == "normal":
        lg = g.standard_normal((T, E)).astype(np.float32)
    else:  # few distinct values: many exact ties, and both signed zeros
        lg = g.integers(-2, 3, (T, E)).astype(np.float32)
        lg[lg == 0] = np.where(g.random((lg == 0).sum()) < 0.5, -0.0, 0.0)
    ids, w = oracle.route(lg, k)
    np.testing.assert_array_equal(ids, brute.topk_lexsort(lg, k))
    np.testing.assert_allclose(w, brute.route_weights(lg, ids), rtol=0, atol=1e-13)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=0, atol=1e-12)


def test_route_k_equals_E_is_softmax(oracle):
    g = np.random.default_rng(3)
    lg = (3 * g.standard_normal((50, 16))).astype(np.float32)
    ids, w = oracle.route(lg, 16)
    # full softmax written out, read in descending-logit order
    ex = np.exp(lg.astype(np.float64))
    p = ex / ex.sum(1, keepdims=True)
    order = np.argsort(-lg.astype(np.float64), axis=1, kind="stable")
    np.testing.assert_array_equal(ids, order)
    np.testing.assert_allclose(w, np.take_along_axis(p, order, 1), rtol=1e-12, atol=0)


def test_route_k1_weight_is_exactly_one(oracle):
    lg = np.random.default_rng(5).standard_normal((40, 9)).astype(np.float32)
    ids, w = oracle.route(lg, 1)
    assert np.all(w == 1.0)
    np.testing.assert_array_equal(ids[:, 0], np.argmax(lg, axis=1))


def test_route_all_equal_logits(oracle):
    for E, k in [(8, 2), (128, 8), (5, 5)]:
        lg = np.full((6, E), 0.75, np.float32)
        ids, w = oracle.route(lg, k)
        assert np.all(ids == np.arange(k))
        np.testing.assert_allclose(w, 1.0 / k, rtol=0, atol=1e-15)


def test_route_closed_forms(oracle):
    with open(os.path.join(GOLDEN, "route_closed_form.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        lg = np.array([[float(v) for v in c["logits"]]], np.float32)  # "-0.0" parses to -0.0
        ids, w = oracle.route(lg, c["k"])
        assert ids[0].tolist() == c["ids"], c["name"]
        np.testing.assert_allclose(w[0], c["w"], rtol=0, atol=c["atol"], err_msg=c["name"])


# ------------------------------------------------------------- permutation
@pytest.mark.parametrize("T,E,k,P", [(1, 8, 2, 1), (37, 8, 2, 8), (300, 128, 8, 8), (64, 256, 8, 8),
                                     (129, 16, 4, 2), (5, 1024, 16, 4)])
def test_permute_matches_stable_argsort(oracle, T, E, k, P):
    ids = mi.random_topk_ids(T, E, k, seed=T + E)
    total = 0
    for r in range(P):
        e0, El = r * E // P, E // P
        counts, offsets, r2p, p2r = oracle.permute(ids, e0, El)
        bc, bo, br, bp = brute.permute_argsort(ids, e0, El)
        np.testing.assert_array_equal(counts, bc)
        np.testing.assert_array_equal(offsets, bo)
        np.testing.assert_array_equal(r2p, br)
        np.testing.assert_array_equal(p2r, bp)
        assert offsets[0] == 0 and np.all(np.diff(offsets) == counts)
        total += int(offsets[-1])
    assert total == T * k   # every pair lands on exactly one rank


def test_permute_all_tokens_one_expert_and_empty(oracle):
    T, E, k = 50, 8, 2
    ids = mi.random_topk_ids(T, E, k, seed=1, hot=3)
    counts, offsets, r2p, p2r = oracle.permute(ids, 0, E)
    assert counts[3] == T
    assert np.all(r2p[offsets[3]:offsets[4]] // k == np.arange(T))
    # no pairs at all
    counts, offsets, r2p, p2r = oracle.permute(np.zeros((0, 2), np.int32), 0, 4)
    assert np.all(counts == 0) and np.all(offsets == 0) and r2p.size == 0
    # a rank that owns none of the chosen experts
    counts, offsets, r2p, p2r = oracle.permute(np.zeros((9, 1), np.int32), 4, 4)
    assert offsets[-1] == 0 and np.all(p2r == -1)


# --------------------------------------------------------- expert FFN/layer
@pytest.mark.parametrize("cfg", [
    tiny(),
    tiny(E=8, k=8, T=5),
    tiny(E=8, k=2, P=2, layout="tp", rank=1, I=32),
    tiny(E=8, k=3, P=4, layout="ep", rank=2),
    tiny(E=16, k=4, P=4, layout="ep", rank=3, H=48, I=40, T=31),
])
def test_layer_matches_dense_masked_evaluation(oracle, cfg):
    inp = mi.make_inputs(cfg)
    ref = brute.dense_layer(inp.x, inp.logits, cfg.k, inp.w13, inp.w2, cfg.e0, cfg.E_l)
    out = oracle.layer(inp)
    scale = np.abs(ref).max()
    assert scale > 0
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12 * scale)


def test_single_expert_is_swiglu_mlp(oracle):
    cfg = tiny(E=1, k=1, T=9, H=40, I=56)
    inp = mi.make_inputs(cfg)
    x = torch.from_numpy(brute.bf16(inp.x))
    w13 = torch.from_numpy(brute.bf16(inp.w13[0]))
    w1, w3 = w13[:cfg.I], w13[cfg.I:]
    w2 = torch.from_numpy(brute.bf16(inp.w2[0]))
    ref = (torch.nn.functional.silu(x @ w1.T) * (x @ w3.T)) @ w2.T
    out = oracle.layer(inp)
    np.testing.assert_allclose(out, ref.numpy(), rtol=0, atol=1e-13 * float(ref.abs().max()))


@pytest.mark.parametrize("layout,P", [("tp", 2), ("tp", 4), ("ep", 2), ("ep", 4)])
def test_partials_sum_to_unsliced_layer(oracle, layout, P):
    base = tiny(E=8, k=2, T=21, H=40, I=32, seed=11)
    full = oracle.layer(mi.make_inputs(base))
    acc = np.zeros_like(full)
    for r in range(P):
        acc += oracle.layer(mi.make_inputs(base.with_(P=P, layout=layout, rank=r)))
    np.testing.assert_allclose(acc, full, rtol=0, atol=1e-12 * np.abs(full).max())


def test_shared_expert_partials(oracle):
    # each rank adds the shared expert to its own DP share of the tokens only
    base = tiny(E=8, k=2, T=16, H=32, I=16, seed=5, shared=True)
    P = 4
    parts = [oracle.layer(mi.make_inputs(base.with_(P=P, layout="ep", rank=r))) for r in range(P)]
    inp = mi.make_inputs(base)                  # P=1: shared expert on every token
    full = oracle.layer(inp)
    np.testing.assert_allclose(sum(parts), full, rtol=0, atol=1e-12 * np.abs(full).max())
    # and the shared part is a plain SwiGLU MLP added with weight 1
    routed = brute.dense_layer(inp.x, inp.logits, base.k, inp.w13, inp.w2, 0, base.E)
    x = brute.bf16(inp.x)
    W = brute.bf16(inp.sw13[0])
    g, u = x @ W[:base.I].T, x @ W[base.I:].T
    sh = (g / (1 + np.exp(-g)) * u) @ brute.bf16(inp.sw2[0]).T
    np.testing.assert_allclose(full - routed, sh, rtol=0, atol=1e-12 * np.abs(full).max())


# --------------------------------------------------------- stage functions
# bf16 rounding (round to nearest even, 8 significant bits: unit roundoff
# 2^-8) moves a value by at most 2^-8 of its magnitude; a double first
# rounded to fp32 adds 2^-24, and the fp32 gate weight another 2^-24.
BF16_REL = 2.0 ** -8 + 2.0 ** -22


def to_bf16(y):
    return mi.f32_to_bf16_bits(np.asarray(y, np.float64).astype(np.float32))


COMPOSE_CFGS = [
    tiny(),
    tiny(E=16, k=2, T=13, H=24, I=16, seed=3),            # several local experts with no rows
    tiny(E=8, k=2, P=2, layout="tp", rank=1, I=32),
    tiny(E=8, k=3, P=4, layout="ep", rank=2),
    tiny(E=16, k=4, P=4, layout="ep", rank=3, H=48, I=40, T=31),
    tiny(E=8, k=2, T=16, H=32, I=16, seed=5, shared=True, P=4, layout="ep", rank=1),
]


@pytest.mark.parametrize("cfg", COMPOSE_CFGS, ids=lambda c: f"{c.layout}{c.P}r{c.rank}E{c.E}k{c.k}T{c.T}")
def test_stages_compose_to_dense_layer(oracle, cfg):
    """The oracle's stages chained as the library chains its calls (route,
    permute, row gather, grouped FFN, combine, with the shared expert as a
    one-expert grouped FFN) give the layer of the dense evaluation: every
    expert on every token, masked by the top-k selection (the same function
    whatever the layout, Sec. 1 and Sec. 3).  The stage boundary carries y
    in bf16 and the gate weights in fp32, so each output element may differ
    from the dense fp64 value by at most the rounding of its terms:
    sum_j w_j |y_j| 2^-8 (+ |shared| 2^-8)."""
    inp = mi.make_inputs(cfg)
    ids, w = oracle.route(inp.logits, cfg.k)
    _, offsets, r2p, p2r = oracle.permute(ids, cfg.e0, cfg.E_l)
    y = oracle.grouped_ffn(inp.x[r2p // cfg.k], offsets, inp.w13, inp.w2)     # [n, H] fp64
    sb, sc = cfg.shared_begin, cfg.shared_count
    sy = None
    ref = brute.dense_layer(inp.x, inp.logits, cfg.k, inp.w13, inp.w2, cfg.e0, cfg.E_l)
    bound = np.zeros_like(ref)
    if sc:
        sy64 = oracle.grouped_ffn(inp.x[sb:sb + sc], np.array([0, sc], np.int32), inp.sw13, inp.sw2)
        sy = to_bf16(sy64)
        dense_sh = brute.swiglu_mlp(inp.x[sb:sb + sc], inp.sw13[0], inp.sw2[0])
        ref[sb:sb + sc] += dense_sh
        bound[sb:sb + sc] += np.abs(dense_sh) * BF16_REL
    out = oracle.combine(to_bf16(y), p2r, w.astype(np.float32), cfg.T, cfg.k, shared_y=sy, sb=sb, sc=sc)
    # rounding bound of the routed terms, from the dense side's own values
    wb = brute.route_weights(inp.logits, brute.topk_lexsort(inp.logits, cfg.k))
    idsb = brute.topk_lexsort(inp.logits, cfg.k)
    xf = brute.bf16(inp.x)
    for le in range(cfg.E_l):
        tok, slot = np.nonzero(idsb == cfg.e0 + le)
        if tok.size:
            ye = brute.swiglu_mlp(inp.x[tok], inp.w13[le], inp.w2[le])
            bound[tok] += wb[tok, slot][:, None] * np.abs(ye) * BF16_REL
    assert xf.shape == ref.shape
    scale = np.abs(ref).max()
    # the bound is loose only by the factor between actual and worst-case
    # rounding; a wrong row or weight moves an element by about |y|
    assert scale > 0
    err = np.abs(out - ref)
    assert np.all(err <= bound * (1 + 1e-9) + 1e-12 * scale), float((err - bound).max())


def test_combine_relabelled_rows(oracle):
    """The combine reads each pair's row through pair_to_row only: storing
    the rows of y in another order (and pair_to_row with them) gives the
    same output bit for bit."""
    T, k, H, E = 23, 3, 16, 6
    ids = mi.random_topk_ids(T, E, k, seed=2)
    _, offsets, r2p, p2r = oracle.permute(ids, 2, 3)
    n = int(offsets[-1])
    y = mi.random_bf16((n, H), seed=4)
    w = mi.random_gate_weights(T, k, seed=4)
    sigma = np.random.default_rng(1).permutation(n)        # new row of old row r: sigma[r]
    y2 = np.empty_like(y)
    y2[sigma] = y
    p2r2 = np.where(p2r >= 0, sigma[np.maximum(p2r, 0)], -1).astype(np.int32)
    np.testing.assert_array_equal(oracle.combine(y, p2r, w, T, k), oracle.combine(y2, p2r2, w, T, k))


def test_combine_accumulate_and_shared_are_additive(oracle):
    """accumulate adds the prior output and the shared term adds shared_y on
    its token rows only, each with weight one; tokens with no local pair,
    no shared row and no prior are exactly zero."""
    T, k, H, E = 23, 3, 16, 6
    ids = mi.random_topk_ids(T, E, k, seed=2)
    _, offsets, r2p, p2r = oracle.permute(ids, 2, 3)
    n = int(offsets[-1])
    y = mi.random_bf16((n, H), seed=4)
    w = mi.random_gate_weights(T, k, seed=4)
    shared = mi.random_bf16((5, H), seed=9)
    prior = mi.random_bf16((T, H), seed=10)
    base = oracle.combine(y, p2r, w, T, k)
    full = oracle.combine(y, p2r, w, T, k, shared_y=shared, sb=7, sc=5, accumulate=1, prior=prior)
    extra = brute.bf16(prior).copy()
    extra[7:12] += brute.bf16(shared)
    np.testing.assert_allclose(full - base, extra, rtol=0, atol=1e-12)
    untouched = np.all(p2r.reshape(T, k) < 0, axis=1)
    assert untouched.any() and np.all(base[untouched] == 0.0)
    # a token whose every slot is local is the sum of its slots' weighted rows:
    # scaling all weights by 2 doubles the routed part exactly
    np.testing.assert_array_equal(oracle.combine(y, p2r, 2 * w, T, k), 2 * base)


def test_grouped_ffn_experts_are_independent(oracle):
    """Each expert's rows depend only on that expert's weights: the grouped
    call over all experts equals one single-expert call per expert, and
    changing one expert's weights changes only its rows."""
    cfg = tiny(E=4, k=2, T=19, H=24, I=16)
    inp = mi.make_inputs(cfg)
    ids, _ = oracle.route(inp.logits, cfg.k)
    _, offsets, r2p, _ = oracle.permute(ids, 0, cfg.E)
    x_perm = inp.x[r2p // cfg.k]
    y = oracle.grouped_ffn(x_perm, offsets, inp.w13, inp.w2)
    for le in range(cfg.E):
        a, b = int(offsets[le]), int(offsets[le + 1])
        one = oracle.grouped_ffn(x_perm[a:b], np.array([0, b - a], np.int32), inp.w13[le:le + 1],
                                 inp.w2[le:le + 1])
        np.testing.assert_array_equal(y[a:b], one)
    w13b = inp.w13.copy()
    w13b[2] = mi.random_bf16(w13b[2].shape, seed=3, std=0.02)
    y2 = oracle.grouped_ffn(x_perm, offsets, w13b, inp.w2)
    other = np.ones(len(y), bool)
    other[offsets[2]:offsets[3]] = False
    np.testing.assert_array_equal(y2[other], y[other])
    assert offsets[3] > offsets[2] and np.any(y2[~other] != y[~other])


# ------------------------------------------------------------- workloads
def test_config_geometry():
    c = mi.CONFIGS
    assert (c["c2"].E_l, c["c2"].I_s, c["c2"].cap) == (8, 1792, 8192)
    assert (c["c3"].E_l, c["c3"].I_s, c["c3"].e0) == (1, 14336, 0)
    assert (c["c4"].E_l, c["c4"].I_s, c["c4"].cap) == (16, 768, 65536)
    assert (c["c5a"].E_l, c["c5a"].shared_count, c["c5b"].shared_count) == (32, 8, 64)
    assert (c["c4h"].E_l, c["c4h"].e0, c["c4h"].zipf_hot) == (16, 0, True)
    for cfg in c.values():
        cfg.validate()


def test_generator_slices_concatenate_to_full_weight():
    base = tiny(E=4, k=2, I=32, H=16, seed=3)
    full13, full2 = mi.expert_weights(base, 2)
    P = 4
    parts = [mi.expert_weights(base.with_(P=P, layout="tp", rank=r), 2) for r in range(P)]
    Is = base.I // P
    g = np.concatenate([p[0][:Is] for p in parts])
    u = np.concatenate([p[0][Is:] for p in parts])
    np.testing.assert_array_equal(np.concatenate([g, u]), full13)
    np.testing.assert_array_equal(np.concatenate([p[1] for p in parts], axis=1), full2)


def test_zipf_hot_bias_follows_expert_id():
    """The stress variant's popularity rank is the expert id: bias_e =
    -s ln(e + 1), largest for expert 0; the seeded variant permutes the
    same values."""
    hot, seeded = mi.zipf_bias(mi.CONFIGS["c4h"]), mi.zipf_bias(mi.CONFIGS["c4"])
    np.testing.assert_allclose(hot, -1.2 * np.log(np.arange(1, 129)), rtol=1e-6)
    assert np.all(np.diff(hot) < 0)
    np.testing.assert_array_equal(np.sort(seeded), np.sort(hot))


def test_bf16_rounding_is_nearest_even():
    a = np.array([1.0, 1.00390625, 1.0078125 + 0.00390625, -2.5, 3.14159265], np.float32)
    b = mi.bf16_bits_to_f32(mi.f32_to_bf16_bits(a))
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1.0) wins;
    # 1 + 3*2^-8 ties between 1+2^-7 and 1+2^-6: even (1 + 2^-6) wins
    np.testing.assert_array_equal(b[:4], np.array([1.0, 1.0, 1.015625, -2.5], np.float32))
    assert abs(b[4] - 3.140625) == 0

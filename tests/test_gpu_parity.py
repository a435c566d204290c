"""GPU path vs the CPU oracle, through the C ABI (needs an MI355X).

Routing ids, counts, offsets and permutation indices must match bit for
bit; gate weights within 1e-6; layer and stage outputs within
max|err| <= 2e-2 * max|ref|.  Full-size workloads compare every integer
output, and every output row for each workload's own seed (a sample of
rows, evaluated one by one by the oracle, for the two further seeds).
"""
import numpy as np
import pytest
import torch

import moe_inputs as mi
import paper_2606_26607_amd as moe
from tests.util import W_ATOL, assert_close_rel, bf16_f64, dev_bf16, host_bf16

pytestmark = pytest.mark.gpu

SEEDS = (0, 1, 2)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    moe.lib()


def gpu_route(logits: np.ndarray, k: int):
    ids, w = moe.route(torch.from_numpy(logits).cuda(), k)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), w.cpu().numpy()


def gpu_permute(ids: np.ndarray, E: int, e0: int, El: int, x: np.ndarray = None):
    o = moe.permute(torch.from_numpy(ids).cuda(), E, e0, El,
                    x=dev_bf16(x) if x is not None else None)
    torch.cuda.synchronize()
    T, k = ids.shape
    n = int(o["offsets"][-1].item())
    res = dict(counts=o["counts"].cpu().numpy(), offsets=o["offsets"].cpu().numpy(),
               row_to_pair=o["row_to_pair"].cpu().numpy()[:n],
               pair_to_row=o["pair_to_row"].cpu().numpy()[:T * k])
    if x is not None:
        res["x_perm"] = host_bf16(o["x_perm"])[:n]
    return res


# ------------------------------------------------------------------ route
@pytest.mark.parametrize("name", list(mi.CONFIGS))
@pytest.mark.parametrize("seed", SEEDS)
def test_route_configs(oracle, name, seed):
    cfg = mi.CONFIGS[name].with_(seed=mi.CONFIGS[name].seed + seed)
    inp = mi.make_inputs(cfg, with_weights=False)
    ids, w = gpu_route(inp.logits, cfg.k)
    rid, rw = oracle.route(inp.logits, cfg.k)
    np.testing.assert_array_equal(ids, rid)
    assert np.abs(w - rw).max() <= W_ATOL
    assert np.abs(w.sum(1) - 1).max() <= 1e-6


@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (3, 8, 8), (257, 16, 4), (100, 33, 5), (64, 64, 16),
                                   (1000, 128, 8), (513, 256, 8), (77, 1000, 16), (64, 1024, 16),
                                   (40000, 8, 2), (4096, 33, 5), (5000, 64, 16), (4097, 256, 8),
                                   (4100, 512, 16)])
def test_route_ties_and_signed_zeros(oracle, T, E, k):
    g = np.random.default_rng(T * 7 + E)
    lg = g.integers(-2, 3, (T, E)).astype(np.float32)
    z = lg == 0
    lg[z] = np.where(g.random(z.sum()) < 0.5, -0.0, 0.0)
    ids, w = gpu_route(lg, k)
    rid, rw = oracle.route(lg, k)
    np.testing.assert_array_equal(ids, rid)
    assert np.abs(w - rw).max() <= W_ATOL


def test_route_extreme_logits(oracle):
    g = np.random.default_rng(9)
    lg = (g.standard_normal((300, 64)) * 40).astype(np.float32)
    lg[5] = 0.0
    lg[6] = -1e30
    lg[7, 3] = 1e30
    ids, w = gpu_route(lg, 8)
    rid, rw = oracle.route(lg, 8)
    np.testing.assert_array_equal(ids, rid)
    assert np.abs(w - rw).max() <= W_ATOL


def test_route_empty_batch():
    ids, w = moe.route(torch.empty((0, 8), dtype=torch.float32, device="cuda"), 2)
    torch.cuda.synchronize()
    assert ids.shape == (0, 2)


# ---------------------------------------------------------------- permute
@pytest.mark.parametrize("name", list(mi.CONFIGS))
def test_permute_configs(oracle, name):
    cfg = mi.CONFIGS[name]
    inp = mi.make_inputs(cfg, with_weights=False)
    rid, _ = oracle.route(inp.logits, cfg.k)
    got = gpu_permute(rid, cfg.E, cfg.e0, cfg.E_l, inp.x)
    c, o, r2p, p2r = oracle.permute(rid, cfg.e0, cfg.E_l)
    np.testing.assert_array_equal(got["counts"], c)
    np.testing.assert_array_equal(got["offsets"], o)
    np.testing.assert_array_equal(got["row_to_pair"], r2p)
    np.testing.assert_array_equal(got["pair_to_row"], p2r)
    np.testing.assert_array_equal(got["x_perm"], inp.x[r2p // cfg.k])


@pytest.mark.parametrize("T,E,k,P", [(1, 8, 2, 1), (1, 8, 2, 8), (1023, 8, 2, 2), (1025, 64, 8, 8),
                                     (5000, 128, 8, 8), (3000, 1024, 16, 4), (2048, 16, 1, 1),
                                     (70000, 8, 2, 8), (8192, 256, 8, 1), (20000, 512, 8, 2),
                                     (2048, 64, 8, 1), (4096, 128, 4, 2), (4097, 128, 4, 2),
                                     (40000, 512, 8, 8), (448, 64, 8, 1), (456, 64, 8, 1)])
def test_permute_every_rank(oracle, T, E, k, P):
    """Every rank's slice of the same routing, against the oracle.  Small
    inputs run in one workgroup: at most 16384 pairs, 64 local experts and
    32768 pair-steps of ballot work (pairs x (index bits + 2)), so 3584 pairs
    over 64 experts do and 3648 do not; above that pairs x local experts up
    to 2^24 take 256-pair chunks, larger ones 1024-pair chunks (20000 x 8
    pairs over 256 experts and 8192 x 8 over 256 sit on either side of that
    line, and 40000 x 8 pairs over 64 local experts is past it), with the
    scan and the scatter in one launch for up to 64 local experts."""
    ids = mi.random_topk_ids(T, E, k, seed=T + E + k)
    total = 0
    for r in range(P):
        e0, El = r * (E // P), E // P
        got = gpu_permute(ids, E, e0, El)
        c, o, r2p, p2r = oracle.permute(ids, e0, El)
        np.testing.assert_array_equal(got["counts"], c)
        np.testing.assert_array_equal(got["offsets"], o)
        np.testing.assert_array_equal(got["row_to_pair"], r2p)
        np.testing.assert_array_equal(got["pair_to_row"], p2r)
        total += int(o[-1])
    assert total == T * k


@pytest.mark.parametrize("T", [131072, 131104, 524288, 524289])
def test_permute_chunk_count_threshold(oracle, T):
    """Either side of the chunk count above which the scan and the scatter
    run as separate launches (4096 chunks): 131072 x 8 pairs over 8 local
    experts make 4096 chunks of 256 pairs and 131104 x 8 make 4097;
    524288 x 8 and 524289 x 8 (pairs x experts above 2^24) make 4096 and
    4097 chunks of 1024 pairs."""
    E, k, P = 64, 8, 8
    ids = mi.random_topk_ids(T, E, k, seed=T)
    for r in (0, P - 1):
        e0, El = r * (E // P), E // P
        got = gpu_permute(ids, E, e0, El)
        c, o, r2p, p2r = oracle.permute(ids, e0, El)
        np.testing.assert_array_equal(got["counts"], c)
        np.testing.assert_array_equal(got["offsets"], o)
        np.testing.assert_array_equal(got["row_to_pair"], r2p)
        np.testing.assert_array_equal(got["pair_to_row"], p2r)


def test_permute_hot_expert_and_empty_experts(oracle):
    T, E, k = 4099, 16, 4
    ids = mi.random_topk_ids(T, E, k, seed=5, hot=7)
    x = mi.random_bf16((T, 64), seed=5)
    got = gpu_permute(ids, E, 4, 8, x)
    c, o, r2p, p2r = oracle.permute(ids, 4, 8)
    assert c[3] == T
    np.testing.assert_array_equal(got["offsets"], o)
    np.testing.assert_array_equal(got["row_to_pair"], r2p)
    np.testing.assert_array_equal(got["pair_to_row"], p2r)
    np.testing.assert_array_equal(got["x_perm"], x[r2p // k])
    # a rank none of whose experts are chosen
    ids0 = np.zeros((300, 1), np.int32)
    got = gpu_permute(ids0, 16, 8, 8)
    assert np.all(got["counts"] == 0) and np.all(got["offsets"] == 0)
    assert np.all(got["pair_to_row"] == -1)


def test_permute_empty_batch():
    o = moe.permute(torch.empty((0, 2), dtype=torch.int32, device="cuda"), 8, 0, 8)
    torch.cuda.synchronize()
    assert np.all(o["offsets"].cpu().numpy() == 0) and np.all(o["counts"].cpu().numpy() == 0)


# -------------------------------------------------------------- grouped FFN
def ffn_case(oracle, El, H, Is, T, k, seed, hot=None):
    E = El
    ids = mi.random_topk_ids(T, E, k, seed=seed, hot=hot)
    _, offs, r2p, _ = oracle.permute(ids, 0, El)
    n = int(offs[-1])
    x_perm = mi.random_bf16((n, H), seed=seed, tag=41)
    w13 = mi.random_bf16((El, 2 * Is, H), seed=seed, tag=42, std=0.05)
    w2 = mi.random_bf16((El, H, Is), seed=seed, tag=43, std=0.05)
    y = moe.grouped_ffn(dev_bf16(x_perm), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2))
    torch.cuda.synchronize()
    got = bf16_f64(host_bf16(y)[:n])
    ref = oracle.grouped_ffn(x_perm, offs, w13, w2)
    return got, ref


@pytest.mark.parametrize("El,H,Is,T,k", [(1, 64, 32, 1, 1), (4, 256, 192, 150, 2), (8, 136, 72, 99, 3),
                                         (3, 512, 256, 300, 1), (16, 128, 64, 400, 4),
                                         (2, 1024, 512, 130, 2), (5, 384, 320, 611, 3)])
def test_grouped_ffn_stage(oracle, El, H, Is, T, k):
    got, ref = ffn_case(oracle, El, H, Is, T, k, seed=El * 100 + H)
    assert_close_rel(got, ref, what=f"ffn El={El} H={H} Is={Is}")


@pytest.mark.parametrize("El,H,Is,T,k", [(1, 512, 8192, 300, 1), (2, 8192, 256, 200, 1)])
def test_grouped_ffn_long_k_split(oracle, El, H, Is, T, k):
    """A long K (at least 128 slices of 64) with fewer large tiles than CUs
    splits K over workgroups and combines the partials in a second kernel
    (down projection in the first case, gate-up in the second); the result
    matches the oracle and is bitwise reproducible."""
    got, ref = ffn_case(oracle, El, H, Is, T, k, seed=El + H)
    assert_close_rel(got, ref, what=f"long-K El={El} H={H} Is={Is}")
    again, _ = ffn_case(oracle, El, H, Is, T, k, seed=El + H)
    np.testing.assert_array_equal(got, again)


@pytest.mark.parametrize("El,E,H,Is,T,k,e0", [(4, 4, 256, 192, 150, 2, 0), (3, 8, 512, 256, 300, 2, 2),
                                              (8, 8, 1024, 512, 257, 2, 0), (2, 16, 136, 72, 99, 3, 6)])
def test_grouped_ffn_fused_gather(oracle, El, E, H, Is, T, k, e0):
    """Rows read straight from the token matrix through row_to_pair equal the
    FFN of the explicitly gathered rows."""
    ids = mi.random_topk_ids(T, E, k, seed=T + H)
    _, offs, r2p, _ = oracle.permute(ids, e0, El)
    n = int(offs[-1])
    x = mi.random_bf16((T, H), seed=T, tag=44)
    w13 = mi.random_bf16((El, 2 * Is, H), seed=T, tag=45, std=0.05)
    w2 = mi.random_bf16((El, H, Is), seed=T, tag=46, std=0.05)
    cap = T * min(k, El)
    r2p_dev = torch.full((cap,), -1, dtype=torch.int32)
    r2p_dev[:n] = torch.from_numpy(r2p)
    y = moe.grouped_ffn(dev_bf16(x), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2),
                        row_to_pair=r2p_dev.cuda(), k=k, cap_rows=cap)
    torch.cuda.synchronize()
    got = bf16_f64(host_bf16(y)[:n])
    ref = oracle.grouped_ffn(x[r2p // k], offs, w13, w2)
    assert_close_rel(got, ref, what=f"fused El={El} H={H} Is={Is}")


@pytest.mark.parametrize("El,E,H,Is,T,k,e0,sb,sc", [(4, 8, 256, 192, 150, 2, 2, 10, 40),
                                                    (3, 3, 512, 256, 300, 1, 0, 0, 300),
                                                    (1, 2, 512, 8192, 300, 1, 0, 50, 250),
                                                    (8, 8, 256, 128, 200, 2, 0, 0, 0),
                                                    (2, 16, 7168 // 4, 512, 64, 8, 6, 56, 8)])
def test_grouped_ffn_shared(oracle, El, E, H, Is, T, k, e0, sb, sc):
    """Routed experts and a shared expert in the same launches: the routed
    rows equal moe_grouped_ffn's result (oracle on the gathered rows), the
    shared rows the shared expert's FFN on x[sb:sb+sc].  Covers a shared
    expert in the small-row class, in the large class, in a long-K split
    (the separate reduction writes its rows) and none at all."""
    ids = mi.random_topk_ids(T, E, k, seed=T + H + sc)
    _, offs, r2p, _ = oracle.permute(ids, e0, El)
    n = int(offs[-1])
    x = mi.random_bf16((T, H), seed=T, tag=47)
    w13 = mi.random_bf16((El, 2 * Is, H), seed=T, tag=48, std=0.05)
    w2 = mi.random_bf16((El, H, Is), seed=T, tag=49, std=0.05)
    sw13 = mi.random_bf16((2 * Is, H), seed=T, tag=50, std=0.05)
    sw2 = mi.random_bf16((H, Is), seed=T, tag=51, std=0.05)
    cap = T * min(k, El)
    r2p_dev = torch.full((cap,), -1, dtype=torch.int32)
    r2p_dev[:n] = torch.from_numpy(r2p)
    y, sy = moe.grouped_ffn_shared(dev_bf16(x), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2),
                                   r2p_dev.cuda(), k, cap, sb, sc, dev_bf16(sw13), dev_bf16(sw2))
    torch.cuda.synchronize()
    got = bf16_f64(host_bf16(y)[:n])
    ref = oracle.grouped_ffn(x[r2p // k], offs, w13, w2)
    assert_close_rel(got, ref, what=f"routed El={El} H={H} Is={Is}")
    if sc:
        got_s = bf16_f64(host_bf16(sy)[:sc])
        ref_s = oracle.grouped_ffn(x[sb:sb + sc], np.array([0, sc], np.int32), sw13[None], sw2[None])
        assert_close_rel(got_s, ref_s, what=f"shared sb={sb} sc={sc}")


@pytest.mark.parametrize("counts,H,Is", [([592] * 16, 512, 1024),
                                         ([1091], 512, 2048),
                                         ([100, 128, 97, 120, 1, 0, 640, 383] * 2, 256, 512)])
def test_grouped_ffn_tall_leftovers(oracle, counts, H, Is):
    """Experts whose rows leave 65-128 after whole 256-row tiles, or have
    97-128 rows in all: the schedule may take 128-row tiles for them (16
    experts of 512 + 80 rows fill exactly one round of large tiles, so the
    80-row leftovers run on every workgroup and one 128-row tile each is
    cheaper than two 64-row ones).  The result matches the oracle and is
    bitwise reproducible."""
    E = len(counts)
    g = np.random.default_rng(sum(counts))
    ids = g.permutation(np.repeat(np.arange(E, dtype=np.int32), counts))[:, None]
    T = ids.shape[0]
    _, offs, _, _ = oracle.permute(ids, 0, E)
    np.testing.assert_array_equal(np.diff(offs), counts)
    x_perm = mi.random_bf16((T, H), seed=T, tag=52)
    w13 = mi.random_bf16((E, 2 * Is, H), seed=T, tag=53, std=0.05)
    w2 = mi.random_bf16((E, H, Is), seed=T, tag=54, std=0.05)
    runs = []
    for _ in range(2):
        y = moe.grouped_ffn(dev_bf16(x_perm), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2))
        torch.cuda.synchronize()
        runs.append(bf16_f64(host_bf16(y)[:T]))
    ref = oracle.grouped_ffn(x_perm, offs, w13, w2)
    assert_close_rel(runs[0], ref, what=f"tall leftovers E={E} H={H} Is={Is}")
    np.testing.assert_array_equal(runs[0], runs[1])


def test_grouped_ffn_skewed_and_empty_experts(oracle):
    got, ref = ffn_case(oracle, 8, 256, 128, 700, 2, seed=3, hot=5)
    assert_close_rel(got, ref, what="skewed")


def test_grouped_ffn_all_rows_empty():
    El, H, Is = 4, 64, 32
    offs = torch.zeros(El + 1, dtype=torch.int32, device="cuda")
    y = torch.full((16, H), 3.0, dtype=torch.bfloat16, device="cuda")
    w13 = torch.zeros((El, 2 * Is, H), dtype=torch.bfloat16, device="cuda")
    w2 = torch.zeros((El, H, Is), dtype=torch.bfloat16, device="cuda")
    moe.grouped_ffn(torch.zeros((16, H), dtype=torch.bfloat16, device="cuda"), offs, w13, w2, y=y)
    torch.cuda.synchronize()
    assert torch.all(y == 3.0)   # rows past offsets[El] untouched


# ------------------------------------------------------------------ combine
@pytest.mark.parametrize("T,k,H,El,E,acc,shared", [(37, 2, 64, 8, 8, 0, False), (200, 8, 7168, 32, 256, 0, True),
                                                   (100, 4, 256, 2, 8, 1, False), (1, 1, 8, 1, 1, 0, False),
                                                   (513, 16, 520, 64, 128, 1, True)])
def test_combine_stage(oracle, T, k, H, El, E, acc, shared):
    ids = mi.random_topk_ids(T, E, k, seed=T + k)
    _, offs, r2p, p2r = oracle.permute(ids, 0, El)
    n = int(offs[-1])
    y = mi.random_bf16((max(n, 1), H), seed=T)
    w = mi.random_gate_weights(T, k, seed=T)
    prior = mi.random_bf16((T, H), seed=T + 1)
    sb, sc = (T // 4, T // 3) if shared else (0, 0)
    sy = mi.random_bf16((max(sc, 1), H), seed=T + 2) if shared else None
    out = dev_bf16(prior)
    moe.combine(dev_bf16(y), torch.from_numpy(p2r).cuda(), torch.from_numpy(w).cuda(), out=out,
                shared_y=dev_bf16(sy[:sc]) if shared else None, shared_begin=sb, accumulate=bool(acc))
    torch.cuda.synchronize()
    ref = oracle.combine(y, p2r, w, T, k, shared_y=sy, sb=sb, sc=sc, accumulate=acc, prior=prior)
    assert_close_rel(bf16_f64(host_bf16(out)), ref, rtol=1e-2, what="combine")


# -------------------------------------------------------------- full layer
def layer_on_gpu(inp: mi.MoeInputs):
    cfg = inp.cfg
    sw13 = dev_bf16(inp.sw13) if cfg.shared else None
    sw2 = dev_bf16(inp.sw2) if cfg.shared else None
    layer = moe.MoeLayer(cfg.T, cfg.E, cfg.k, cfg.e0, dev_bf16(inp.w13), dev_bf16(inp.w2), sw13, sw2,
                         cfg.shared_begin, cfg.shared_count)
    out = layer.forward(dev_bf16(inp.x), torch.from_numpy(inp.logits).cuda())
    torch.cuda.synchronize()
    return layer, host_bf16(out)


def sample_tokens(cfg, ids, n=24, seed=0):
    """Tokens to check at full size: random ones, plus (EP) tokens with no
    local pair, the first and last token, and shared-expert rows."""
    g = np.random.default_rng(seed)
    picks = set(g.choice(cfg.T, size=min(n, cfg.T), replace=False).tolist()) | {0, cfg.T - 1}
    local = ((ids >= cfg.e0) & (ids < cfg.e0 + cfg.E_l)).any(1)
    none = np.nonzero(~local)[0]
    if none.size:
        picks |= set(none[:3].tolist())
    if cfg.shared:
        picks |= {cfg.shared_begin, cfg.shared_begin + cfg.shared_count - 1, cfg.shared_count}
    return np.array(sorted(picks), np.int64)


@pytest.mark.parametrize("name", list(mi.CONFIGS))
@pytest.mark.parametrize("seed", SEEDS)
def test_layer_configs(oracle, name, seed):
    """The whole chain on every workload and three input seeds (the
    config's own and the next two)."""
    cfg = mi.CONFIGS[name]
    cfg = cfg.with_(seed=cfg.seed + seed)
    inp = mi.make_inputs(cfg)
    layer, out = layer_on_gpu(inp)
    rid, rw = oracle.route(inp.logits, cfg.k)
    np.testing.assert_array_equal(layer.topk_ids.cpu().numpy(), rid)
    assert np.abs(layer.topk_w.cpu().numpy() - rw).max() <= W_ATOL
    c, o, r2p, p2r = oracle.permute(rid, cfg.e0, cfg.E_l)
    np.testing.assert_array_equal(layer.bufs["offsets"].cpu().numpy(), o)
    np.testing.assert_array_equal(layer.bufs["row_to_pair"].cpu().numpy()[:o[-1]], r2p)
    np.testing.assert_array_equal(layer.bufs["pair_to_row"].cpu().numpy()[:cfg.T * cfg.k], p2r)
    # every token for the workload's own seed (the oracle takes a few
    # seconds at full size), a sample of rows for the next two
    toks = np.arange(cfg.T) if seed == 0 or cfg.T * cfg.k * cfg.H * cfg.I_s <= 64 * 2 * 256 * 512 else \
        sample_tokens(cfg, rid)
    ref = oracle.layer_tokens(inp.x, rid, rw, cfg.e0, cfg.E_l, inp.w13, inp.w2, toks, inp.sw13,
                              inp.sw2, cfg.shared_begin, cfg.shared_count)
    assert_close_rel(bf16_f64(out[toks]), ref, what=f"{name} seed+{seed}")
    # tokens with no local pair and no shared term are exactly zero
    local = ((rid >= cfg.e0) & (rid < cfg.e0 + cfg.E_l)).any(1)
    if cfg.shared:
        local[cfg.shared_begin:cfg.shared_begin + cfg.shared_count] = True
    assert np.all(out[~local] == 0)


@pytest.mark.parametrize("layout,B", [("tp", 16), ("ep", 16), ("tp", 256), ("ep", 256)])
def test_layer_qwen3_slices(oracle, layout, B):
    """The TP and EP slices of the Qwen3-235B-shaped layer that the layout
    crossover sweep times (128 experts, top-8, I_s = 192 under TP)."""
    cfg = mi.qwen3_layer(B, layout)
    inp = mi.make_inputs(cfg)
    layer, out = layer_on_gpu(inp)
    rid, rw = oracle.route(inp.logits, cfg.k)
    np.testing.assert_array_equal(layer.topk_ids.cpu().numpy(), rid)
    c, o, r2p, p2r = oracle.permute(rid, cfg.e0, cfg.E_l)
    np.testing.assert_array_equal(layer.bufs["offsets"].cpu().numpy(), o)
    toks = np.arange(cfg.T) if B <= 16 else sample_tokens(cfg, rid)
    ref = oracle.layer_tokens(inp.x, rid, rw, cfg.e0, cfg.E_l, inp.w13, inp.w2, toks, None, None, 0, 0)
    assert_close_rel(bf16_f64(out[toks]), ref, what=cfg.name)


@pytest.mark.parametrize("layout,P", [("tp", 4), ("ep", 4)])
def test_layer_slices_sum_to_unsliced(oracle, layout, P):
    base = mi.MoeConfig("small", T=130, H=256, E=8, k=2, I=512, seed=77)
    ref = oracle.layer(mi.make_inputs(base))
    acc = np.zeros_like(ref)
    for r in range(P):
        _, out = layer_on_gpu(mi.make_inputs(base.with_(P=P, layout=layout, rank=r)))
        acc += bf16_f64(out)
    assert_close_rel(acc, ref, what=f"{layout} partial sum")


def test_layer_is_deterministic():
    inp = mi.make_inputs(mi.CONFIGS["c4"].with_(T=2048))
    layer, out1 = layer_on_gpu(inp)
    y1 = host_bf16(layer.y).copy()
    out2 = host_bf16(layer.forward(dev_bf16(inp.x), torch.from_numpy(inp.logits).cuda()))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out1, out2)
    np.testing.assert_array_equal(y1, host_bf16(layer.y))


@pytest.mark.parametrize("seed", range(8))
def test_grouped_ffn_random_row_mixes(oracle, seed):
    """Seeded random shapes and per-expert row counts (empty experts, a few
    rows, leftovers of every size after whole 256-row tiles, several whole
    tiles), large-tile and general shapes alike: the schedule's choices
    (tail threshold, small tile height, die ranges, idle-slot placement)
    all give the oracle's result, bitwise reproducibly."""
    g = np.random.default_rng(900 + seed)
    El = int(g.integers(1, 41))
    H = int(g.choice([128, 256, 384, 512, 136]))
    Is = int(g.choice([128, 192, 256, 512, 72]))
    kinds = g.integers(0, 5, El)
    counts = []
    for kd in kinds:
        if kd == 0:
            counts.append(0)
        elif kd == 1:
            counts.append(int(g.integers(1, 33)))
        elif kd == 2:
            counts.append(int(g.integers(33, 257)))
        elif kd == 3:
            counts.append(256 * int(g.integers(1, 4)) + int(g.integers(0, 256)))
        else:
            counts.append(256 * int(g.integers(1, 3)))
    if sum(counts) == 0:
        counts[0] = 5
    ids = g.permutation(np.repeat(np.arange(El, dtype=np.int32), counts))[:, None]
    T = ids.shape[0]
    _, offs, _, _ = oracle.permute(ids, 0, El)
    x_perm = mi.random_bf16((T, H), seed=seed, tag=55)
    w13 = mi.random_bf16((El, 2 * Is, H), seed=seed, tag=56, std=0.05)
    w2 = mi.random_bf16((El, H, Is), seed=seed, tag=57, std=0.05)
    runs = []
    for _ in range(2):
        y = moe.grouped_ffn(dev_bf16(x_perm), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2))
        torch.cuda.synchronize()
        runs.append(bf16_f64(host_bf16(y)[:T]))
    ref = oracle.grouped_ffn(x_perm, offs, w13, w2)
    assert_close_rel(runs[0], ref, what=f"random mix seed={seed} El={El} H={H} Is={Is} rows={counts}")
    np.testing.assert_array_equal(runs[0], runs[1])


@pytest.mark.parametrize("counts,H,Is", [([33 * 256 + 100, 500, 60, 7], 2048, 768),
                                         ([16 * 256 + 17, 16 * 256 + 5, 90], 2048, 1024)])
def test_grouped_ffn_moved_tiles(oracle, counts, H, Is):
    """A layer whose down projection has a few more 256-row tiles than one
    round of workgroups: the schedule moves the last m-tiles of the largest
    expert to small-row tiles run whole on all workgroups (and keeps the
    gate-up GEMM's own cut).  Rows sampled across every expert, the moved
    rows included, match the oracle (each output row depends only on its own
    input row and its expert's weights), and the result is bitwise
    reproducible."""
    E = len(counts)
    g = np.random.default_rng(sum(counts))
    ids = g.permutation(np.repeat(np.arange(E, dtype=np.int32), counts))[:, None]
    T = ids.shape[0]
    _, offs, _, _ = oracle.permute(ids, 0, E)
    x_perm = mi.random_bf16((T, H), seed=T, tag=58)
    w13 = mi.random_bf16((E, 2 * Is, H), seed=T, tag=59, std=0.05)
    w2 = mi.random_bf16((E, H, Is), seed=T, tag=60, std=0.05)
    runs = []
    for _ in range(2):
        y = moe.grouped_ffn(dev_bf16(x_perm), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2))
        torch.cuda.synchronize()
        runs.append(host_bf16(y)[:T])
    np.testing.assert_array_equal(runs[0], runs[1])
    got = bf16_f64(runs[0])
    for e in range(E):
        a, b = int(offs[e]), int(offs[e + 1])
        # the last 8 m-tiles (where moved rows lie) every 5th row, the rest every 41st
        tail = max(a, b - 8 * 256)
        rows = np.unique(np.concatenate([np.arange(a, tail, 41), np.arange(tail, b, 5), [b - 1]]))
        ref = oracle.grouped_ffn(x_perm[rows], np.array([0, len(rows)], np.int32), w13[e:e + 1], w2[e:e + 1])
        assert_close_rel(got[rows], ref, what=f"moved tiles expert {e} of {counts}")


def test_grouped_ffn_max_experts(oracle):
    """The most local experts the library takes (1024), most of them small
    (empty, a few rows, 97-128 rows that take two 64-row or one 128-row
    m-tile), some with whole 256-row tiles and a leftover, one large enough
    for the schedule to move its last m-tiles: the schedule's per-expert
    m-tile list is at its widest, and the result matches the oracle,
    bitwise reproducibly."""
    g = np.random.default_rng(4242)
    El, H, Is = 1024, 128, 192
    kinds = g.integers(0, 4, El)
    counts = np.where(kinds == 0, 0, np.where(kinds == 1, g.integers(1, 33, El), g.integers(97, 129, El)))
    counts[g.choice(El, 12, replace=False)] = 256 * g.integers(1, 3, 12) + g.integers(1, 100, 12)
    counts[7] = 256 * 9 + 40
    ids = g.permutation(np.repeat(np.arange(El, dtype=np.int32), counts))[:, None]
    T = ids.shape[0]
    _, offs, _, _ = oracle.permute(ids, 0, El)
    x_perm = mi.random_bf16((T, H), seed=11, tag=58)
    w13 = mi.random_bf16((El, 2 * Is, H), seed=11, tag=59, std=0.05)
    w2 = mi.random_bf16((El, H, Is), seed=11, tag=60, std=0.05)
    runs = []
    for _ in range(2):
        y = moe.grouped_ffn(dev_bf16(x_perm), torch.from_numpy(offs).cuda(), dev_bf16(w13), dev_bf16(w2))
        torch.cuda.synchronize()
        runs.append(bf16_f64(host_bf16(y)[:T]))
    ref = oracle.grouped_ffn(x_perm, offs, w13, w2)
    assert_close_rel(runs[0], ref, what=f"max experts El={El} rows={T}")
    np.testing.assert_array_equal(runs[0], runs[1])

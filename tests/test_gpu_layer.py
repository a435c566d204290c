"""The whole layer in one call (moe_layer_forward) against the four calls
(needs an MI355X).

moe_layer_forward computes exactly what route -> permute -> grouped FFN ->
combine compute, with routing, permutation and tile schedule in fused
launches where the shapes allow; every output and intermediate must be
identical bit for bit to the four calls' (the full-size layer tests compare
the one-call path with the oracle).
"""
import numpy as np
import pytest
import torch

import moe_inputs as mi
import paper_2606_26607_amd as moe
from tests.util import dev_bf16, host_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    moe.lib()


def snapshot(layer):
    b = layer.bufs
    n = int(b["offsets"][-1].item())
    T, k = layer.T, layer.k
    snap = {"topk_ids": layer.topk_ids.cpu().numpy(), "topk_w": layer.topk_w.cpu().numpy().view(np.uint32),
            "counts": b["counts"].cpu().numpy(), "offsets": b["offsets"].cpu().numpy(),
            "row_to_pair": b["row_to_pair"].cpu().numpy()[:n], "pair_to_row": b["pair_to_row"].cpu().numpy()[:T * k],
            "y": host_bf16(layer.y)[:n], "out": host_bf16(layer.out)}
    if layer.sc:
        snap["shared_y"] = host_bf16(layer.s_y)
    return {key: v.copy() for key, v in snap.items()}


def both_paths(cfg, x=None, lg=None):
    inp = mi.make_inputs(cfg)
    sw13 = dev_bf16(inp.sw13) if cfg.shared else None
    sw2 = dev_bf16(inp.sw2) if cfg.shared else None
    layer = moe.MoeLayer(cfg.T, cfg.E, cfg.k, cfg.e0, dev_bf16(inp.w13), dev_bf16(inp.w2), sw13, sw2,
                         cfg.shared_begin, cfg.shared_count)
    assert layer.one_call
    x = dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    layer.forward_calls(x, lg)
    torch.cuda.synchronize()
    ref = snapshot(layer)
    for t in (layer.topk_ids, layer.topk_w, layer.y, layer.out, *layer.bufs.values()):
        t.view(torch.uint8).fill_(0xA5)  # the one call must write everything again
    moe.timing_reset()
    moe.timing_enable(True)
    layer.forward(x, lg)
    torch.cuda.synchronize()
    moe.timing_enable(False)
    got = snapshot(layer)
    _, fused = moe.timing_read("layer_prep")
    return ref, got, fused


def assert_same(ref, got, what):
    assert ref.keys() == got.keys()
    for key in ref:
        np.testing.assert_array_equal(got[key], ref[key], err_msg=f"{what}: {key}")


@pytest.mark.parametrize("name", list(mi.CONFIGS))
def test_one_call_equals_four_calls(name):
    cfg = mi.CONFIGS[name]
    ref, got, fused = both_paths(cfg)
    assert_same(ref, got, cfg.name)
    # every workload has at most 64 local experts and large-tile shapes except
    # the tiny one (H = 256, I = 512: large-tile shapes too): all take the
    # fused launches
    assert fused >= 1


@pytest.mark.parametrize("T,H,E,k,I,P,layout,shared,fused", [
    (700, 256, 16, 3, 256, 1, "replicated", False, True),     # one workgroup (2100 pairs); 3 pairs per token
    (1000, 256, 16, 3, 256, 1, "replicated", False, True),    # 3000 pairs: two fused launches
    (6000, 256, 16, 3, 256, 2, "ep", False, True),            # 256-pair chunks straddled by tokens
    (7000, 128, 64, 6, 128, 1, "replicated", False, True),    # 64 local experts, 6 pairs per token
    (300000, 128, 64, 8, 128, 8, "ep", False, True),          # pairs x experts above 2^24: 1024-pair chunks
    (4096, 1024, 256, 8, 512, 8, "ep", True, True),           # shared expert, two fused launches
    (700, 256, 128, 4, 256, 1, "replicated", False, False),   # 128 local experts: the four calls' launches
    (700, 136, 8, 2, 256, 1, "replicated", False, False),     # H not a multiple of 64: the general GEMM path
    (0, 256, 8, 2, 256, 1, "replicated", False, False),       # no tokens
])
def test_one_call_edges(T, H, E, k, I, P, layout, shared, fused):
    cfg = mi.MoeConfig("edge", T=T, H=H, E=E, k=k, I=I, P=P, layout=layout, shared=shared, seed=T + E + k)
    ref, got, nfused = both_paths(cfg)
    assert_same(ref, got, f"T={T} H={H} E={E} k={k} {layout}{P}")
    assert (nfused > 0) == fused

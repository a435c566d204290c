"""The four-call chain captured in a HIP graph (needs an MI355X).

The library's calls enqueue no host reads and no allocations, so a layer
forward can be captured once and replayed (the paper's serving system keeps
captured graphs valid across layout switches, Sec. 4.4).  Each replay here
runs on new inputs copied into the captured buffers, with eager work and
synchronisations between the replays, and must give exactly what an eager
forward gives on the same inputs (every kernel is deterministic).
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


def _layer(cfg, inp):
    sw13 = dev_bf16(inp.sw13) if cfg.shared else None
    sw2 = dev_bf16(inp.sw2) if cfg.shared else None
    return moe.MoeLayer(cfg.T, cfg.E, cfg.k, cfg.e0, dev_bf16(inp.w13), dev_bf16(inp.w2), sw13, sw2,
                        cfg.shared_begin, cfg.shared_count)


def _snapshot(layer):
    return (host_bf16(layer.out).copy(), layer.topk_ids.cpu().numpy().copy(),
            layer.bufs["offsets"].cpu().numpy().copy(), host_bf16(layer.y).copy())


@pytest.mark.parametrize("name,T", [("c1", None), ("c2", 1024), ("c4", 2048), ("c5a", None), ("c4h", 2048)])
def test_graph_replays_match_eager(name, T):
    cfg = mi.CONFIGS[name]
    if T is not None:
        cfg = cfg.with_(T=T)
    inp = mi.make_inputs(cfg)
    layer = _layer(cfg, inp)
    x = dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    # warm up on a side stream, then capture one forward
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer.forward(x, lg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        layer.forward(x, lg)
    torch.cuda.synchronize()
    for rep in range(3):
        # new inputs: other seeds' tokens and logits, copied into the captured buffers
        c2 = cfg.with_(seed=cfg.seed + 10 + rep)
        xs = mi.make_x(c2)
        ls = mi.make_logits(c2, xs)
        x.copy_(dev_bf16(xs))
        lg.copy_(torch.from_numpy(ls).cuda())
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(layer)
        # eager forward on the same inputs
        layer.out.zero_()
        layer.forward(x, lg)
        torch.cuda.synchronize()
        ref = _snapshot(layer)
        for g, r, what in zip(got, ref, ("out", "topk_ids", "offsets", "y")):
            if what == "y":
                n = int(ref[2][-1])
                g, r = g[:n], r[:n]
            np.testing.assert_array_equal(g, r, err_msg=f"{name} replay {rep}: {what}")


def test_multi_step_graph_matches_eager():
    """Several forwards captured back to back in one graph (as the benchmark
    times them), replayed twice: the result equals one eager forward."""
    cfg = mi.CONFIGS["c4"].with_(T=2048)
    inp = mi.make_inputs(cfg)
    layer = _layer(cfg, inp)
    x = dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    layer.forward(x, lg)
    torch.cuda.synchronize()
    ref = _snapshot(layer)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer.forward(x, lg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(4):
            layer.forward(x, lg)
    for rep in range(2):
        layer.out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(layer)
        n = int(ref[2][-1])
        np.testing.assert_array_equal(got[0], ref[0], err_msg=f"replay {rep}: out")
        np.testing.assert_array_equal(got[3][:n], ref[3][:n], err_msg=f"replay {rep}: y")


def test_device_timestamps_time_graph_replays():
    """GEMM launches captured while device timing is on are timed in every
    replay: after a reset, one replay of a graph of three forwards gives three
    gate-up and three down durations, close to the host-launched events."""
    cfg = mi.CONFIGS["c4"].with_(T=4096)
    inp = mi.make_inputs(cfg)
    layer = _layer(cfg, inp)
    x = dev_bf16(inp.x)
    lg = torch.from_numpy(inp.logits).cuda()
    layer.forward(x, lg)
    moe.timing_reset()
    moe.timing_enable(True)
    for _ in range(3):
        layer.forward(x, lg)
    torch.cuda.synchronize()
    moe.timing_enable(False)
    ev_ms, ev_n = moe.timing_read("gate_up")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer.forward(x, lg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    moe.timing_device_clear()
    moe.timing_device_enable(True)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(3):
            layer.forward(x, lg)
    moe.timing_device_enable(False)
    graph.replay()
    torch.cuda.synchronize()
    moe.timing_device_reset()
    assert moe.timing_device_read("gate_up") == (0.0, 0)
    graph.replay()
    torch.cuda.synchronize()
    for kind in ("gate_up", "down"):
        ms, n = moe.timing_device_read(kind)
        assert n == 3 and ms > 0, (kind, ms, n)
    ms, n = moe.timing_device_read("gate_up")
    assert 0.5 < (ms / n) / (ev_ms / ev_n) < 1.5
    moe.timing_device_clear()

"""Benchmark: one GPU's share of the MoE layer forward (libmoe on MI355X).

A step is the whole hot path over one batch: route -> permute (with the row
gather) -> grouped SwiGLU FFN (+ the shared expert where the layer has one)
-> combine.  Inputs (tokens, router logits, expert weights) are resident in
HBM before the timed region starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c2]

Prints ONE JSON line on stdout; details go to stderr.  The default workload
is the Mixtral-shaped TP=8 slice (4096 tokens, hidden 4096, 8 experts,
top-2, intermediate 14336 sliced to 1792).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s per GPU + % bf16 MFMA peak (prefill) / % HBM BW (decode)"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
REPLAYS = 10                # graph replays of the K steps (step time = median over them)
API = ["moe_layer_forward"]  # the library entry the step calls (--four-calls: the four calls)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_work(cfg, counts: np.ndarray):
    """Flops and bytes the method must move for this step (no tile padding,
    only experts with rows have their weights read)."""
    H, Is = cfg.H, cfg.I_s
    n = int(counts.sum())
    active = int((counts > 0).sum())
    sc = cfg.shared_count
    gate_up_flops = 4.0 * H * Is * n + 4.0 * H * cfg.I * sc
    down_flops = 2.0 * H * Is * n + 2.0 * H * cfg.I * sc
    gate_up_bytes = active * 2 * Is * H * 2 + n * H * 2 + n * Is * 2
    if sc:  # the shared expert's gate-up: its weights plus its token rows in, h rows out
        gate_up_bytes += 2 * cfg.I * H * 2 + sc * H * 2 + sc * cfg.I * 2
    down_bytes = active * H * Is * 2 + n * Is * 2 + n * H * 2
    sh_flops = 0.0  # already in gate_up_flops / down_flops
    sh_bytes = (3 * cfg.I * H * 2 + sc * H * 4 + sc * cfg.I * 4) if sc else 0
    touched = n  # x rows read once per routed pair by the gather, out written once per token
    step_bytes = (active * 3 * Is * H * 2 + (touched + cfg.T) * H * 2 + sh_bytes)
    return dict(n=n, active=active, gate_up_flops=gate_up_flops, down_flops=down_flops,
                gate_up_bytes=gate_up_bytes, down_bytes=down_bytes,
                flops=gate_up_flops + down_flops + sh_flops, bytes=step_bytes)


def kernel_source_sha() -> str:
    """Hash of the grouped-FFN kernel source: counter summaries taken on
    another version of the kernel no longer describe this one."""
    import hashlib
    path = os.path.join(ROOT, "paper_2606_26607_amd", "csrc", "ffn.hip")
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def measured_traffic(workload: str, per: str = "dispatch"):
    """HBM bytes of the gate-up GEMM per launch (per="dispatch") or summed
    over one step's launches (per="step") from the committed rocprofv3
    counter summary (FETCH_SIZE + WRITE_SIZE scaled by the copy-kernel
    calibration), or None when there is none for this kernel source."""
    path = os.path.join(ROOT, "profiles", f"gate_up_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_sha():
        return None
    try:
        return float(kv[f"hbm_bytes_per_{per}"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    """The host CPU's model name (lscpu), for the oracle's timing line."""
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    return platform.processor() or platform.machine()


def oracle_flops(cfg, ids, tokens) -> float:
    """Flops of the layer on `tokens`: 6 H I_s per local pair, 6 H I per
    shared-expert row."""
    t = np.asarray(tokens, np.int64)
    sel = ids[t]
    pairs = int(((sel >= cfg.e0) & (sel < cfg.e0 + cfg.E_l)).sum())
    sh = int(((t >= cfg.shared_begin) & (t < cfg.shared_begin + cfg.shared_count)).sum()) if cfg.shared else 0
    return 6.0 * cfg.H * cfg.I_s * pairs + 6.0 * cfg.H * cfg.I * sh


def cpu_baseline(inp, target_s: float, runs: int = 3):
    """The CPU oracle, timed on a bounded sample of the workload's tokens
    (routing, permutation, expert FFNs and combine for those tokens): the
    median of `runs` runs, or one run when one takes more than 10 s."""
    from oracle import Oracle, build
    build()
    orc = Oracle()
    cfg = inp.cfg
    g = np.random.default_rng(123)
    # calibrate on a few tokens, then size the sample to ~target_s
    probe = np.sort(g.choice(cfg.T, size=min(8, cfg.T), replace=False)).astype(np.int64)

    t0 = time.perf_counter()
    ids, w = orc.route(inp.logits, cfg.k)
    orc.permute(ids, cfg.e0, cfg.E_l)
    t_rp = time.perf_counter() - t0   # routing + permutation of all T tokens

    def run(tokens):
        t0 = time.perf_counter()
        orc.layer_tokens(inp.x, ids, w, cfg.e0, cfg.E_l, inp.w13, inp.w2, tokens, inp.sw13,
                         inp.sw2, cfg.shared_begin, cfg.shared_count)
        return time.perf_counter() - t0 + t_rp * len(tokens) / cfg.T
    dt = run(probe)
    per_tok = max(dt / len(probe), 1e-6)
    S = int(min(cfg.T, max(8, target_s / per_tok)))
    sample = np.sort(g.choice(cfg.T, size=S, replace=False)).astype(np.int64)
    times = [run(sample)]
    while len(times) < runs and times[0] <= 10.0:
        times.append(run(sample))
    dt = float(np.median(times))
    fl = oracle_flops(cfg, ids, sample)
    how = f"median of {len(times)} runs" if len(times) > 1 else "one run"
    return dict(value=S / (cfg.P * dt), unit="tokens/s", cores=orc.threads(), kind="oracle",
                sample=f"{S} of {cfg.T} tokens: expert FFNs + combine for those tokens, plus "
                       f"routing+permutation of all tokens scaled by {S}/{cfg.T}; fp64; {dt:.2f} s ({how})",
                seconds=dt, slice_tokens_per_s=S / dt, gflops=fl / dt / 1e9, runs=len(times))


def cpu_single_thread_c1(mi):
    """The tiny replicated layer (all 64 tokens) on one oracle thread:
    median of 3 runs, in seconds."""
    from oracle import Oracle
    orc = Oracle()
    inp = mi.make_inputs(mi.CONFIGS["c1"])
    n = orc.threads()
    orc.set_threads(1)
    try:
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            orc.layer(inp)
            ts.append(time.perf_counter() - t0)
    finally:
        orc.set_threads(n)
    return float(np.median(ts))


# xGMI of one MI355X: 7 links of about 153 GB/s each way to the 7 peers of
# an 8-GPU node.  Start-up cost of one collective: a stated model parameter.
XGMI_GBS = 7 * 153.0
ALLREDUCE_US = 10.0
ALLTOALL_US = 15.0


def crossover(args, torch, mi, moe):
    """TP slice vs EP slice of the same layer (P = 8) over batch sizes B:
    the measured MoE compute of one rank (the whole four-call chain,
    replayed from a HIP graph) plus the exchange each layout needs, modelled
    from xGMI bandwidth: TP all-reduces out [B, H] (2 (P-1)/P B H 2 bytes
    per GPU); EP dispatches each rank's B/P tokens' k rows to the expert
    owners and combines them back ((P-1)/P (B/P) k H 2 bytes each way).
    Under EP each rank routes only its own B/P tokens; here the slice routes
    all B (a few microseconds more), and its local pairs are the B k / P
    that land on its 16 experts."""
    dev = torch.device("cuda:0")
    batches = [8, 16, 32, 64, 128, 256, 512, 1024, 2048]
    total = {"tp": {}, "ep": {}}

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    for layout in ("tp", "ep"):
        base = mi.qwen3_layer(batches[0], layout)
        t0 = time.time()
        inp = mi.make_inputs(base)
        w13, w2 = up(inp.w13), up(inp.w2)
        log(f"[crossover] {layout} weights in {time.time() - t0:.1f}s")
        for B in batches:
            cfg = mi.qwen3_layer(B, layout)
            x = mi.make_x(cfg)
            lg = mi.make_logits(cfg, x)
            xd, lgd = up(x), torch.from_numpy(lg).to(dev)
            layer = moe.MoeLayer(cfg.T, cfg.E, cfg.k, cfg.e0, w13, w2)
            for _ in range(3):
                layer.forward(xd, lgd)
            torch.cuda.synchronize()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                layer.forward(xd, lgd)
            torch.cuda.current_stream().wait_stream(side)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                for _ in range(args.steps):
                    layer.forward(xd, lgd)
            graph.replay()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            graph.replay()
            b.record()
            torch.cuda.synchronize()
            us = a.elapsed_time(b) * 1e3 / args.steps
            counts = layer.bufs["counts"].cpu().numpy()
            P, H, k = cfg.P, cfg.H, cfg.k
            if layout == "tp":
                comm = ALLREDUCE_US + 2 * (P - 1) / P * B * H * 2 / (XGMI_GBS * 1e3)
            else:
                comm = 2 * (ALLTOALL_US + (P - 1) / P * (B / P) * k * H * 2 / (XGMI_GBS * 1e3))
            print(json.dumps({"crossover": layout, "workload": cfg.name, "B": B, "moe_us": us,
                              "comm_model_us": comm, "total_us": us + comm,
                              "local_pairs": int(counts.sum()), "active_experts": int((counts > 0).sum()),
                              "weight_gb_read": float((counts > 0).sum() * 3 * H * cfg.I_s * 2 / 1e9)}),
                  flush=True)
            total[layout][B] = us + comm
            del graph, layer
    # the coordinator's start-up calibration: the probed crossover is the initial threshold
    th = moe.policy_crossover(batches, [total["tp"][B] for B in batches], [total["ep"][B] for B in batches])
    print(json.dumps({"calibrated_t_high": th if math.isfinite(th) else None, "probed_batches": batches,
                      "cost": "moe_us + comm_model_us"}), flush=True)


def reshard_bench(args, torch, mi, moe):
    """Expert-weight reshard of one Qwen3-235B-shaped layer (128 experts,
    H 4096, I 1536, P 8) for rank 0, both directions: the part a switch keeps
    on the GPU (its own 1/P) and the whole destination view (all P sources in
    this GPU's memory, standing in for peers' buffers).  Each element is read
    once and written once: bytes = 2 x copied bytes, against the HBM peak and
    a measured device copy."""
    dev = torch.device("cuda:0")
    base = mi.qwen3_layer(8, "ep")
    E, H, I, P = base.E, base.H, base.I, base.P
    El, Is = E // P, I // P
    g = torch.Generator(device=dev).manual_seed(7)
    rnd = lambda *shape: torch.randint(-32768, 32767, shape, generator=g, dtype=torch.int16,  # noqa: E731
                                       device=dev).view(torch.bfloat16)
    ep13 = [rnd(El, 2 * I, H) for _ in range(P)]
    ep2 = [rnd(El, H, I) for _ in range(P)]
    tp13 = [rnd(E, 2 * Is, H) for _ in range(P)]
    tp2 = [rnd(E, H, Is) for _ in range(P)]
    slot_bytes = (ep13[0].numel() + ep2[0].numel()) * 2

    def timed(fn, reps=10):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3

    src = torch.empty(slot_bytes // 2, dtype=torch.int16, device=dev)
    dst = torch.empty_like(src)
    copy_gbs = 2 * slot_bytes / timed(lambda: dst.copy_(src)) / 1e9
    del src, dst
    r = 0
    for direction, name in ((moe.EP_TO_TP, "ep_to_tp"), (moe.TP_TO_EP, "tp_to_ep")):
        s13, s2 = (ep13, ep2) if direction == moe.EP_TO_TP else (tp13, tp2)
        d13, d2 = (torch.empty_like(tp13[0]), torch.empty_like(tp2[0])) if direction == moe.EP_TO_TP else \
            (torch.empty_like(ep13[0]), torch.empty_like(ep2[0]))
        for part in ("own", "all"):
            a13 = [t if (part == "all" or q == r) else None for q, t in enumerate(s13)]
            a2 = [t if (part == "all" or q == r) else None for q, t in enumerate(s2)]
            t = timed(lambda: moe.reshard_experts(direction, r, E, H, I, a13, a2, d13, d2))
            moved = slot_bytes if part == "all" else slot_bytes // P
            gbs = 2 * moved / t / 1e9
            print(json.dumps({"reshard": name, "part": part, "workload": "qwen3-235b-shaped-layer",
                              "E": E, "H": H, "I": I, "P": P, "rank": r, "bytes_copied": moved,
                              "us": t * 1e6, "hbm_gbs": gbs, "frac_hbm_peak": gbs / PEAK_HBM_GBS,
                              "frac_of_copy": gbs / copy_gbs, "copy_gbs": copy_gbs}), flush=True)


def kvmove_bench(args, torch, moe):
    """KV-cache moves of one layer for an EP->TP switch of a decode batch:
    256 requests of 500..3500 tokens (seeded) over 8 EP ranks, 4 KV heads of
    128 (two TP ranks per head), 16-token pages in shuffled order.  Rank 0's
    TP pool receives head r*4/8 of every request: `own` moves the part that
    comes from its own EP pool, `all` the whole pool from the 8 EP pools
    (held in this GPU's memory, standing in for peers') in one launch.  The
    page tables serve every layer, so their expansion into slot vectors
    (two kv_slots calls) is timed once per switch and the per-layer figure
    is one kv_move launch for K and V; bytes moved = 2 x the copied bytes."""
    dev = torch.device("cuda:0")
    P, Hkv, D, ps = 8, 4, 128, 16
    rng = np.random.default_rng(2606)
    lengths = rng.integers(500, 3501, 256)
    owner = rng.integers(0, P, 256)
    n_tok = int(lengths.sum())
    width = int(max(-(-int(n) // ps) for n in lengths))

    def tables(ls, n_pages):
        perm = rng.permutation(n_pages).astype(np.int32)
        tab = np.zeros((max(len(ls), 1), width), np.int32)
        k = 0
        for q, n in enumerate(ls):
            m = -(-int(n) // ps)
            tab[q, :m] = perm[k:k + m]
            k += m
        return tab

    pages_ep = [int(sum(-(-int(n) // ps) for n in lengths[owner == q])) + 8 for q in range(P)]
    ep_k = [torch.empty((pg * ps, Hkv, D), dtype=torch.bfloat16, device=dev) for pg in pages_ep]
    ep_v = [torch.empty_like(t) for t in ep_k]
    # the EP owners' page tables stacked in owner order (row i indexes its owner's pool)
    ep_tab = np.concatenate([tables(lengths[owner == q], pages_ep[q])[:int((owner == q).sum())]
                             for q in range(P)])
    pages_tp = int(sum(-(-int(n) // ps) for n in lengths)) + 8
    tp_k = torch.empty((pages_tp * ps, 1, D), dtype=torch.bfloat16, device=dev)
    tp_v = torch.empty_like(tp_k)
    order = np.concatenate([np.nonzero(owner == q)[0] for q in range(P)])
    tp_tab = tables(lengths[order], pages_tp)         # rank 0's TP table, rows in owner order
    counts = [int(lengths[owner == q].sum()) for q in range(P)]
    n_req0 = int((owner == 0).sum())
    cases = {"own": (1, counts[0], ep_tab[:n_req0], tp_tab[:n_req0], lengths[order][:n_req0]),
             "all": (P, n_tok, ep_tab, tp_tab, lengths[order])}
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    csrc = torch.empty(n_tok * D * 2, dtype=torch.int16, device=dev)     # the "all" part's K and V bytes
    cdst = torch.empty_like(csrc)
    cdst.copy_(csrc)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        cdst.copy_(csrc)
    b.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * csrc.numel() * 2 / (a.elapsed_time(b) / reps * 1e-3) / 1e9
    del csrc, cdst
    for part, (n_src, toks, tab_s, tab_d, ls) in cases.items():
        first = torch.from_numpy(np.concatenate([[0], np.cumsum(ls)]).astype(np.int32)).to(dev)
        tab_s, tab_d = torch.from_numpy(tab_s).to(dev), torch.from_numpy(tab_d).to(dev)
        slots_s = torch.empty(toks, dtype=torch.int32, device=dev)
        slots_d = torch.empty(toks, dtype=torch.int32, device=dev)

        def expand():
            moe.kv_slots(tab_s, first, ps, out=slots_s)
            moe.kv_slots(tab_d, first, ps, out=slots_d)

        def move():
            moe.kv_move(ep_k[:n_src], ep_v[:n_src], tp_k, tp_v, slots_s, slots_d, 0, 0, 1,
                        src_tokens=counts[:n_src])

        times = {}
        for name, fn in (("slots", expand), ("move", move)):
            fn()
            torch.cuda.synchronize()
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            times[name] = a.elapsed_time(b) / reps * 1e-3
        copied = toks * D * 2 * 2
        gbs = 2 * copied / times["move"] / 1e9
        print(json.dumps({"kvmove": "ep_to_tp", "part": part, "sources": n_src, "requests": len(ls),
                          "tokens": toks, "kv_heads": Hkv, "head_dim": D, "page_size": ps, "P": P,
                          "bytes_copied": copied, "us_per_layer": times["move"] * 1e6,
                          "slots_us_per_switch": times["slots"] * 1e6, "hbm_gbs": gbs,
                          "frac_hbm_peak": gbs / PEAK_HBM_GBS, "copy_gbs": copy_gbs,
                          "frac_of_copy": gbs / copy_gbs}), flush=True)


def measure(cfg, args, torch, mi, moe, headline: bool):
    """One workload: warmup, a host-launched kernel timing pass (per-kernel
    HIP events recorded by the library on its own stream), then the step
    captured in a HIP graph and replayed K times, each replay timed with
    events; the step time is the median replay.  Returns the measurement,
    the inputs and the algorithmic work."""
    dev = torch.device("cuda:0")
    t0 = time.time()
    inp = mi.make_inputs(cfg)
    log(f"[bench] inputs for {cfg.name} in {time.time() - t0:.1f}s")

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
    x = up(inp.x)
    logits = torch.from_numpy(inp.logits).to(dev)
    layer = moe.MoeLayer(cfg.T, cfg.E, cfg.k, cfg.e0, up(inp.w13), up(inp.w2),
                         up(inp.sw13) if cfg.shared else None, up(inp.sw2) if cfg.shared else None,
                         cfg.shared_begin, cfg.shared_count)
    for _ in range(args.warmup):
        layer.forward_calls(x, logits) if args.four_calls else layer.forward(x, logits)
    torch.cuda.synchronize()
    if headline and args.copy_calib_mib:
        # a plain copy of known size: its FETCH_SIZE / WRITE_SIZE calibrate the counters
        src = torch.empty(args.copy_calib_mib << 19, dtype=torch.int16, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    counts = layer.bufs["counts"].cpu().numpy()
    work = algorithmic_work(cfg, counts)

    # one moe_layer_forward call (fused first launches), or the four calls
    step = (lambda: layer.forward_calls(x, logits)) if args.four_calls else (lambda: layer.forward(x, logits))

    # Kernel timing pass: K steps launched from the host, every kernel
    # bracketed by HIP events on its own stream (the library records them);
    # the roofline's kernel durations come from here.
    moe.timing_reset()
    moe.timing_enable(True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t_start) * 1e3 / args.steps
    moe.timing_enable(False)

    replay_ms = []
    single_ms = None
    graph_kern = {}  # GEMM durations inside the graph replays (device timestamps)
    graph_kern_replay_ms = None  # the step time of the replay they come from
    if args.eager:
        ms_per_step = eager_ms
    else:
        # Throughput pass: the K steps captured back to back in one HIP graph
        # (the kernels run without host launch gaps, as a layer does inside a
        # model's captured forward), replayed REPLAYS times; the step time is
        # the median over the replays of replay time / K.  Event records are
        # not captured (ROCm graphs have no timed event nodes), which is why
        # the kernel durations come from the pass above.
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        # the captured GEMM launches take device-timestamp slots, so their
        # durations inside the replays can be read back (no event can be
        # recorded between the kernels of a graph)
        moe.timing_device_clear()
        moe.timing_device_enable(True)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(args.steps):
                step()
        moe.timing_device_enable(False)
        graph.replay()  # untimed: first replay of the graph
        torch.cuda.synchronize()
        for r in range(REPLAYS):
            if r == REPLAYS - 1:
                moe.timing_device_reset()  # the last timed replay also gives the GEMMs' device times
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            graph.replay()
            b.record()
            torch.cuda.synchronize()
            replay_ms.append(a.elapsed_time(b) / args.steps)
        ms_per_step = float(np.median(replay_ms))
        for kind in ("gate_up", "down"):
            ms, n = moe.timing_device_read(kind)
            if n:
                graph_kern[kind] = dict(avg_us=1e3 * ms / n, launches=n)
        graph_kern_replay_ms = replay_ms[-1]
        del graph
        # Latency view: one step per graph, replayed K times in a row with an
        # event between consecutive replays (replay i takes from event i to
        # event i+1; the host queues replays faster than the GPU runs them).
        # Each replay ends the graph, whose completion writes back the step's
        # outputs from the caches: reported beside the throughput figure.
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        graph.replay()
        torch.cuda.synchronize()
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 2)]
        graph.replay()  # keeps the stream busy while the timed replays are queued
        marks[0].record()
        for i in range(args.steps + 1):
            graph.replay()
            marks[i + 1].record()
        torch.cuda.synchronize()
        # the first timed replay may still have waited for the host: dropped
        single_ms = float(np.median([marks[i].elapsed_time(marks[i + 1]) for i in range(1, args.steps + 1)]))
        del graph

    # Cold steps: a 512 MiB buffer is written before each step (outside the
    # timed span), so the step finds no weights in L2 or the 256 MB MALL.
    cold_ms = None
    if headline and args.cold_steps > 0:
        scratch = torch.empty(256 << 20, dtype=torch.int16, device=dev)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.cold_steps)]
        for i, (a, b) in enumerate(ev):
            scratch.fill_(i)
            a.record()
            step()
            b.record()
        torch.cuda.synchronize()
        cold_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
        del scratch

    kern = {}
    for kind in moe.binding.KERNEL_KINDS:
        ms, n = moe.timing_read(kind)
        if n:
            kern[kind] = dict(avg_us=1e3 * ms / n, launches=n)
    log(f"[bench] {cfg.name}: step {ms_per_step:.4f} ms (median of {len(replay_ms)} replays of a "
        f"{args.steps}-step graph; {single_ms or 0:.4f} per one-step graph); kernels: " +
        ", ".join(f"{k}={v['avg_us']:.1f}us x{v['launches']}" for k, v in kern.items()) +
        "; in the graph: " + ", ".join(f"{k}={v['avg_us']:.1f}us" for k, v in graph_kern.items()) +
        (f" (replay step {graph_kern_replay_ms:.4f} ms)" if graph_kern_replay_ms else ""))

    decode = cfg.name.startswith("dsv3")
    # dominant kernel: the gate-up GEMM (2/3 of the flops and of the weight
    # bytes); its launches per step (the routed experts and, where present,
    # the shared expert) are summed.  Prefill is priced on MFMA, decode
    # (a few rows per expert, weights streamed once) on HBM.
    # The duration is the one inside the timed graph replays (device
    # timestamps); the host-launched pass's events are reported beside it.
    dom = "gate_up"
    gu = kern.get(dom)
    gg = graph_kern.get(dom)
    roof = None
    if gu is not None:
        per_step = gu["launches"] / args.steps
        ev_s = gu["avg_us"] * 1e-6 * per_step   # kernel time per step, events, host-launched pass
        dur_s = gg["avg_us"] * 1e-6 * per_step if gg else ev_s
        how = ("device timestamps of the launches in the last of the timed graph replays" if gg else
               "HIP events around the launches of the host-launched pass")
        if decode:
            achieved = work["gate_up_bytes"] / dur_s / 1e9
            roof = dict(bound="hbm", achieved=achieved, peak=PEAK_HBM_GBS, unit="GB/s",
                        frac=achieved / PEAK_HBM_GBS, traffic=measured_traffic(cfg.name, "step"), kernel=dom,
                        launches_per_step=per_step, algorithmic_per_step=work["gate_up_bytes"],
                        duration_us=dur_s * 1e6 / per_step, duration_from=how,
                        achieved_events_host_launched=work["gate_up_bytes"] / ev_s / 1e9)
        else:
            achieved = work["gate_up_flops"] / dur_s / 1e12
            roof = dict(bound="mfma", achieved=achieved, peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                        frac=achieved / PEAK_BF16_TFLOPS, traffic=measured_traffic(cfg.name), kernel=dom,
                        algorithmic_per_launch=work["gate_up_flops"],
                        algorithmic_bytes_per_launch=work["gate_up_bytes"],
                        duration_us=dur_s * 1e6 / per_step, duration_from=how,
                        achieved_events_host_launched=work["gate_up_flops"] / ev_s / 1e12)
    step_s = ms_per_step * 1e-3
    res = {
        "ms_per_step": ms_per_step,
        "ms_per_step_replays": replay_ms,
        "ms_per_step_single_step_graph": single_ms,
        "value": cfg.T / (cfg.P * step_s),
        "slice_tokens_per_s": cfg.T / step_s,
        "pairs_per_s": work["n"] / step_s,
        "chain_tflops": work["flops"] / step_s / 1e12,
        "chain_frac_mfma": work["flops"] / step_s / 1e12 / PEAK_BF16_TFLOPS,
        "chain_gbs": work["bytes"] / step_s / 1e9,
        "chain_frac_hbm": work["bytes"] / step_s / 1e9 / PEAK_HBM_GBS,
        "kernels_us": {k: round(v["avg_us"], 2) for k, v in kern.items()},
        "kernels_us_in_graph": {k: round(v["avg_us"], 2) for k, v in graph_kern.items()},
        "kernels_us_in_graph_replay_ms_per_step": graph_kern_replay_ms,
        "eager_ms_per_step": eager_ms,
        "cold_ms_per_step": cold_ms,
        "roofline": roof,
    }
    return res, inp, work, layer


def config_block(cfg, work, graph: bool):
    return {"workload": cfg.name, "T": cfg.T, "H": cfg.H, "E": cfg.E, "k": cfg.k,
            "I": cfg.I, "I_s": cfg.I_s, "P": cfg.P, "layout": cfg.layout, "rank": cfg.rank,
            "local_experts": cfg.E_l, "local_pairs": work["n"], "active_experts": work["active"],
            "shared_expert": cfg.shared, "global_batch": cfg.T, "parallelism": "single-gpu-slice",
            "graph": graph, "seed": cfg.seed}


# Workloads measured beside the headline one in the default run, with a
# shorter oracle sample each: the other prefill slices and both decode
# batch sizes (the metric's HBM half).
PER_CONFIG = ("c3", "c4", "c4h", "c5a", "c5b")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c2")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--eager", action="store_true",
                    help="report the host-launched kernel timing pass as the step time instead of "
                         "graph replays of the step")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--per-config-cpu-seconds", type=float, default=2.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--per-config", default=None,
                    help="comma-separated workloads measured beside the headline one "
                         "(default: the others of the five configs when --config is c2; 'none' skips)")
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="steps timed one by one after writing a 512 MiB buffer (caches flushed); 0 skips")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the vendor-GEMM and device-copy reference measurements")
    ap.add_argument("--crossover", action="store_true",
                    help="instead of one workload: time the TP and the EP slice of a Qwen3-235B-shaped "
                         "layer over a range of batch sizes (one JSON line per batch size)")
    ap.add_argument("--reshard", action="store_true",
                    help="instead of one workload: time the expert-weight reshard (EP <-> TP) of a "
                         "Qwen3-235B-shaped layer (one JSON line per case)")
    ap.add_argument("--kvmove", action="store_true",
                    help="instead of one workload: time the paged KV head moves of an EP->TP switch "
                         "for a decode batch (one JSON line per case)")
    ap.add_argument("--four-calls", action="store_true",
                    help="time the four calls (route, permute, grouped FFN, combine) instead of the one-call "
                         "layer forward")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="also run one device copy of this many MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the layer; --gpus {args.gpus} is not "
              "supported (libmoe has no multi-GPU collectives: the TP all-reduce and the EP "
              "all-to-alls are left to the caller)", file=sys.stderr)
        sys.exit(2)

    import torch
    import moe_inputs as mi
    import paper_2606_26607_amd as moe

    assert torch.cuda.is_available(), "bench needs a GPU"
    if args.four_calls:
        API[0] = "moe_route+moe_permute+moe_grouped_ffn+moe_combine"
    if args.crossover:
        crossover(args, torch, mi, moe)
        return
    if args.reshard:
        reshard_bench(args, torch, mi, moe)
        return
    if args.kvmove:
        kvmove_bench(args, torch, moe)
        return
    cfg = mi.CONFIGS[args.config]
    cfg = cfg.with_(seed=cfg.seed + args.seed)
    dev = torch.device("cuda:0")
    res, inp, work, layer = measure(cfg, args, torch, mi, moe, headline=True)
    roof = res["roofline"]
    decode = cfg.name.startswith("dsv3")

    # Measured ceilings on this GPU (references, not part of the path): the
    # vendor GEMM (torch.matmul, hipBLASLt) on the dense shape of the
    # gate-up GEMM, the library's matrix-core reference loop (bf16 MFMAs
    # with no memory traffic, on random and on zero operands), and a
    # device-to-device copy.
    ceilings = None
    if not args.no_ceilings:
        def timed(fn, reps=20):
            fn()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / reps * 1e-3
        ceilings = {}
        m = max(work["n"], 1)
        if not decode:
            A = torch.randn(m, cfg.H, device=dev).to(torch.bfloat16)
            B = torch.randn(cfg.H, 2 * cfg.I_s, device=dev).to(torch.bfloat16).contiguous()
            t = timed(lambda: torch.matmul(A, B))
            ceilings["vendor_gemm_tflops"] = 2.0 * m * cfg.H * 2 * cfg.I_s / t / 1e12
            ceilings["vendor_gemm_shape"] = [m, 2 * cfg.I_s, cfg.H]
            del A, B
            # the clock settles over the first calls of a sustained MFMA load:
            # the best of 8 back-to-back calls of about 6 ms each
            out = torch.empty(torch.cuda.get_device_properties(0).multi_processor_count * 512,
                              dtype=torch.float32, device=dev)
            for key, zero in (("mfma_loop_random_tflops", False), ("mfma_loop_zero_tflops", True)):
                best = 0.0
                for _ in range(8):
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record()
                    flops = moe.calib_mfma(out, 20000, zero_operands=zero)
                    b.record()
                    torch.cuda.synchronize()
                    best = max(best, flops / (a.elapsed_time(b) * 1e-3) / 1e12)
                ceilings[key] = best
            del out
        src = torch.empty(256 << 20, dtype=torch.int16, device=dev).fill_(1)
        dst = torch.empty_like(src)
        t = timed(lambda: dst.copy_(src), reps=10)
        ceilings["copy_gbs"] = 2.0 * src.numel() * 2 / t / 1e9
        del src, dst
        if roof is not None:
            if roof["bound"] == "mfma" and "vendor_gemm_tflops" in ceilings:
                roof["frac_of_vendor_gemm"] = roof["achieved"] / ceilings["vendor_gemm_tflops"]
                roof["frac_of_mfma_loop_random"] = roof["achieved"] / ceilings["mfma_loop_random_tflops"]
            if roof["bound"] == "hbm":
                roof["frac_of_copy"] = roof["achieved"] / ceilings["copy_gbs"]

    result = {
        "metric": METRIC,
        "value": res["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": config_block(cfg, work, not args.eager),
        "timing": f"median over {REPLAYS} replays of one HIP graph of the {args.steps} steps "
                  f"(replay time / {args.steps})" if not args.eager
                  else f"mean of {args.steps} host-launched steps",
    }
    result.update({k: v for k, v in res.items() if k not in ("value", "ms_per_step", "roofline")})
    result["ceilings"] = ceilings
    result["roofline"] = roof
    result["cpu_baseline"] = None
    cpu_name = cpu_model()
    if not args.no_cpu:
        cb = cpu_baseline(inp, args.cpu_seconds)
        log(f"[bench] cpu oracle: {cb['sample']} on {cb['cores']} threads ({cpu_name}); "
            f"{cb['gflops']:.2f} GFLOP/s")
        c1_s = cpu_single_thread_c1(mi)
        log(f"[bench] cpu oracle, tiny-replicated (64 tokens) on 1 thread: {c1_s:.3f} s")
        result["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample")}
        result["cpu_baseline"].update(cpu=cpu_name, gflops=cb["gflops"], seconds=cb["seconds"],
                                      c1_single_thread_s=c1_s)
    del layer, inp

    # The other workloads, each with its own step time, roofline (MFMA for
    # prefill, HBM for decode), counter traffic where committed, and a short
    # oracle sample timed on the same host.
    names = args.per_config
    if names is None:
        names = ",".join(PER_CONFIG) if args.config == "c2" else "none"
    per = {}
    if names != "none":
        for key in names.split(","):
            c = mi.CONFIGS[key]
            c = c.with_(seed=c.seed + args.seed)
            r, cinp, cwork, clayer = measure(c, args, torch, mi, moe, headline=False)
            entry = {"config": config_block(c, cwork, not args.eager),
                     "ms_per_step": r["ms_per_step"], "value": r["value"], "unit": "tokens/s",
                     "ms_per_step_single_step_graph": r["ms_per_step_single_step_graph"],
                     "kernels_us": r["kernels_us"], "kernels_us_in_graph": r["kernels_us_in_graph"],
                     "roofline": r["roofline"],
                     "chain_frac_mfma": r["chain_frac_mfma"], "chain_frac_hbm": r["chain_frac_hbm"],
                     "chain_tflops": r["chain_tflops"], "chain_gbs": r["chain_gbs"],
                     "eager_ms_per_step": r["eager_ms_per_step"]}
            if not args.no_cpu:
                cb = cpu_baseline(cinp, args.per_config_cpu_seconds)
                entry["oracle"] = {"seconds": cb["seconds"], "tokens_per_s": cb["value"],
                                   "gflops": cb["gflops"], "cores": cb["cores"], "sample": cb["sample"]}
                log(f"[bench] cpu oracle {c.name}: {cb['sample']}; {cb['gflops']:.2f} GFLOP/s")
            per[c.name] = entry
            del clayer, cinp
            torch.cuda.empty_cache()
    if per:
        result["per_config"] = per
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

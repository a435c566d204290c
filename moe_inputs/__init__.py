"""Seeded synthetic inputs for the MoE layer forward (shared by the GPU path's
tests/bench and by the CPU oracle's tests).

This module only *draws* inputs: token activations, router logits, expert
weights and the per-rank slicing of those weights.  It holds none of the
layer's own arithmetic (routing, permutation, expert FFN, combine).

Shapes follow the paper's statement of the two expert layouts (Sec. 3.1,
"Weights Resharding"):

* expert-parallel (EP): a rank owns E/P whole experts,
  W13 (E/P, 2I, H) with the gate projection stacked before the up
  projection, and W2 (E/P, H, I);
* tensor-parallel (TP): a rank owns one I/P slice of every expert,
  W13 (E, 2I/P, H) and W2 (E, H, I/P).  Gate-up is sliced along its output
  intermediate dimension and down along its input intermediate dimension;
  the rank keeps the *matching* gate and up rows so SwiGLU stays local.

The paper's workloads (Qwen3-235B weights, ShareGPT, DeepMath) are not
available; these synthetic layers stand in for them, with the model shapes
of Mixtral, Qwen-MoE and DeepSeek-V3.

Random draws are keyed per (tensor, expert, chunk of rows), so a TP or EP
slice of a weight is generated without generating the whole weight, and the
slices of all P ranks concatenate to exactly the unsliced tensor.  The chunk
is 64 rows when I is a multiple of 512 and 8 rows otherwise; a TP slice
width must be a multiple of it.
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import math
import os
from typing import Optional

import numpy as np

# Distinct stream tags for each drawn tensor.
_TAG_X, _TAG_WR, _TAG_W1, _TAG_W3, _TAG_W2 = 11, 12, 13, 14, 15
_TAG_SW1, _TAG_SW3, _TAG_SW2, _TAG_ZIPF, _TAG_Y, _TAG_W = 16, 17, 18, 19, 20, 21
EXPERT_STD = 0.02


def weight_chunk(I: int) -> int:
    """Rows (W1/W3) or columns (W2) drawn per generator stream."""
    return 64 if I % 512 == 0 else 8


@dataclasses.dataclass(frozen=True)
class MoeConfig:
    """One MoE layer and the slice of it that one GPU computes."""
    name: str
    T: int                 # tokens in the step
    H: int                 # hidden size
    E: int                 # routed experts
    k: int                 # experts per token
    I: int                 # full expert intermediate size
    P: int = 1             # ranks in the TP/EP group
    layout: str = "replicated"   # "replicated" | "tp" | "ep"
    rank: int = 0
    zipf_s: Optional[float] = None   # per-expert Zipf log-bias on the logits
    zipf_hot: bool = False  # Zipf popularity rank = expert id (rank 0 holds the hottest experts)
    shared: bool = False   # one shared expert, applied to the rank's DP share
    seed: int = 0

    # ---- derived slice geometry ----
    @property
    def e0(self) -> int:
        return self.rank * (self.E // self.P) if self.layout == "ep" else 0

    @property
    def E_l(self) -> int:
        return self.E // self.P if self.layout == "ep" else self.E

    @property
    def I_s(self) -> int:
        return self.I // self.P if self.layout == "tp" else self.I

    @property
    def cap(self) -> int:
        """Rows the permuted buffers must hold: dropless, T*min(k, E_l)."""
        return self.T * min(self.k, self.E_l)

    @property
    def shared_begin(self) -> int:
        return self.rank * (self.T // self.P) if self.shared else 0

    @property
    def shared_count(self) -> int:
        return self.T // self.P if self.shared else 0

    @property
    def router_std(self) -> float:
        return 1.0 / math.sqrt(self.H)

    def validate(self) -> None:
        assert self.layout in ("replicated", "tp", "ep")
        assert 1 <= self.k <= self.E
        if self.layout == "replicated":
            assert self.P == 1
        if self.layout == "ep":
            assert self.E % self.P == 0
        if self.layout == "tp":
            assert self.I % self.P == 0 and (self.I // self.P) % weight_chunk(self.I) == 0
        assert 0 <= self.rank < self.P
        assert self.H % 8 == 0 and self.I % 8 == 0

    def with_(self, **kw) -> "MoeConfig":
        return dataclasses.replace(self, **kw)


# The five workloads: one tiny replicated layer, three prefill-sized slices
# (the Qwen-shaped one also in a skew-stress variant) and one decode-sized
# slice at two batch sizes.  Seeds are 1000 + index.
CONFIGS = {
    "c1": MoeConfig("tiny-replicated", T=64, H=256, E=8, k=2, I=512, P=1,
                    layout="replicated", seed=1000),
    "c2": MoeConfig("mixtral-tp8-slice", T=4096, H=4096, E=8, k=2, I=14336,
                    P=8, layout="tp", seed=1001),
    "c3": MoeConfig("mixtral-ep8-slice", T=4096, H=4096, E=8, k=2, I=14336,
                    P=8, layout="ep", seed=1002),
    "c4": MoeConfig("qwen-moe-ep8-slice-zipf", T=8192, H=2048, E=128, k=8,
                    I=768, P=8, layout="ep", zipf_s=1.2, seed=1003),
    # stress variant of the Qwen-shaped slice: popularity follows the expert
    # id, so rank 0's 16 experts are the 16 most popular (about 56k pairs)
    "c4h": MoeConfig("qwen-moe-ep8-slice-zipf-hot", T=8192, H=2048, E=128, k=8,
                     I=768, P=8, layout="ep", zipf_s=1.2, zipf_hot=True, seed=1003),
    "c5a": MoeConfig("dsv3-ep8-decode-t64", T=64, H=7168, E=256, k=8, I=2048,
                     P=8, layout="ep", shared=True, seed=1004),
    "c5b": MoeConfig("dsv3-ep8-decode-t512", T=512, H=7168, E=256, k=8,
                     I=2048, P=8, layout="ep", shared=True, seed=1004),
}


# ---------------------------------------------------------------- helpers
def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns
    the uint16 bit patterns.  Inputs are finite."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _normal_bf16(shape, std: float, *key: int) -> np.ndarray:
    g = _rng(*key).standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        g *= np.float32(std)
    return f32_to_bf16_bits(g)


def _rows(tag: int, seed: int, e: int, r0: int, r1: int, H: int, std: float, ch: int) -> np.ndarray:
    """Rows [r0, r1) of a (rows, H) weight, drawn in chunks of ch rows."""
    assert r0 % ch == 0 and r1 % ch == 0
    out = np.empty((r1 - r0, H), dtype=np.uint16)
    for c in range(r0 // ch, r1 // ch):
        out[c * ch - r0:(c + 1) * ch - r0] = _normal_bf16((ch, H), std, seed, tag, e, c)
    return out


def _cols(tag: int, seed: int, e: int, c0: int, c1: int, H: int, std: float, ch: int) -> np.ndarray:
    """Columns [c0, c1) of an (H, I) weight, drawn in chunks of ch columns."""
    assert c0 % ch == 0 and c1 % ch == 0
    out = np.empty((H, c1 - c0), dtype=np.uint16)
    for c in range(c0 // ch, c1 // ch):
        out[:, c * ch - c0:(c + 1) * ch - c0] = _normal_bf16((H, ch), std, seed, tag, e, c)
    return out


# ---------------------------------------------------------------- inputs
def qwen3_layer(B: int, layout: str, rank: int = 0) -> MoeConfig:
    """One rank's slice (TP or EP, P = 8) of a Qwen3-235B-shaped MoE layer
    (H 4096, 128 experts, top-8, expert intermediate 1536; dimensions from
    the public model configuration) for a step of B tokens.  The weights do
    not depend on B."""
    return MoeConfig(f"qwen3-235b-{layout}8-b{B}", T=B, H=4096, E=128, k=8, I=1536, P=8,
                     layout=layout, rank=rank, seed=1100)


@dataclasses.dataclass
class MoeInputs:
    cfg: MoeConfig
    x: np.ndarray          # [T, H] bf16 bits
    logits: np.ndarray     # [T, E] float32
    w13: np.ndarray        # [E_l, 2*I_s, H] bf16 bits, gate rows then up rows
    w2: np.ndarray         # [E_l, H, I_s] bf16 bits
    sw13: Optional[np.ndarray] = None   # shared expert [1, 2*I, H]
    sw2: Optional[np.ndarray] = None    # shared expert [1, H, I]


def make_x(cfg: MoeConfig) -> np.ndarray:
    return _normal_bf16((cfg.T, cfg.H), 1.0, cfg.seed, _TAG_X)


def make_router(cfg: MoeConfig) -> np.ndarray:
    return _normal_bf16((cfg.E, cfg.H), cfg.router_std, cfg.seed, _TAG_WR)


def zipf_bias(cfg: MoeConfig) -> np.ndarray:
    """Log of a Zipf(s) popularity over experts, up to a constant:
    bias_e = -s * ln(pi(e)) with pi a seeded permutation of 1..E (the
    identity with zipf_hot: expert 0 the most popular)."""
    if cfg.zipf_s is None:
        return np.zeros(cfg.E, dtype=np.float32)
    if cfg.zipf_hot:
        perm = np.arange(cfg.E) + 1
    else:
        perm = _rng(cfg.seed, _TAG_ZIPF).permutation(cfg.E) + 1
    return (-cfg.zipf_s * np.log(perm.astype(np.float64))).astype(np.float32)


def make_logits(cfg: MoeConfig, x: np.ndarray) -> np.ndarray:
    """Router logits, the fp32 input that the routing step receives:
    fp32(sum_h x*Wr in fp64) + bias (fp32 add)."""
    wr = bf16_bits_to_f32(make_router(cfg)).astype(np.float64)
    xf = bf16_bits_to_f32(x).astype(np.float64)
    lg = (xf @ wr.T).astype(np.float32)
    return lg + zipf_bias(cfg)[None, :]


def expert_weights(cfg: MoeConfig, e: int):
    """This rank's slice of routed expert e (a global expert id):
    (w13 [2*I_s, H], w2 [H, I_s])."""
    c0 = cfg.rank * cfg.I_s if cfg.layout == "tp" else 0
    c1 = c0 + cfg.I_s
    ch = weight_chunk(cfg.I)
    g = _rows(_TAG_W1, cfg.seed, e, c0, c1, cfg.H, EXPERT_STD, ch)
    u = _rows(_TAG_W3, cfg.seed, e, c0, c1, cfg.H, EXPERT_STD, ch)
    w2 = _cols(_TAG_W2, cfg.seed, e, c0, c1, cfg.H, EXPERT_STD, ch)
    return np.concatenate([g, u], axis=0), w2


def shared_weights(cfg: MoeConfig):
    ch = weight_chunk(cfg.I)
    g = _rows(_TAG_SW1, cfg.seed, 0, 0, cfg.I, cfg.H, EXPERT_STD, ch)
    u = _rows(_TAG_SW3, cfg.seed, 0, 0, cfg.I, cfg.H, EXPERT_STD, ch)
    w2 = _cols(_TAG_SW2, cfg.seed, 0, 0, cfg.I, cfg.H, EXPERT_STD, ch)
    return np.concatenate([g, u], axis=0)[None], w2[None]


def make_inputs(cfg: MoeConfig, with_weights: bool = True) -> MoeInputs:
    cfg.validate()
    x = make_x(cfg)
    logits = make_logits(cfg, x)
    El, Is, H = cfg.E_l, cfg.I_s, cfg.H
    if with_weights:
        w13 = np.empty((El, 2 * Is, H), dtype=np.uint16)
        w2 = np.empty((El, H, Is), dtype=np.uint16)

        def fill(le):
            w13[le], w2[le] = expert_weights(cfg, cfg.e0 + le)
        workers = max(1, min(8, El, len(os.sched_getaffinity(0))))
        with cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(El)))
    else:
        w13 = np.empty((El, 2 * Is, H), dtype=np.uint16)[:0]
        w2 = np.empty((El, H, Is), dtype=np.uint16)[:0]
    sw13 = sw2 = None
    if cfg.shared and with_weights:
        sw13, sw2 = shared_weights(cfg)
    return MoeInputs(cfg, x, logits, w13, w2, sw13, sw2)


# ------------------------------------------------- stage-level test inputs
def random_topk_ids(T: int, E: int, k: int, seed: int, hot: Optional[int] = None) -> np.ndarray:
    """Distinct expert ids per token (as routing would produce); with `hot`
    set, every token's first choice is that expert."""
    g = _rng(seed, 31)
    ids = np.argsort(g.random((T, E)), axis=1)[:, :k].astype(np.int32)
    if hot is not None:
        for t in range(T):
            row = ids[t]
            w = np.where(row == hot)[0]
            if w.size:
                row[w[0]] = row[0]
            row[0] = hot
    return np.ascontiguousarray(ids)


def random_bf16(shape, seed: int, tag: int = _TAG_Y, std: float = 1.0) -> np.ndarray:
    return _normal_bf16(shape, std, seed, tag)


def random_gate_weights(T: int, k: int, seed: int) -> np.ndarray:
    """Positive fp32 weights per token (stage input for the combine step)."""
    g = _rng(seed, _TAG_W).random((T, k), dtype=np.float32) + np.float32(0.05)
    return np.ascontiguousarray(g)

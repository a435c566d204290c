"""Thin ctypes binding over libmoe.so (the C ABI in include/libmoe.h).

Each function takes torch tensors that already live on the GPU, checks
dtype/shape/contiguity, and passes raw device pointers plus the current HIP
stream to the library.  No arithmetic of the layer happens here: every step
runs in the library's HIP kernels.  If libmoe.so is missing the import of a
call raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoe.so")

MAX_TOPK = 16
MAX_EXPERTS = 1024
KERNEL_KINDS = {"route": 0, "permute": 1, "gather": 2, "schedule": 3, "gate_up": 4, "down": 5,
                "combine": 6, "splitk_reduce": 7, "reshard": 8, "kv_move": 9, "layer_prep": 10}
EP_TO_TP, TP_TO_EP = 0, 1
MODE_TP, MODE_EP = 0, 1
STAY, SWITCH, SWITCH_CANCELLED = 0, 1, 2
POLICY_MAX_WINDOW = 1024


class _Policy(ctypes.Structure):
    """struct moe_policy (include/libmoe.h)."""
    _fields_ = [("t_high", ctypes.c_double), ("t_low", ctypes.c_double), ("cooldown_s", ctypes.c_double),
                ("window", ctypes.c_int32), ("mode", ctypes.c_int32), ("n_hist", ctypes.c_int32),
                ("head", ctypes.c_int32), ("has_event", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("last_event_s", ctypes.c_double), ("hist_sum", ctypes.c_int64),
                ("hist", ctypes.c_int64 * POLICY_MAX_WINDOW)]


class MoeError(RuntimeError):
    """A libmoe call returned a non-OK status."""

    def __init__(self, status: int, name: str, msg: str):
        super().__init__(f"{name}: {msg}")
        self.status = status
        self.name = name


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libmoe.so not found at {LIB_PATH}; build it with "
                          "`python -m paper_2606_26607_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    i64, i32, vp, sz = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
    sigs = {
        "moe_status_str": ([i32], ctypes.c_char_p),
        "moe_last_error": ([], ctypes.c_char_p),
        "moe_version": ([], i32),
        "moe_route": ([vp, i64, i32, i32, vp, vp, vp], i32),
        "moe_permute_workspace_size": ([i64, i32, i32], sz),
        "moe_permute": ([vp, i64, i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, vp, vp, sz, vp], i32),
        "moe_permute_noalloc": ([vp, i64, i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, vp, vp], i32),
        "moe_ffn_workspace_size": ([i64, i32, i32, i32], sz),
        "moe_grouped_ffn": ([vp, i64, vp, i32, vp, i32, i64, i32, i32, vp, vp, vp, vp, sz, vp], i32),
        "moe_grouped_ffn_shared": ([vp, i64, vp, i32, vp, i32, i64, i32, i32, vp, vp, vp, i64, i64, vp, vp, vp,
                                    vp, sz, vp], i32),
        "moe_layer_workspace_size": ([i64, i32, i32, i32, i32, i64], sz),
        "moe_layer_forward": ([vp, vp, i64, i32, i32, i32, i32, i32, i32, vp, vp, i64, i64, vp, vp, vp, vp, vp, vp,
                               vp, vp, vp, vp, vp, vp, sz, vp], i32),
        "moe_combine": ([vp, i64, vp, vp, i64, i32, i32, vp, i64, i64, i32, vp, vp], i32),
        "moe_reshard_experts": ([i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp], i32),
        "moe_kv_slots": ([vp, i64, vp, i32, i32, vp, i64, vp], i32),
        "moe_kv_move": ([i32, vp, vp, vp, vp, i32, vp, vp, i64, i32, i32, i32, i32, i32, vp, vp, vp], i32),
        "moe_policy_init": ([ctypes.POINTER(_Policy), ctypes.c_double, ctypes.c_double, i32, ctypes.c_double,
                             i32], i32),
        "moe_policy_step": ([ctypes.POINTER(_Policy), i64, ctypes.c_double, i32, ctypes.POINTER(ctypes.c_int)],
                            i32),
        "moe_partition_requests": ([vp, i32, i32, vp, vp, vp], i32),
        "moe_kv_fits": ([i32, vp, i32, vp, i32, i32, i32, i64, ctypes.POINTER(ctypes.c_int)], i32),
        "moe_policy_crossover": ([vp, vp, vp, i32, ctypes.POINTER(ctypes.c_double)], i32),
        "moe_timing_device_enable": ([i32], i32),
        "moe_timing_device_clear": ([], i32),
        "moe_timing_device_reset": ([], i32),
        "moe_timing_device_read": ([i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)], i32),
        "moe_timing_enable": ([i32], i32),
        "moe_timing_enable_mask": ([ctypes.c_uint32], i32),
        "moe_timing_reset": ([], i32),
        "moe_timing_read": ([i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)], i32),
        "moe_calib_mfma": ([i32, i32, i32, vp, vp], i32),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _check(status: int) -> None:
    if status != 0:
        L = lib()
        raise MoeError(status, L.moe_status_str(status).decode(), L.moe_last_error().decode())


def _stream(stream=None) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream or None


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else (t.data_ptr() or None)


def _need(t: torch.Tensor, dtype, name: str, ndim: Optional[int] = None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")


# ------------------------------------------------------------- the 4 calls
def route(logits: torch.Tensor, k: int, topk_ids: Optional[torch.Tensor] = None,
          topk_w: Optional[torch.Tensor] = None, stream=None):
    _need(logits, torch.float32, "logits", 2)
    T, E = logits.shape
    if topk_ids is None:
        topk_ids = torch.empty((T, k), dtype=torch.int32, device=logits.device)
    if topk_w is None:
        topk_w = torch.empty((T, k), dtype=torch.float32, device=logits.device)
    _check(lib().moe_route(_ptr(logits), T, E, k, _ptr(topk_ids), _ptr(topk_w), _stream(stream)))
    return topk_ids, topk_w


def permute_workspace_size(T: int, k: int, n_local: int) -> int:
    return int(lib().moe_permute_workspace_size(T, k, n_local))


def ffn_workspace_size(cap_rows: int, n_local: int, H: int, I_s: int) -> int:
    return int(lib().moe_ffn_workspace_size(cap_rows, n_local, H, I_s))


def layer_workspace_size(T: int, k: int, n_local: int, H: int, I_s: int, shared_count: int = 0) -> int:
    return int(lib().moe_layer_workspace_size(T, k, n_local, H, I_s, shared_count))


def permute(topk_ids: torch.Tensor, E: int, expert_begin: int, n_local: int,
            x: Optional[torch.Tensor] = None, gather: bool = True, out: Optional[dict] = None,
            workspace: Optional[torch.Tensor] = None, stream=None) -> dict:
    _need(topk_ids, torch.int32, "topk_ids", 2)
    T, k = topk_ids.shape
    dev = topk_ids.device
    cap = T * min(k, n_local)
    o = dict(out or {})
    o.setdefault("counts", torch.empty(n_local, dtype=torch.int32, device=dev))
    o.setdefault("offsets", torch.empty(n_local + 1, dtype=torch.int32, device=dev))
    o.setdefault("row_to_pair", torch.empty(max(cap, 1), dtype=torch.int32, device=dev))
    o.setdefault("pair_to_row", torch.empty(max(T * k, 1), dtype=torch.int32, device=dev))
    H = 0
    if x is not None and gather:
        _need(x, torch.bfloat16, "x", 2)
        H = x.shape[1]
        o.setdefault("x_perm", torch.empty((max(cap, 1), H), dtype=torch.bfloat16, device=dev))
    else:
        o["x_perm"] = None
    if workspace is None:
        workspace = torch.empty(permute_workspace_size(T, k, n_local), dtype=torch.uint8, device=dev)
    _check(lib().moe_permute(_ptr(topk_ids), T, k, E, expert_begin, n_local, _ptr(o["counts"]),
                             _ptr(o["offsets"]), _ptr(o["row_to_pair"]), _ptr(o["pair_to_row"]),
                             _ptr(x) if o["x_perm"] is not None else None, H, _ptr(o["x_perm"]),
                             _ptr(workspace), workspace.numel(), _stream(stream)))
    return o


def grouped_ffn(x: torch.Tensor, offsets: torch.Tensor, w13: torch.Tensor, w2: torch.Tensor,
                row_to_pair: Optional[torch.Tensor] = None, k: int = 1, cap_rows: Optional[int] = None,
                y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """SwiGLU expert FFN over the expert row blocks given by `offsets`.

    Without `row_to_pair`, `x` is an already permuted [cap_rows, H] buffer.
    With it, `x` is the token matrix and row r's input is
    x[row_to_pair[r] // k] (the row gather is fused into the GEMM).
    """
    _need(x, torch.bfloat16, "x", 2)
    _need(offsets, torch.int32, "offsets", 1)
    _need(w13, torch.bfloat16, "w13", 3)
    _need(w2, torch.bfloat16, "w2", 3)
    x_rows, H = x.shape
    if row_to_pair is not None:
        _need(row_to_pair, torch.int32, "row_to_pair", 1)
        cap = row_to_pair.numel() if cap_rows is None else cap_rows
        if row_to_pair.numel() < cap:
            raise ValueError("row_to_pair must hold cap_rows entries")
    else:
        cap = x_rows if cap_rows is None else cap_rows
    El = offsets.numel() - 1
    I_s = w2.shape[2]
    if tuple(w13.shape) != (El, 2 * I_s, H) or tuple(w2.shape) != (El, H, I_s):
        raise ValueError(f"weight shapes {tuple(w13.shape)}, {tuple(w2.shape)} do not match "
                         f"El={El}, H={H}, I_s={I_s}")
    if y is None:
        y = torch.empty((max(cap, 1), H), dtype=torch.bfloat16, device=x.device)
    _need(y, torch.bfloat16, "y", 2)
    if y.shape[0] < cap or y.shape[1] != H:
        raise ValueError("y must be [cap_rows, H]")
    if workspace is None:
        workspace = torch.empty(ffn_workspace_size(cap, El, H, I_s), dtype=torch.uint8, device=x.device)
    _check(lib().moe_grouped_ffn(_ptr(x), x_rows, _ptr(row_to_pair), k, _ptr(offsets), El, cap, H, I_s,
                                 _ptr(w13), _ptr(w2), _ptr(y), _ptr(workspace), workspace.numel(),
                                 _stream(stream)))
    return y


def grouped_ffn_shared(x: torch.Tensor, offsets: torch.Tensor, w13: torch.Tensor, w2: torch.Tensor,
                       row_to_pair: torch.Tensor, k: int, cap_rows: int, shared_begin: int,
                       shared_count: int, sw13: torch.Tensor, sw2: torch.Tensor,
                       y: Optional[torch.Tensor] = None, shared_y: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None):
    """The routed experts' FFN (rows gathered through `row_to_pair`) and the
    shared expert's FFN on x[shared_begin : shared_begin + shared_count], in
    the same launches.  Returns (y, shared_y)."""
    _need(x, torch.bfloat16, "x", 2)
    _need(offsets, torch.int32, "offsets", 1)
    _need(w13, torch.bfloat16, "w13", 3)
    _need(w2, torch.bfloat16, "w2", 3)
    _need(row_to_pair, torch.int32, "row_to_pair", 1)
    _need(sw13, torch.bfloat16, "sw13", 2)
    _need(sw2, torch.bfloat16, "sw2", 2)
    x_rows, H = x.shape
    El = offsets.numel() - 1
    I_s = w2.shape[2]
    if tuple(w13.shape) != (El, 2 * I_s, H) or tuple(w2.shape) != (El, H, I_s):
        raise ValueError(f"weight shapes {tuple(w13.shape)}, {tuple(w2.shape)} do not match "
                         f"El={El}, H={H}, I_s={I_s}")
    if tuple(sw13.shape) != (2 * I_s, H) or tuple(sw2.shape) != (H, I_s):
        raise ValueError("the shared expert must have the routed experts' shapes")
    if row_to_pair.numel() < cap_rows:
        raise ValueError("row_to_pair must hold cap_rows entries")
    if y is None:
        y = torch.empty((max(cap_rows, 1), H), dtype=torch.bfloat16, device=x.device)
    if shared_y is None:
        shared_y = torch.empty((max(shared_count, 1), H), dtype=torch.bfloat16, device=x.device)
    _need(y, torch.bfloat16, "y", 2)
    _need(shared_y, torch.bfloat16, "shared_y", 2)
    if y.shape[0] < cap_rows or y.shape[1] != H or shared_y.shape[0] < shared_count or shared_y.shape[1] != H:
        raise ValueError("y must be [cap_rows, H] and shared_y [shared_count, H]")
    ne = El + (1 if shared_count > 0 else 0)
    if workspace is None:
        workspace = torch.empty(ffn_workspace_size(cap_rows + shared_count, ne, H, I_s), dtype=torch.uint8,
                                device=x.device)
    _check(lib().moe_grouped_ffn_shared(_ptr(x), x_rows, _ptr(row_to_pair), k, _ptr(offsets), El, cap_rows,
                                        H, I_s, _ptr(w13), _ptr(w2), _ptr(y), shared_begin, shared_count,
                                        _ptr(sw13), _ptr(sw2), _ptr(shared_y), _ptr(workspace),
                                        workspace.numel(), _stream(stream)))
    return y, shared_y


def combine(y: torch.Tensor, pair_to_row: torch.Tensor, topk_w: torch.Tensor,
            out: Optional[torch.Tensor] = None, shared_y: Optional[torch.Tensor] = None,
            shared_begin: int = 0, accumulate: bool = False, stream=None) -> torch.Tensor:
    _need(y, torch.bfloat16, "y", 2)
    _need(topk_w, torch.float32, "topk_w", 2)
    _need(pair_to_row, torch.int32, "pair_to_row")
    T, k = topk_w.shape
    H = y.shape[1]
    if pair_to_row.numel() < T * k:
        raise ValueError("pair_to_row must hold T*k entries")
    if out is None:
        out = torch.empty((T, H), dtype=torch.bfloat16, device=y.device)
    _need(out, torch.bfloat16, "out", 2)
    sc = 0
    if shared_y is not None:
        _need(shared_y, torch.bfloat16, "shared_y", 2)
        sc = shared_y.shape[0]
    _check(lib().moe_combine(_ptr(y), y.shape[0], _ptr(pair_to_row), _ptr(topk_w), T, k, H,
                             _ptr(shared_y), shared_begin, sc, 1 if accumulate else 0, _ptr(out),
                             _stream(stream)))
    return out


# ------------------------------------------------------------ resharding
def reshard_experts(direction: int, rank: int, E: int, H: int, I: int, src_w13: list, src_w2: list,
                    dst_w13: torch.Tensor, dst_w2: torch.Tensor, stream=None) -> None:
    """Write rank `rank`'s TP view (direction EP_TO_TP) or EP view
    (TP_TO_EP) of the expert weights from the other layout's views of ranks
    0..P-1 (P = len(src_w13)); a None source is skipped and the part of the
    destination it would supply is left as it was."""
    P = len(src_w13)
    if len(src_w2) != P:
        raise ValueError("src_w13 and src_w2 must list the same ranks")
    for t in list(src_w13) + list(src_w2):
        if t is not None:
            _need(t, torch.bfloat16, "source view", t.dim())
    _need(dst_w13, torch.bfloat16, "dst_w13", 3)
    _need(dst_w2, torch.bfloat16, "dst_w2", 3)
    arr = ctypes.c_void_p * max(P, 1)
    a13 = arr(*[_ptr(t) for t in src_w13])
    a2 = arr(*[_ptr(t) for t in src_w2])
    _check(lib().moe_reshard_experts(direction, P, rank, E, H, I, a13, a2, _ptr(dst_w13), _ptr(dst_w2),
                                     _stream(stream)))


class ExpertSlots:
    """One rank's expert weights for n_layers MoE layers in n_layers + 1
    fixed slots of one buffer, viewed either way: layer i's TP view lives in
    slot i and its EP view in slot i + 1, so a switch moves every layer into
    a slot other than the one it reads (EP->TP walks layers upward, TP->EP
    downward) and no buffer is allocated while switching.  Both views of a
    slot hold w13 then w2 (the same element counts)."""

    def __init__(self, n_layers: int, E: int, H: int, I: int, P: int, rank: int, device):
        self.n_layers, self.E, self.H, self.I, self.P, self.rank = n_layers, E, H, I, P, rank
        self.El, self.Is = E // P, I // P
        self.n13 = self.El * 2 * I * H
        self.slot = self.n13 + self.El * H * I
        self.buf = torch.empty((n_layers + 1) * self.slot, dtype=torch.bfloat16, device=device)

    def _views(self, s: int, layout: str):
        base = self.buf[s * self.slot:(s + 1) * self.slot]
        w13, w2 = base[:self.n13], base[self.n13:]
        if layout == "ep":
            return w13.view(self.El, 2 * self.I, self.H), w2.view(self.El, self.H, self.I)
        return w13.view(self.E, 2 * self.Is, self.H), w2.view(self.E, self.H, self.Is)

    def ep(self, layer: int):
        """(w13 [E/P, 2I, H], w2 [E/P, H, I]) of `layer` in the EP layout."""
        return self._views(layer + 1, "ep")

    def tp(self, layer: int):
        """(w13 [E, 2I/P, H], w2 [E, H, I/P]) of `layer` in the TP layout."""
        return self._views(layer, "tp")

    @staticmethod
    def switch(ranks: list, direction: int, stream=None) -> None:
        """Reshard every layer of every rank in `ranks` (all P ranks' slots,
        reachable from this process) into the other layout, in place."""
        first = ranks[0]
        layers = range(first.n_layers) if direction == EP_TO_TP else range(first.n_layers - 1, -1, -1)
        for i in layers:
            if direction == EP_TO_TP:
                srcs = [r.ep(i) for r in ranks]
                for r in ranks:
                    reshard_experts(direction, r.rank, r.E, r.H, r.I, [s[0] for s in srcs],
                                    [s[1] for s in srcs], *r.tp(i), stream=stream)
            else:
                srcs = [r.tp(i) for r in ranks]
                for r in ranks:
                    reshard_experts(direction, r.rank, r.E, r.H, r.I, [s[0] for s in srcs],
                                    [s[1] for s in srcs], *r.ep(i), stream=stream)


# ------------------------------------------------------------- KV moves
def kv_slots(page_table: torch.Tensor, first: torch.Tensor, page_size: int,
             out: Optional[torch.Tensor] = None, capacity: Optional[int] = None, stream=None) -> torch.Tensor:
    """Slot of every token of the requests (request order) from their page
    tables: page_table [n_req, pages_per_req] int32, first [n_req + 1] int32
    (exclusive prefix of the lengths); out [capacity] int32."""
    _need(page_table, torch.int32, "page_table", 2)
    _need(first, torch.int32, "first", 1)
    n_req = first.numel() - 1
    if page_table.shape[0] < n_req:
        raise ValueError("page_table has fewer rows than requests")
    if out is None:
        if capacity is None:
            raise ValueError("give out or capacity")
        out = torch.empty(max(capacity, 1), dtype=torch.int32, device=page_table.device)
    _need(out, torch.int32, "out", 1)
    cap = out.numel() if capacity is None else capacity
    _check(lib().moe_kv_slots(_ptr(page_table), page_table.stride(0), _ptr(first), n_req, page_size, _ptr(out),
                              cap, _stream(stream)))
    return out


def kv_move(src_k, src_v, dst_k: torch.Tensor, dst_v: Optional[torch.Tensor],
            src_slot: torch.Tensor, dst_slot: torch.Tensor, src_head0: int, dst_head0: int, n_heads: int,
            src_tokens=None, stream=None) -> None:
    """Copy heads [src_head0, +n_heads) of the listed source slots into heads
    [dst_head0, +n_heads) of the listed destination slots (pools [slots,
    heads, head_dim] bf16), for K and optionally V, in one launch.

    src_k / src_v: one pool or a list of pools (at most 16); with a list,
    src_tokens gives how many consecutive entries of the slot vectors each
    pool supplies.  With one pool src_tokens is that count (default: all
    entries)."""
    many = isinstance(src_k, (list, tuple))
    ks = list(src_k) if many else [src_k]
    vs = None if src_v is None else (list(src_v) if many else [src_v])
    if vs is not None and len(vs) != len(ks):
        raise ValueError("src_k and src_v must list the same pools")
    _need(src_slot, torch.int32, "src_slot", 1)
    _need(dst_slot, torch.int32, "dst_slot", 1)
    avail = min(src_slot.numel(), dst_slot.numel())
    if src_tokens is None:
        if many and len(ks) > 1:
            raise ValueError("give src_tokens for several source pools")
        counts = [avail]
    else:
        counts = list(src_tokens) if many else [src_tokens]
    if len(counts) != len(ks):
        raise ValueError("src_tokens needs one count per source pool")
    first = [0]
    for c in counts:
        if c < 0:
            raise ValueError("negative token count")
        first.append(first[-1] + int(c))
    if first[-1] > avail:
        raise ValueError("token counts exceed the slot vectors")
    _need(dst_k, torch.bfloat16, "dst_k", 3)
    if dst_v is not None:
        _need(dst_v, torch.bfloat16, "dst_v", 3)
        if dst_v.shape != dst_k.shape:
            raise ValueError("K and V pools must have the same shape")
    for q, k in enumerate(ks):
        _need(k, torch.bfloat16, "src_k", 3)
        if k.shape[1:] != ks[0].shape[1:]:
            raise ValueError("source pools must share heads and head_dim")
        if vs is not None:
            _need(vs[q], torch.bfloat16, "src_v", 3)
            if vs[q].shape != k.shape:
                raise ValueError("K and V pools must have the same shape")
    if ks[0].shape[2] != dst_k.shape[2]:
        raise ValueError("source and destination head_dim differ")
    n = len(ks)
    ak = (ctypes.c_void_p * n)(*[_ptr(t) for t in ks])
    av = None if vs is None else (ctypes.c_void_p * n)(*[_ptr(t) for t in vs])
    sl = (ctypes.c_int64 * n)(*[t.shape[0] for t in ks])
    fi = (ctypes.c_int64 * (n + 1))(*first)
    _check(lib().moe_kv_move(n, ak, av, sl, fi, ks[0].shape[1], _ptr(dst_k), _ptr(dst_v), dst_k.shape[0],
                             dst_k.shape[1], ks[0].shape[2], src_head0, dst_head0, n_heads, _ptr(src_slot),
                             _ptr(dst_slot), _stream(stream)))


# ------------------------------------------------- layout-switch control
def _host(a, dtype):
    """A contiguous host numpy array of `dtype` (a copy when needed)."""
    import numpy as np
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def _hptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a.size else None


class SwitchPolicy:
    """The layout-switch coordinator (host only): feed step() the global
    in-flight request count once per decode iteration; it returns STAY,
    SWITCH (mode has flipped) or SWITCH_CANCELLED (the other mode could not
    hold the live KV cache; retried after the cooldown)."""

    def __init__(self, t_high: float, t_low: float, window: int, cooldown_s: float, mode: int = MODE_TP):
        self._p = _Policy()
        _check(lib().moe_policy_init(ctypes.byref(self._p), t_high, t_low, window, cooldown_s, mode))

    @property
    def mode(self) -> int:
        return self._p.mode

    def step(self, in_flight: int, now_s: float, target_fits: bool = True) -> int:
        d = ctypes.c_int(-1)
        _check(lib().moe_policy_step(ctypes.byref(self._p), int(in_flight), float(now_s), 1 if target_fits else 0,
                                     ctypes.byref(d)))
        return d.value


def partition_requests(tokens, P: int):
    """Owner rank of every request for a TP->EP switch, plus each rank's
    token and request totals (numpy arrays)."""
    import numpy as np
    t = _host(tokens, np.int64)
    owner = np.empty(t.size, np.int32)
    rt = np.empty(P, np.int64)
    rr = np.empty(P, np.int32)
    _check(lib().moe_partition_requests(_hptr(t), t.size, P, _hptr(owner), _hptr(rt), _hptr(rr)))
    return owner, rt, rr


def kv_fits(mode: int, tokens, P: int, n_kv_heads: int, page_size: int, capacity: int, owner=None) -> bool:
    """Whether every rank's KV pool (`capacity` (page, head) units) holds the
    live requests in `mode` (EP needs the owner of every request)."""
    import numpy as np
    t = _host(tokens, np.int64)
    o = None if owner is None else _host(owner, np.int32)
    if o is not None and o.size != t.size:
        raise ValueError("owner needs one entry per request")
    f = ctypes.c_int(-1)
    _check(lib().moe_kv_fits(mode, _hptr(t), t.size, None if o is None else _hptr(o), P, n_kv_heads, page_size,
                             int(capacity), ctypes.byref(f)))
    return bool(f.value)


def policy_crossover(batch, tp_cost, ep_cost) -> float:
    """Initial switch threshold from decode costs probed in both modes."""
    import numpy as np
    b, tc, ec = _host(batch, np.int64), _host(tp_cost, np.float64), _host(ep_cost, np.float64)
    if not (b.size == tc.size == ec.size):
        raise ValueError("one cost per probed batch size in each mode")
    th = ctypes.c_double(0.0)
    _check(lib().moe_policy_crossover(_hptr(b), _hptr(tc), _hptr(ec), b.size, ctypes.byref(th)))
    return th.value


# ---------------------------------------------------------------- timing
def timing_enable(on: bool = True, kinds=None) -> None:
    """Time every kernel kind (on), none, or only the named `kinds`."""
    if kinds is None:
        _check(lib().moe_timing_enable(1 if on else 0))
    else:
        mask = 0
        for k in kinds:
            mask |= 1 << KERNEL_KINDS[k]
        _check(lib().moe_timing_enable_mask(mask if on else 0))


def timing_reset() -> None:
    _check(lib().moe_timing_reset())


def timing_read(kind: str):
    """(total milliseconds, launches) for one kernel kind since the last reset."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().moe_timing_read(KERNEL_KINDS[kind], ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ------------------------------------------------------------ the layer
class MoeLayer:
    """One GPU's share of an MoE layer forward with every buffer allocated
    once (fixed addresses, so the four-call chain can be replayed from a HIP
    graph).

    w13 [El, 2*I_s, H], w2 [El, H, I_s]: this rank's routed-expert weights
    (an EP slice of whole experts or a TP slice of every expert).  sw13/sw2:
    an optional shared expert applied with weight 1 to tokens
    [shared_begin, shared_begin + shared_count).
    """

    def __init__(self, T: int, E: int, k: int, expert_begin: int, w13: torch.Tensor,
                 w2: torch.Tensor, sw13: Optional[torch.Tensor] = None,
                 sw2: Optional[torch.Tensor] = None, shared_begin: int = 0, shared_count: int = 0):
        dev = w13.device
        self.T, self.E, self.k, self.e0 = T, E, k, expert_begin
        self.El, two_is, self.H = w13.shape
        self.I_s = two_is // 2
        self.w13, self.w2 = w13, w2
        self.cap = T * min(k, self.El)
        cap1 = max(self.cap, 1)
        self.topk_ids = torch.empty((T, k), dtype=torch.int32, device=dev)
        self.topk_w = torch.empty((T, k), dtype=torch.float32, device=dev)
        self.bufs = {
            "counts": torch.empty(self.El, dtype=torch.int32, device=dev),
            "offsets": torch.empty(self.El + 1, dtype=torch.int32, device=dev),
            "row_to_pair": torch.empty(cap1, dtype=torch.int32, device=dev),
            "pair_to_row": torch.empty(max(T * k, 1), dtype=torch.int32, device=dev),
        }
        self.ws_perm = torch.empty(max(permute_workspace_size(T, k, self.El), 256), dtype=torch.uint8,
                                   device=dev)
        self.ws_ffn = torch.empty(ffn_workspace_size(cap1, self.El, self.H, self.I_s), dtype=torch.uint8,
                                  device=dev)
        self.y = torch.empty((cap1, self.H), dtype=torch.bfloat16, device=dev)
        self.out = torch.empty((T, self.H), dtype=torch.bfloat16, device=dev)
        self.sw13, self.sw2 = sw13, sw2
        self.sb, self.sc = shared_begin, shared_count if sw13 is not None else 0
        # the shared expert joins the routed experts' launches when it has their
        # width and the large-tile kernels serve the shapes, else it is a
        # grouped FFN call of its own
        self.fused_shared = False
        if self.sc:
            sIs = sw2.shape[2]
            self.s_y = torch.empty((self.sc, self.H), dtype=torch.bfloat16, device=dev)
            self.fused_shared = (sIs == self.I_s and self.H % 64 == 0 and self.I_s % 64 == 0
                                 and self.H >= 128 and self.I_s >= 128)
            if self.fused_shared:
                self.sw13_2d, self.sw2_2d = sw13.reshape(2 * sIs, self.H), sw2.reshape(self.H, sIs)
                self.ws_ffn = torch.empty(ffn_workspace_size(cap1 + self.sc, self.El + 1, self.H, self.I_s),
                                          dtype=torch.uint8, device=dev)
            else:
                self.s_offsets = torch.tensor([0, self.sc], dtype=torch.int32, device=dev)
                self.ws_sh = torch.empty(ffn_workspace_size(self.sc, 1, self.H, sIs), dtype=torch.uint8,
                                         device=dev)

        # the whole-layer call (fused launches) serves every layer whose shared
        # expert, if any, shares the routed experts' launches
        self.one_call = self.sc == 0 or self.fused_shared
        if self.one_call:
            self.ws_layer = torch.empty(max(layer_workspace_size(T, k, self.El, self.H, self.I_s, self.sc), 256),
                                        dtype=torch.uint8, device=dev)
            if self.sc == 0:
                self.s_y = None

    def forward(self, x: torch.Tensor, logits: torch.Tensor, stream=None) -> torch.Tensor:
        """The layer forward: one moe_layer_forward call where it serves the
        layer, else the four calls."""
        if not self.one_call:
            return self.forward_calls(x, logits, stream)
        _need(x, torch.bfloat16, "x", 2)
        _need(logits, torch.float32, "logits", 2)
        if tuple(x.shape) != (self.T, self.H) or tuple(logits.shape) != (self.T, self.E):
            raise ValueError("x must be [T, H] and logits [T, E]")
        b = self.bufs
        _check(lib().moe_layer_forward(
            _ptr(x), _ptr(logits), self.T, self.E, self.k, self.e0, self.El, self.H, self.I_s, _ptr(self.w13),
            _ptr(self.w2), self.sb, self.sc, _ptr(self.sw13_2d) if self.sc else None,
            _ptr(self.sw2_2d) if self.sc else None, _ptr(self.topk_ids), _ptr(self.topk_w), _ptr(b["counts"]),
            _ptr(b["offsets"]), _ptr(b["row_to_pair"]), _ptr(b["pair_to_row"]), _ptr(self.y), _ptr(self.s_y),
            _ptr(self.out), _ptr(self.ws_layer), self.ws_layer.numel(), _stream(stream)))
        return self.out

    def forward_calls(self, x: torch.Tensor, logits: torch.Tensor, stream=None) -> torch.Tensor:
        """The same forward as the four calls route, permute, grouped FFN and
        combine, each with its own launches."""
        route(logits, self.k, self.topk_ids, self.topk_w, stream=stream)
        # the permutation's row gather is fused into the gate-up GEMM
        permute(self.topk_ids, self.E, self.e0, self.El, out=self.bufs, workspace=self.ws_perm,
                stream=stream)
        shared_y = None
        if self.fused_shared:
            grouped_ffn_shared(x, self.bufs["offsets"], self.w13, self.w2, self.bufs["row_to_pair"], self.k,
                               self.cap, self.sb, self.sc, self.sw13_2d, self.sw2_2d, y=self.y,
                               shared_y=self.s_y, workspace=self.ws_ffn, stream=stream)
            shared_y = self.s_y
        else:
            grouped_ffn(x, self.bufs["offsets"], self.w13, self.w2, row_to_pair=self.bufs["row_to_pair"],
                        k=self.k, cap_rows=self.cap, y=self.y, workspace=self.ws_ffn, stream=stream)
            if self.sc:
                grouped_ffn(x[self.sb:self.sb + self.sc], self.s_offsets, self.sw13, self.sw2, y=self.s_y,
                            workspace=self.ws_sh, stream=stream)
                shared_y = self.s_y
        combine(self.y, self.bufs["pair_to_row"], self.topk_w, out=self.out, shared_y=shared_y,
                shared_begin=self.sb, stream=stream)
        return self.out


def timing_device_enable(on: bool) -> None:
    """Grouped GEMM launches made while on take device-timestamp slots
    (captured launches too, so graph replays are timed)."""
    _check(lib().moe_timing_device_enable(1 if on else 0))


def timing_device_clear() -> None:
    _check(lib().moe_timing_device_clear())


def timing_device_reset() -> None:
    _check(lib().moe_timing_device_reset())


def timing_device_read(kind: str):
    """(summed ms, launches) of the device-timed launches of `kind` that ran
    since the last reset."""
    ms = ctypes.c_double(0)
    n = ctypes.c_int64(0)
    _check(lib().moe_timing_device_read(KERNEL_KINDS[kind], ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def calib_mfma(out: torch.Tensor, iters: int, zero_operands: bool = False, stream=None) -> float:
    """Enqueue the matrix-core reference loop (one workgroup per 512 floats
    of `out`) and return the floating-point operations it performs."""
    _need(out, torch.float32, "out", 1)
    if out.numel() == 0 or out.numel() % 512:
        raise ValueError("calib_mfma: out must hold a positive multiple of 512 floats")
    grid = out.numel() // 512
    _check(lib().moe_calib_mfma(grid, int(iters), 1 if zero_operands else 0, _ptr(out), _stream(stream)))
    return float(grid) * 8 * iters * 8 * 32768


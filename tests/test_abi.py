"""The C ABI without a GPU: the library loads, exports every symbol that
include/libmoe.h declares, sizes workspaces, and rejects bad arguments on the
host before anything is enqueued (the checks below make no HIP call, so
they run on a machine with no GPU)."""
import ctypes
import os
import re

import pytest

import paper_2606_26607_amd as moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libmoe.h")
OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: every call below fails validation


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = moe.lib()
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), f"missing export {n}"


def test_status_strings_and_version():
    L = moe.lib()
    assert L.moe_version() >= 1
    for s, name in [(0, b"MOE_OK"), (1, b"MOE_ERR_INVALID_ARG"), (2, b"MOE_ERR_UNSUPPORTED"),
                    (3, b"MOE_ERR_WORKSPACE"), (4, b"MOE_ERR_HIP")]:
        assert L.moe_status_str(s) == name


def test_workspace_sizes():
    assert moe.permute_workspace_size(4096, 2, 8) >= (4096 * 2 // 1024 + 1) * 8 * 4
    assert moe.permute_workspace_size(-1, 2, 8) == 0
    assert moe.ffn_workspace_size(8192, 8, 4096, 1792) >= 8192 * 1792 * 2
    assert moe.ffn_workspace_size(8192, 0, 4096, 1792) == 0


@pytest.mark.parametrize("T,E,k,st", [(4, 8, 0, INVALID), (4, 8, 9, INVALID), (4, 0, 1, INVALID),
                                      (-1, 8, 2, INVALID), (4, 2048, 2, UNSUPPORTED),
                                      (4, 64, 17, UNSUPPORTED), (1 << 29, 64, 8, UNSUPPORTED)])
def test_route_rejects(T, E, k, st):
    L = moe.lib()
    assert L.moe_route(FAKE, T, E, k, FAKE, FAKE, None) == st
    assert L.moe_last_error()


def test_route_null_pointers():
    assert moe.lib().moe_route(None, 4, 8, 2, FAKE, FAKE, None) == INVALID


def test_permute_rejects():
    L = moe.lib()
    big = 1 << 20
    args = dict(ids=FAKE, T=16, k=2, E=8, e0=0, El=8, counts=FAKE, offsets=FAKE, r2p=FAKE, p2r=FAKE,
                x=FAKE, H=64, xp=FAKE, ws=FAKE, wsb=big)

    def call(**kw):
        a = dict(args, **kw)
        return L.moe_permute(a["ids"], a["T"], a["k"], a["E"], a["e0"], a["El"], a["counts"],
                             a["offsets"], a["r2p"], a["p2r"], a["x"], a["H"], a["xp"], a["ws"],
                             a["wsb"], None)
    assert call(e0=4, El=8) == INVALID          # local range past E
    assert call(El=0) == INVALID
    assert call(e0=-1) == INVALID
    assert call(counts=None) == INVALID
    assert call(ids=None) == INVALID
    assert call(H=60) == UNSUPPORTED           # not a multiple of 8
    assert call(x=None) == INVALID             # x_perm without x
    assert call(ws=None) == WORKSPACE
    assert call(wsb=16) == WORKSPACE
    assert call(k=17, E=32) == UNSUPPORTED


def test_permute_noalloc_rejects():
    """The allocation-free permutation checks what moe_permute checks, and
    rejects on the host any size whose histograms exceed its static scratch."""
    L = moe.lib()
    limit = L.moe_permute_noalloc and 4 << 20

    def call(T, k, E, El, ids=FAKE, counts=FAKE):
        return L.moe_permute_noalloc(ids, T, k, E, 0, El, counts, FAKE, FAKE, FAKE, None, 0, None, None)
    assert moe.permute_workspace_size(1 << 20, 16, 1024) > limit
    assert call(1 << 20, 16, 1024, 1024) == UNSUPPORTED
    assert b"scratch" in L.moe_last_error()
    assert call(16, 2, 8, 0) == INVALID
    assert call(16, 2, 8, 8, counts=None) == INVALID
    assert call(16, 2, 8, 8, ids=None) == INVALID
    assert call(16, 17, 32, 8) == UNSUPPORTED
    # the largest accepted inputs of either chunk size stay within the scratch
    assert moe.permute_workspace_size(1 << 18, 8, 8) <= limit          # 2^24 pair-experts: 256-pair chunks
    assert moe.permute_workspace_size(1 << 18, 8, 256) <= limit         # 1024-pair chunks


def test_layer_forward_rejects():
    """moe_layer_forward checks what the four calls check, on the host."""
    L = moe.lib()
    big = 1 << 30
    args = dict(x=FAKE, lg=FAKE, T=16, E=8, k=2, e0=0, El=8, H=256, Is=256, w13=FAKE, w2=FAKE, sb=0, sc=0,
                sw13=None, sw2=None, ids=FAKE, w=FAKE, counts=FAKE, offsets=FAKE, r2p=FAKE, p2r=FAKE, y=FAKE,
                sy=None, out=FAKE, ws=ctypes.c_void_p(0x100000), wsb=big)

    def call(**kw):
        a = dict(args, **kw)
        return L.moe_layer_forward(a["x"], a["lg"], a["T"], a["E"], a["k"], a["e0"], a["El"], a["H"], a["Is"],
                                   a["w13"], a["w2"], a["sb"], a["sc"], a["sw13"], a["sw2"], a["ids"], a["w"],
                                   a["counts"], a["offsets"], a["r2p"], a["p2r"], a["y"], a["sy"], a["out"], a["ws"],
                                   a["wsb"], None)
    assert call(k=0) == INVALID
    assert call(k=17, E=32) == UNSUPPORTED
    assert call(e0=4) == INVALID                  # local experts past E
    assert call(H=60) == UNSUPPORTED              # not a multiple of 8
    assert call(offsets=None) == INVALID
    assert call(counts=None) == INVALID
    assert call(lg=None) == INVALID
    assert call(out=None) == INVALID
    assert call(sb=10, sc=8) == INVALID           # shared rows past T
    assert call(sc=4) == INVALID                  # shared rows without shared weights
    assert call(sc=4, sw13=FAKE, sw2=FAKE, sy=FAKE, H=136) == UNSUPPORTED   # shared expert needs H % 64 == 0
    assert call(wsb=16) == WORKSPACE
    assert call(ws=None) == WORKSPACE
    assert moe.layer_workspace_size(16, 2, 8, 256, 256) >= (moe.permute_workspace_size(16, 2, 8) +
                                                            moe.ffn_workspace_size(32, 8, 256, 256))


def test_ffn_rejects():
    L = moe.lib()
    big = 1 << 30

    def call(xp=FAKE, xr=64, r2p=None, k=1, off=FAKE, El=8, cap=64, H=64, Is=32, w13=FAKE, w2=FAKE, y=FAKE,
             ws=FAKE, wsb=big):
        return L.moe_grouped_ffn(xp, xr, r2p, k, off, El, cap, H, Is, w13, w2, y, ws, wsb, None)
    assert call(El=0) == INVALID
    assert call(El=1025) == UNSUPPORTED
    assert call(H=12) == UNSUPPORTED
    assert call(Is=0) == INVALID
    assert call(cap=-1) == INVALID
    assert call(off=None) == INVALID
    assert call(w2=None) == INVALID
    assert call(wsb=100) == WORKSPACE
    assert call(ws=ctypes.c_void_p(0x100010)) == WORKSPACE   # not 256-byte aligned
    assert call(xp=ctypes.c_void_p(0x100002)) == INVALID     # not 16-byte aligned
    assert call(xr=32) == INVALID                            # permuted x shorter than cap_rows
    assert call(xr=-1) == INVALID
    assert call(r2p=FAKE, k=0) == INVALID                    # gather without a slot count


def test_ffn_shared_rejects():
    L = moe.lib()
    big = 1 << 30

    def call(xr=64, r2p=FAKE, El=8, cap=64, H=256, Is=128, sb=0, sc=16, sw13=FAKE, sw2=FAKE, sy=FAKE, wsb=big):
        return L.moe_grouped_ffn_shared(FAKE, xr, r2p, 2, FAKE, El, cap, H, Is, FAKE, FAKE, FAKE, sb, sc, sw13,
                                        sw2, sy, FAKE, wsb, None)
    assert call(r2p=None) == INVALID                          # the shared variant gathers rows
    assert call(sb=60, sc=16) == INVALID                      # shared rows beyond x
    assert call(sb=-1) == INVALID
    assert call(sc=-1) == INVALID
    assert call(sw2=None) == INVALID
    assert call(sy=ctypes.c_void_p(0x100004)) == INVALID      # not 16-byte aligned
    assert call(H=200) == UNSUPPORTED                         # shared path needs 64-multiples
    assert call(Is=64) == UNSUPPORTED                         # ... and K of at least 128
    assert call(El=1024) == UNSUPPORTED                       # one more expert than allowed
    assert call(El=0) == INVALID
    assert call(wsb=100) == WORKSPACE
    # the workspace must hold the shared rows and the extra expert
    need = L.moe_ffn_workspace_size(64 + 16, 9, 256, 128)
    assert need > L.moe_ffn_workspace_size(64, 8, 256, 128)
    assert call(wsb=need - 1) == WORKSPACE


def test_reshard_rejects():
    L = moe.lib()
    arr = ctypes.c_void_p * 4
    srcs = arr(FAKE, FAKE, FAKE, FAKE)

    def call(d=0, P=4, r=0, E=16, H=64, I=256, s13=srcs, s2=srcs, d13=FAKE, d2=FAKE):
        return L.moe_reshard_experts(d, P, r, E, H, I, s13, s2, d13, d2, None)
    assert call(d=2) == INVALID
    assert call(P=0) == INVALID
    assert call(P=17) == UNSUPPORTED
    assert call(r=4) == INVALID
    assert call(E=10) == INVALID                       # not a multiple of P
    assert call(I=102) == INVALID                      # not a multiple of P
    assert call(I=100) == UNSUPPORTED                  # I/P = 25, not a multiple of 8
    assert call(H=12) == UNSUPPORTED
    assert call(s13=None) == INVALID
    assert call(d2=None) == INVALID
    assert call(d13=ctypes.c_void_p(0x100002)) == INVALID
    half = arr(FAKE, None, FAKE, FAKE)
    assert call(s2=half) == INVALID                    # a source with only one of its two tensors


def test_kv_rejects():
    L = moe.lib()

    def move(ns=64, sh=8, nd=64, dh=4, D=128, s0=0, d0=0, n=2, sv=None, dv=None, ntok=5, sk=FAKE, dk=FAKE,
             nsrc=1, first=None):
        vp = ctypes.c_void_p * 2
        k = vp(sk, FAKE)
        v = None if sv is None else vp(sv, FAKE)
        slots = (ctypes.c_int64 * 2)(ns, ns)
        f = (ctypes.c_int64 * 3)(*(first or (0, ntok, ntok)))
        return L.moe_kv_move(nsrc, k, v, slots, f, sh, dk, dv, nd, dh, D, s0, d0, n, FAKE, FAKE, None)
    assert move(D=12) == UNSUPPORTED
    assert move(D=0) == INVALID
    assert move(s0=7) == INVALID                       # source heads past the pool
    assert move(d0=3) == INVALID
    assert move(n=0) == INVALID
    assert move(sv=FAKE) == INVALID                    # V given on one side only
    assert move(ntok=-1) == INVALID                    # token offsets decrease
    assert move(first=(1, 5, 5)) == INVALID            # offsets start at 0
    assert move(sk=None) == INVALID
    assert move(sk=ctypes.c_void_p(0x100004)) == INVALID
    assert move(dk=ctypes.c_void_p(0x100008)) == INVALID
    assert move(ns=-1) == INVALID
    assert move(nsrc=0) == INVALID
    assert move(nsrc=17) == UNSUPPORTED
    assert move(nsrc=2, first=(0, 3, 2)) == INVALID
    assert move(ntok=0) == OK                          # nothing to do, nothing launched
    assert move(sk=None, ntok=0) == OK                 # an empty source may be null
    assert L.moe_kv_slots(FAKE, 4, FAKE, 2, 0, FAKE, 8, None) == INVALID      # page_size 0
    assert L.moe_kv_slots(FAKE, 4, FAKE, -1, 16, FAKE, 8, None) == INVALID
    assert L.moe_kv_slots(None, 4, FAKE, 2, 16, FAKE, 8, None) == INVALID
    assert L.moe_kv_slots(FAKE, 4, FAKE, 0, 16, FAKE, 8, None) == OK          # no requests


def test_combine_rejects():
    L = moe.lib()

    def call(y=FAKE, yr=8, p2r=FAKE, w=FAKE, T=4, k=2, H=64, sy=None, sb=0, sc=0, acc=0, out=FAKE):
        return L.moe_combine(y, yr, p2r, w, T, k, H, sy, sb, sc, acc, out, None)
    assert call(k=0) == INVALID
    assert call(k=17) == UNSUPPORTED
    assert call(H=63) == UNSUPPORTED
    assert call(out=None) == INVALID
    assert call(y=None) == INVALID
    assert call(sy=FAKE, sb=3, sc=2) == INVALID   # shared rows past T
    assert call(T=-1) == INVALID


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2606_26607_amd import binding
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        binding.lib()


@pytest.mark.parametrize("grid,iters", [(0, 1), (65537, 1), (1, 0), (1, 1 << 25)])
def test_calib_mfma_rejects(grid, iters):
    L = moe.lib()
    assert L.moe_calib_mfma(grid, iters, 0, FAKE, None) == INVALID
    assert L.moe_calib_mfma(1, 1, 0, None, None) == INVALID

"""ctypes wrapper around the CPU oracle (moe_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg; never by the product path.  Arrays are numpy.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(src: str = _SRC, out: str = LIB_PATH, extra=()) -> str:
    """Compile the oracle with gcc (plain -O2: no fast-math, so floating-point
    evaluation order is the source order)."""
    tmp = f"{out}.{os.getpid()}.tmp"  # concurrent builders (test workers) each rename a whole file
    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", *extra, src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def load(path: str = LIB_PATH):
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        build(out=path)
    lib = ctypes.CDLL(path)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    lib.oracle_route.argtypes = [vp, i64, i32, i32, vp, vp]
    lib.oracle_permute.argtypes = [vp, i64, i32, i32, i32, vp, vp, vp, vp]
    lib.oracle_grouped_ffn.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp]
    lib.oracle_combine.argtypes = [vp, vp, vp, i64, i32, i32, vp, i64, i64, i32, vp, vp]
    lib.oracle_layer_tokens.argtypes = [vp, i32, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp,
                                        i32, i64, i64, vp, i64, vp]
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [i32]
    if path == LIB_PATH:
        _lib = lib
    return lib


class Oracle:
    """Typed entry points over one loaded oracle library."""

    def __init__(self, path: str = LIB_PATH):
        self.lib = load(path)

    @staticmethod
    def _c(a, dtype):
        a = np.ascontiguousarray(a, dtype=dtype)
        return a, a.ctypes.data

    def threads(self) -> int:
        return self.lib.oracle_threads()

    def set_threads(self, n: int) -> None:
        self.lib.oracle_set_threads(n)

    def route(self, logits: np.ndarray, k: int):
        logits, lp = self._c(logits, np.float32)
        T, E = logits.shape
        ids = np.empty((T, k), np.int32)
        w = np.empty((T, k), np.float64)
        self.lib.oracle_route(lp, T, E, k, ids.ctypes.data, w.ctypes.data)
        return ids, w

    def permute(self, ids: np.ndarray, e0: int, El: int):
        ids, ip = self._c(ids, np.int32)
        T, k = ids.shape
        counts = np.empty(El, np.int32)
        offsets = np.empty(El + 1, np.int32)
        r2p = np.full(max(T * k, 1), -7, np.int32)
        p2r = np.empty(max(T * k, 1), np.int32)
        self.lib.oracle_permute(ip, T, k, e0, El, counts.ctypes.data, offsets.ctypes.data,
                                r2p.ctypes.data, p2r.ctypes.data)
        n = int(offsets[El])
        return counts, offsets, r2p[:n].copy(), p2r[:T * k].copy()

    def grouped_ffn(self, x_perm, offsets, w13, w2):
        x_perm, xp = self._c(x_perm, np.uint16)
        offsets, op = self._c(offsets, np.int32)
        w13, ap = self._c(w13, np.uint16)
        w2, bp = self._c(w2, np.uint16)
        El = offsets.shape[0] - 1
        H = x_perm.shape[1]
        Is = w2.shape[2]
        n = int(offsets[El])
        y = np.zeros((max(n, 1), H), np.float64)
        self.lib.oracle_grouped_ffn(xp, op, El, H, Is, ap, bp, y.ctypes.data)
        return y[:n]

    def combine(self, y, pair_to_row, w, T, k, shared_y=None, sb=0, sc=0, accumulate=0, prior=None):
        y, yp = self._c(y, np.uint16)
        pair_to_row, pp = self._c(pair_to_row, np.int32)
        w, wp = self._c(w, np.float32)
        H = y.shape[1]
        syp = 0
        if shared_y is not None:
            shared_y, syp = self._c(shared_y, np.uint16)
        prp = 0
        if accumulate:
            prior, prp = self._c(prior, np.uint16)
        out = np.empty((T, H), np.float64)
        self.lib.oracle_combine(yp, pp, wp, T, k, H, syp or None, sb, sc, accumulate, prp or None,
                                out.ctypes.data)
        return out

    def layer_tokens(self, x, ids, w, e0, El, w13, w2, tokens, sw13=None, sw2=None, sb=0, sc=0):
        x, xp = self._c(x, np.uint16)
        ids, ip = self._c(ids, np.int32)
        w, wp = self._c(w, np.float64)
        w13, ap = self._c(w13, np.uint16)
        w2, bp = self._c(w2, np.uint16)
        tokens, tp = self._c(tokens, np.int64)
        H = x.shape[1]
        k = ids.shape[1]
        Is = w2.shape[2] if w2.ndim == 3 and w2.shape[0] else 0
        s13p = s2p = 0
        Is_sh = 0
        if sc > 0:
            sw13, s13p = self._c(sw13, np.uint16)
            sw2, s2p = self._c(sw2, np.uint16)
            Is_sh = sw2.shape[-1]
        out = np.empty((max(len(tokens), 1), H), np.float64)
        self.lib.oracle_layer_tokens(xp, H, ip, wp, k, e0, El, Is, ap, bp, s13p or None, s2p or None,
                                     Is_sh, sb, sc, tp, len(tokens), out.ctypes.data)
        return out[:len(tokens)]

    def layer(self, inp, tokens=None):
        """Full layer on the config's inputs (all tokens unless listed)."""
        cfg = inp.cfg
        ids, w = self.route(inp.logits, cfg.k)
        if tokens is None:
            tokens = np.arange(cfg.T, dtype=np.int64)
        return self.layer_tokens(inp.x, ids, w, cfg.e0, cfg.E_l, inp.w13, inp.w2, tokens,
                                 inp.sw13, inp.sw2, cfg.shared_begin, cfg.shared_count)

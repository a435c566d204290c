"""Brute-force references that pin the CPU oracle.

They compute the same quantities from their definitions by a different
route: library sorts and softmax, and a dense evaluation of *every* expert on
*every* token followed by a top-k mask.  None of this code is shared with the
oracle or with the HIP library.
"""
import numpy as np
from scipy.special import softmax


def bf16(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def topk_lexsort(logits, k):
    """Order each row by (logit desc, id asc) with numpy's lexsort; -0.0 is
    mapped to +0.0 first so that both compare equal as keys."""
    l = np.asarray(logits, np.float64) + 0.0  # -0.0 + 0.0 == +0.0
    T, E = l.shape
    ids = np.empty((T, k), np.int32)
    for t in range(T):
        order = np.lexsort((np.arange(E), -l[t]))
        ids[t] = order[:k]
    return ids


def route_weights(logits, ids):
    p = softmax(np.asarray(logits, np.float64), axis=1)
    sel = np.take_along_axis(p, ids.astype(np.int64), axis=1)
    return sel / sel.sum(axis=1, keepdims=True)


def permute_argsort(ids, e0, El):
    """Permutation by a stable library argsort of the flattened expert ids."""
    flat = ids.reshape(-1).astype(np.int64)
    local = (flat >= e0) & (flat < e0 + El)
    key = np.where(local, flat - e0, El)          # non-local pairs sort last
    order = np.argsort(key, kind="stable")
    n = int(local.sum())
    row_to_pair = order[:n].astype(np.int32)
    pair_to_row = np.full(flat.shape[0], -1, np.int32)
    pair_to_row[row_to_pair] = np.arange(n, dtype=np.int32)
    counts = np.bincount(key[local], minlength=El).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    return counts, offsets, row_to_pair, pair_to_row


def dense_layer(x, logits, k, w13, w2, e0, El):
    """Every local expert evaluated on every token (fp64 matmuls), then
    masked by the top-k selection and weighted by the renormalised softmax."""
    xf = bf16(x)
    T = xf.shape[0]
    Is = w2.shape[2]
    ids = topk_lexsort(logits, k)
    wts = route_weights(logits, ids)
    gate = np.zeros((T, El))
    for j in range(k):
        e = ids[:, j]
        loc = (e >= e0) & (e < e0 + El)
        gate[np.nonzero(loc)[0], e[loc] - e0] = wts[loc, j]
    out = np.zeros((T, xf.shape[1]))
    for le in range(El):
        W13 = bf16(w13[le])
        g = xf @ W13[:Is].T
        u = xf @ W13[Is:].T
        a = g / (1.0 + np.exp(-g)) * u
        out += gate[:, le:le + 1] * (a @ bf16(w2[le]).T)
    return out


def swiglu_mlp(x, w13, w2):
    """A dense SwiGLU MLP on every row of x (fp64 matmuls): w13 [2I, H] holds
    the gate rows, then the up rows; w2 [H, I]."""
    xf = bf16(x)
    W = bf16(w13)
    I = W.shape[0] // 2
    g, u = xf @ W[:I].T, xf @ W[I:].T
    return (g / (1.0 + np.exp(-g)) * u) @ bf16(w2).T

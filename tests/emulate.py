"""Numpy emulation of Algorithms 1-3 over the tensors that hb_compile built.

This is test code: it validates the host-side compile step (the tables a
kernel reads) without a GPU, by running the paper's algorithms on the
exported tables and comparing with the oracle. It is neither the oracle nor
the product path.
"""
from __future__ import annotations

import numpy as np


def _f32(bits):
    return np.asarray(bits, np.uint32).view(np.float32)


def _aggregate(model, values):
    """values: [n, T, leaf_dim] float32 leaf values -> [n, K] float64 margins."""
    n, T, ld = values.shape
    K = model["n_outputs"]
    v = values.astype(np.float64)
    if ld == 1:
        cls = model.get("tree_class")
        cls = np.zeros(T, np.int64) if cls is None else np.asarray(cls, np.int64)
        raw = np.zeros((n, K))
        for k in range(K):
            raw[:, k] = v[:, cls == k, 0].sum(axis=1)
    else:
        raw = v.sum(axis=1)
    if model["aggregation"] == "mean":
        raw /= T
    if model.get("base_score") is not None:
        raw += np.asarray(model["base_score"], np.float64)
    return raw


def _tile(h, X, strategy):
    """The feature tile the kernels stage: the input columns some decision node
    tests, in the order the compiled tables index them; a column flagged for
    nodes that send missing values left reads NaN as -inf; a categorical
    column is 0 where the row goes left (its category, the integer part of a
    non-negative value inside the bit set, is in the set; NaN where the
    column's nodes send missing values left) and 1 elsewhere."""
    table = h.table(strategy, "features", np.int32).astype(np.int64)
    n_cols = h.info()["n_used_features"]
    cols = table[:n_cols]
    mask = (1 << 29) - 1
    cat = (cols >> 29) & 1 == 1
    nan_left = (cols >> 30) & 1 == 1
    tile = np.empty((X.shape[0], n_cols), np.float32)
    for j in range(n_cols):
        if not cat[j]:
            v = X[:, cols[j] & mask].copy()
            if nan_left[j]:
                v[np.isnan(v)] = -np.inf
            tile[:, j] = v
            continue
        at = int(cols[j] & mask)
        col, W = int(table[at]), int(table[at + 1])
        words = table[at + 2:at + 2 + W].astype(np.uint32)
        x = X[:, col].astype(np.float64)
        left = np.zeros(X.shape[0], bool)
        ok = (x >= 0) & (x < 32 * W)
        k = np.where(ok, x, 0).astype(np.int64)
        if W:
            left[ok] = (words[k[ok] // 32] >> (k[ok] % 32).astype(np.uint32)) & 1 == 1
        left[np.isnan(x)] = bool(nan_left[j])
        tile[:, j] = np.where(left, 0.0, 1.0)
    return tile


def ptt(h, model, X):
    """Algorithm 3 (PerfectTreeTraversal) on the compiled heap tables."""
    X = _tile(h, X, "ptt")
    info = h.info()
    T, D, ld = info["n_trees"], info["ptt_depth"], info["leaf_dim"]
    S = 1 << D
    node = h.table("ptt", "node", np.uint32).reshape(T, max(S, 2), 2)
    lv = h.table("ptt", "leaf_value", np.float32).reshape(T, S, ld)
    lid = h.table("ptt", "leaf_id", np.int32).reshape(T, S)
    n = X.shape[0]
    tix = np.arange(T)[None, :]
    idx = np.ones((n, T), np.int64)
    for _ in range(D):
        rec = node[tix, idx]                      # [n, T, 2]
        x = X[np.arange(n)[:, None], rec[..., 1].astype(np.int64)]
        idx = 2 * idx + np.where(x < _f32(rec[..., 0]), 0, 1)
    slot = idx - S
    return lid[tix, slot], _aggregate(model, lv[tix, slot])


def tt(h, model, X):
    """Algorithm 2 (TreeTraversal) on the compiled child tables."""
    X = _tile(h, X, "tt")
    info = h.info()
    T, ld = info["n_trees"], info["leaf_dim"]
    n_pad = int(h.table("tt", "dims", np.int32)[0])
    node = h.table("tt", "node", np.uint32).reshape(T, n_pad, 2)
    depth = h.table("tt", "depth", np.int32)
    lv = h.table("tt", "leaf_value", np.float32).reshape(T, n_pad, ld)
    lid = h.table("tt", "leaf_id", np.int32).reshape(T, n_pad)
    n = X.shape[0]
    tix = np.arange(T)[None, :]
    idx = np.zeros((n, T), np.int64)
    for _ in range(int(depth.max(initial=0))):
        rec = node[tix, idx]
        feat = (rec[..., 1] & 0xFFFF).astype(np.int64)
        right = (rec[..., 1] >> 16).astype(np.int64)
        x = X[np.arange(n)[:, None], feat]
        idx = right - (x < _f32(rec[..., 0])).astype(np.int64)
    return lid[tix, idx], _aggregate(model, lv[tix, idx])


def gemm(h, model, X, check_unique=True):
    """Algorithm 1 (GEMM) on the compiled A/B (node), C^T, D (bias) and E tables."""
    X = _tile(h, X, "gemm")
    info = h.info()
    T, ld = info["n_trees"], info["leaf_dim"]
    k_pad, l_pad, S = (int(v) for v in h.table("gemm", "dims", np.int32))
    node = h.table("gemm", "node", np.uint32).reshape(T, k_pad, 2)
    shape = h.table("gemm", "shape", np.int32)
    ct = h.table("gemm", "ct", np.int8).reshape(S, l_pad, k_pad).astype(np.int64)
    bias = h.table("gemm", "bias", np.int32).reshape(S, l_pad).astype(np.int64)
    lv = h.table("gemm", "leaf_value", np.float32).reshape(T, l_pad, ld)
    lid = h.table("gemm", "leaf_id", np.int32).reshape(T, l_pad)
    n = X.shape[0]
    cols = np.empty((n, T), np.int64)
    for t in range(T):
        feat = node[t, :, 1].astype(np.int64)
        P = np.where(X[:, feat] < _f32(node[t, :, 0])[None, :], 64, 0)   # T <- X.A < B
        acc = bias[shape[t]][None, :] + P @ ct[shape[t]].T               # 256 (T.C - D) + l
        c = acc.argmax(axis=1)
        if check_unique:
            assert np.all((acc >= 0).sum(axis=1) == 1), f"tree {t}: not exactly one leaf column"
            assert np.all(acc[np.arange(n), c] == c)
        cols[:, t] = c
    tix = np.arange(T)[None, :]
    return lid[tix, cols], _aggregate(model, lv[tix, cols])

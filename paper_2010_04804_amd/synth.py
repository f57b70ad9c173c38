"""Seeded synthetic ensembles and inputs.

This module only draws random numbers and lays them out as plain node arrays;
it holds none of the scoring arithmetic, so both the product library and the
test oracle can be fed from it.

A model is a dict of numpy arrays in "caller" form, one entry per tree node:

    n_trees, n_features, n_outputs, leaf_dim       ints
    tree_node_offset  int64 [n_trees + 1]  tree t owns nodes [off[t], off[t+1])
    feature           int32 [nodes]  feature tested by an internal node, -1 at a leaf
    threshold         float32 [nodes]  rule: x[feature] < threshold goes left
    left, right       int32 [nodes]  tree-local child ids, -1 at a leaf
    leaf_value        float32 [nodes * leaf_dim]  read only at leaves
    tree_class        int32 [n_trees] or None  output column of a scalar-leaf tree
    aggregation       "sum" | "mean"
    transform         "none" | "sigmoid" | "softmax"
    base_score        float32 [n_outputs] or None

Every draw is made in float64 and rounded once to float32. Each config uses
``SeedSequence(seed).spawn(2)`` as [model stream, data stream], so the rows of
a smaller batch are a prefix of a larger batch of the same config.

The five workloads stand in for the paper's evaluation models (Sec. 6.1.1:
500 trees of maximum depth 8 trained on Fraud, Epsilon, Year, Covtype, Higgs
and Airline), whose datasets and trained models are not available here; they
copy the shapes only (feature counts, tree counts and depths, class counts).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "CONFIGS",
    "perfect_forest",
    "leafwise_forest",
    "make_model",
    "make_rows",
    "make_config",
    "permute_nodes",
    "model_stats",
    "SWEEP",
    "sweep_model",
    "sweep_rows",
    "RF_VECTOR",
    "rf_vector_model",
    "rf_vector_rows",
    "narrow_use_model",
    "narrow_use_rows",
    "with_missing",
]


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    m, d = ss.spawn(2)
    return np.random.Generator(np.random.PCG64(m)), np.random.Generator(np.random.PCG64(d))


def _f32(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64).astype(np.float32)


def perfect_forest(rng, n_trees, depth, n_features, draw_threshold, draw_leaves, leaf_dim=1):
    """Perfect binary trees of ``depth`` levels of decisions, numbered in
    breadth-first order (node i has children 2i+1, 2i+2).

    ``draw_threshold(rng, features)`` returns one threshold per internal node
    given the feature it tests; ``draw_leaves(rng, n)`` returns ``n`` leaf
    values (``[n, leaf_dim]`` when ``leaf_dim > 1``).
    """
    n_int = (1 << depth) - 1
    n_nodes = 2 * n_int + 1
    feature = np.full((n_trees, n_nodes), -1, np.int32)
    threshold = np.zeros((n_trees, n_nodes), np.float32)
    left = np.full((n_trees, n_nodes), -1, np.int32)
    right = np.full((n_trees, n_nodes), -1, np.int32)
    value = np.zeros((n_trees, n_nodes, leaf_dim), np.float32)
    ids = np.arange(n_int, dtype=np.int32)
    for t in range(n_trees):
        f = rng.integers(0, n_features, size=n_int).astype(np.int32)
        feature[t, :n_int] = f
        threshold[t, :n_int] = _f32(draw_threshold(rng, f))
        left[t, :n_int] = 2 * ids + 1
        right[t, :n_int] = 2 * ids + 2
        v = np.asarray(draw_leaves(rng, n_int + 1), np.float64).reshape(n_int + 1, leaf_dim)
        value[t, n_int:, :] = _f32(v)
    return {
        "n_trees": n_trees,
        "n_features": n_features,
        "leaf_dim": leaf_dim,
        "tree_node_offset": np.arange(n_trees + 1, dtype=np.int64) * n_nodes,
        "feature": feature.reshape(-1),
        "threshold": threshold.reshape(-1),
        "left": left.reshape(-1),
        "right": right.reshape(-1),
        "leaf_value": value.reshape(-1),
    }


def leafwise_forest(rng, n_trees, n_leaves, max_depth, p_deepen, n_features,
                    draw_threshold, draw_leaves):
    """Unbalanced trees grown one split at a time until ``n_leaves`` leaves.

    Reading of "random split side chosen with p=0.7 to deepen": after a split,
    with probability ``p_deepen`` the next split is on one of the two new
    children (chosen uniformly) if its depth is below ``max_depth``; otherwise
    the next split is on a leaf drawn uniformly from all leaves of depth below
    ``max_depth``. Children are appended as (left, right), so node ids follow
    creation order and the root is node 0.
    """
    offs = [0]
    feats, thrs, lefts, rights, vals = [], [], [], [], []
    for _ in range(n_trees):
        depth = [0]
        feat = [-1]
        left = [-1]
        right = [-1]
        leaves = [0]
        target = 0
        while len(leaves) < n_leaves:
            c1, c2 = len(depth), len(depth) + 1
            d = depth[target] + 1
            depth += [d, d]
            feat += [-1, -1]
            left += [-1, -1]
            right += [-1, -1]
            feat[target] = int(rng.integers(0, n_features))
            left[target], right[target] = c1, c2
            leaves.remove(target)
            leaves += [c1, c2]
            if len(leaves) >= n_leaves:
                break
            if rng.random() < p_deepen:
                cand = c1 if rng.random() < 0.5 else c2
                if depth[cand] < max_depth:
                    target = cand
                    continue
            eligible = [l for l in leaves if depth[l] < max_depth]
            target = eligible[int(rng.integers(0, len(eligible)))]
        n = len(depth)
        feat_a = np.asarray(feat, np.int32)
        internal = feat_a >= 0
        thr = np.zeros(n, np.float32)
        thr[internal] = _f32(draw_threshold(rng, feat_a[internal]))
        val = np.zeros(n, np.float32)
        val[~internal] = _f32(draw_leaves(rng, int((~internal).sum())))
        feats.append(feat_a)
        thrs.append(thr)
        lefts.append(np.asarray(left, np.int32))
        rights.append(np.asarray(right, np.int32))
        vals.append(val)
        offs.append(offs[-1] + n)
    return {
        "n_trees": n_trees,
        "n_features": n_features,
        "leaf_dim": 1,
        "tree_node_offset": np.asarray(offs, np.int64),
        "feature": np.concatenate(feats),
        "threshold": np.concatenate(thrs),
        "left": np.concatenate(lefts),
        "right": np.concatenate(rights),
        "leaf_value": np.concatenate(vals),
    }


# ---------------------------------------------------------------------------
# The five workloads. Each entry gives the recipe; make_config builds it.

CONFIGS = {
    1: dict(name="tiny GBDT regressor: 10 perfect trees depth 3, 8 features",
            seed=0, n_rows=1_000),
    2: dict(name="GBDT binary classifier: 500 perfect trees depth 8, 28 features",
            seed=2, n_rows=1_000_000, n_rows_small=10_000),
    3: dict(name="random forest, wide input: 500 perfect trees depth 8, 2000 features, 2 classes",
            seed=3, n_rows=100_000),
    4: dict(name="multiclass GBDT: 7 classes x 500 trees depth 8, 54 features",
            seed=4, n_rows=1_000_000),
    5: dict(name="unbalanced GBDT: 500 leaf-wise trees, 256 leaves, depth <= 12, 100 features",
            seed=5, n_rows=1_000_000),
}

_CFG4_CONT = 10  # config 4: columns 0..9 continuous, 10..53 binary


def make_model(cfg: int) -> dict:
    """The seeded ensemble of workload ``cfg`` (1..5)."""
    rng, _ = _streams(CONFIGS[cfg]["seed"])
    if cfg == 1:
        m = perfect_forest(rng, 10, 3, 8,
                           lambda r, f: r.random(f.size),
                           lambda r, n: r.normal(0.0, 0.1, n))
        m.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
    elif cfg == 2:
        m = perfect_forest(rng, 500, 8, 28,
                           lambda r, f: r.standard_normal(f.size),
                           lambda r, n: r.normal(0.0, 0.05, n))
        m.update(n_outputs=1, tree_class=None, aggregation="sum", transform="sigmoid", base_score=None)
    elif cfg == 3:
        def leaves(r, n):
            p = r.random(n)
            return np.stack([1.0 - p, p], axis=1)
        m = perfect_forest(rng, 500, 8, 2000,
                           lambda r, f: r.uniform(-1.0, 1.0, f.size),
                           leaves, leaf_dim=2)
        m.update(n_outputs=2, tree_class=None, aggregation="mean", transform="none", base_score=None)
    elif cfg == 4:
        def thr(r, f):
            cont = r.standard_normal(f.size)
            return np.where(f < _CFG4_CONT, cont, 0.5)
        m = perfect_forest(rng, 3500, 8, 54, thr, lambda r, n: r.normal(0.0, 0.05, n))
        m.update(n_outputs=7, tree_class=(np.arange(3500) % 7).astype(np.int32),
                 aggregation="sum", transform="softmax", base_score=None)
    elif cfg == 5:
        m = leafwise_forest(rng, 500, 256, 12, 0.7, 100,
                            lambda r, f: r.random(f.size),
                            lambda r, n: r.normal(0.0, 0.02, n))
        m.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
    else:
        raise ValueError(f"unknown config {cfg}")
    return m


# Strategy-crossover sweep (the trees-implementation experiment of Sec. 6):
# 100 trees over 200 features at depth 3, 7 and 12, scored at batch sizes
# from 1 to 1M. Depth 12 comes both perfect (4096 leaves, no GEMM) and
# leaf-wise with 256 leaves (the unbalanced shape GEMM can still hold).
SWEEP = dict(
    models=("perfect-d3", "perfect-d7", "perfect-d12", "leafwise-d12",
            "perfect-d3-n28", "perfect-d11-n28", "perfect-d12-n28", "leafwise-d12-n28"),
    batches=(1, 10, 100, 1_000, 10_000, 100_000, 1_000_000),
    n_trees=100, n_features=200, seed=6,
)


def sweep_features(kind: str) -> int:
    """Input columns of a sweep model: 200, or 28 for the ``-n28`` models."""
    return 28 if kind.endswith("-n28") else SWEEP["n_features"]


def sweep_model(kind: str) -> dict:
    """One model of the crossover sweep: ``perfect-d{3,7,11,12}`` or
    ``leafwise-d12`` over 200 features, or with ``-n28`` over 28 (narrow
    rows: the row-parallel kernels' tile holds them); thresholds N(0,1),
    leaves N(0, 0.05), SUM -> sigmoid."""
    rng, _ = _streams(SWEEP["seed"] + SWEEP["models"].index(kind))
    T, F = SWEEP["n_trees"], sweep_features(kind)
    base = kind[:-len("-n28")] if kind.endswith("-n28") else kind
    thr = lambda r, f: r.standard_normal(f.size)
    leaves = lambda r, n: r.normal(0.0, 0.05, n)
    if base.startswith("perfect-d"):
        m = perfect_forest(rng, T, int(base[len("perfect-d"):]), F, thr, leaves)
    elif base == "leafwise-d12":
        m = leafwise_forest(rng, T, 256, 12, 0.7, F, thr, leaves)
    else:
        raise ValueError(f"unknown sweep model {kind}")
    m.update(n_outputs=1, tree_class=None, aggregation="sum", transform="sigmoid", base_score=None)
    return m


def sweep_rows(n_rows: int, n_features: int = SWEEP["n_features"]) -> np.ndarray:
    """Input rows of the crossover sweep: N(0,1) over 200 (or 28) features."""
    _, rng = _streams(SWEEP["seed"])
    return np.ascontiguousarray(_f32(rng.standard_normal((n_rows, n_features))))


# A binary random-forest classifier over narrow rows (the shape of the
# paper's RandomForest models on 28-feature data): 500 perfect trees of
# depth 8, leaves holding class probabilities (1 - p, p), MEAN aggregation.
RF_VECTOR = dict(name="random forest, narrow input: 500 perfect trees depth 8, 28 features, 2-vector leaves",
                 n_trees=500, depth=8, n_features=28, seed=7, n_rows=1_000_000)


def rf_vector_model() -> dict:
    rng, _ = _streams(RF_VECTOR["seed"])

    def leaves(r, n):
        p = r.random(n)
        return np.stack([1.0 - p, p], axis=1)

    m = perfect_forest(rng, RF_VECTOR["n_trees"], RF_VECTOR["depth"], RF_VECTOR["n_features"],
                       lambda r, f: r.standard_normal(f.size), leaves, leaf_dim=2)
    m.update(n_outputs=2, tree_class=None, aggregation="mean", transform="none", base_score=None)
    return m


def rf_vector_rows(n_rows: int) -> np.ndarray:
    """Input rows of the narrow random forest: N(0,1) over 28 features."""
    _, rng = _streams(RF_VECTOR["seed"])
    return np.ascontiguousarray(_f32(rng.standard_normal((n_rows, RF_VECTOR["n_features"]))))


def narrow_use_model(n_features: int, n_used: int, n_trees: int, depth: int, seed: int,
                     leaf_dim: int = 1) -> dict:
    """Perfect trees over a wide input whose decision nodes test only
    ``n_used`` of its ``n_features`` columns (a seeded random subset), the
    case feature pruning serves. Thresholds N(0,1); scalar leaves N(0, 0.05)
    summed, or (leaf_dim 2) probability pairs averaged."""
    rng, _ = _streams(seed)
    cols = np.sort(rng.choice(n_features, size=n_used, replace=False)).astype(np.int32)
    if leaf_dim == 1:
        leaves = lambda r, n: r.normal(0.0, 0.05, n)
    else:
        def leaves(r, n):
            p = r.random(n)
            return np.stack([1.0 - p, p], axis=1)
    m = perfect_forest(rng, n_trees, depth, n_used, lambda r, f: r.standard_normal(f.size), leaves,
                       leaf_dim=leaf_dim)
    f = m["feature"]
    m["feature"] = np.where(f >= 0, cols[np.maximum(f, 0)], -1).astype(np.int32)
    m["n_features"] = n_features
    if leaf_dim == 1:
        m.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
    else:
        m.update(n_outputs=leaf_dim, tree_class=None, aggregation="mean", transform="none", base_score=None)
    return m


def narrow_use_rows(n_features: int, n_rows: int, seed: int) -> np.ndarray:
    """Rows for ``narrow_use_model``: N(0,1) in every column."""
    _, rng = _streams(seed)
    return np.ascontiguousarray(_f32(rng.standard_normal((n_rows, n_features))))


def with_missing(model: dict, X: np.ndarray, seed: int, p_left: float = 0.5, p_missing: float = 0.1):
    """The same model with a random default direction per node (left with
    probability ``p_left``) and a copy of ``X`` with a fraction ``p_missing``
    of its values replaced by NaN; returns ``(model, X)``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    m = dict(model)
    m["default_left"] = (rng.random(model["feature"].size) < p_left).astype(np.uint8)
    # a default-left node may not test against -inf
    m["default_left"][(model["feature"] >= 0) & (model["threshold"] == -np.inf)] = 0
    Xm = np.array(X, np.float32, copy=True)
    Xm[rng.random(Xm.shape) < p_missing] = np.nan
    return m, Xm


def with_categories(model: dict, X: np.ndarray, seed: int, cat_cols, n_categories: int,
                    p_member: float = 0.5):
    """The same model with every internal node that tests a column of
    ``cat_cols`` made categorical, and a copy of ``X`` whose ``cat_cols`` hold
    category values; returns ``(model, X)``.

    Each such node gets a random set over categories ``[0, n_categories)``
    (each category in it with probability ``p_member``) as
    ``ceil(n_categories / 32)`` 32-bit words, one node in four with an extra
    all-zero word. The rows' category columns hold integers drawn from
    ``[0, n_categories + 4)``, a quarter of them with a fractional part added,
    and a few negative values, NaN, +inf and -0.0.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    m = dict(model)
    cat_cols = np.asarray(cat_cols, np.int64)
    feat = np.asarray(model["feature"])
    words = (n_categories + 31) // 32
    off = [0]
    bits = []
    for i in range(feat.size):
        if feat[i] >= 0 and np.isin(feat[i], cat_cols):
            w = words + (1 if rng.random() < 0.25 else 0)
            member = rng.random(32 * w) < p_member
            member[n_categories:] = False
            node_bits = np.zeros(w, np.uint64)
            for c in np.flatnonzero(member):
                node_bits[c // 32] |= np.uint64(1) << np.uint64(c % 32)
            bits.extend(int(b) for b in node_bits)
            off.append(off[-1] + w)
        else:
            off.append(off[-1])
    m["cat_offset"] = np.asarray(off, np.int64)
    m["cat_bits"] = np.asarray(bits, np.uint32)
    Xc = np.array(X, np.float32, copy=True)
    n = Xc.shape[0]
    for c in cat_cols:
        v = rng.integers(0, n_categories + 4, size=n).astype(np.float64)
        frac = rng.random(n) < 0.25
        v[frac] += rng.random(int(frac.sum()))
        u = rng.random(n)
        v[u < 0.03] = -rng.random(int((u < 0.03).sum())) * 3.0
        v[(u >= 0.03) & (u < 0.05)] = np.nan
        v[(u >= 0.05) & (u < 0.06)] = np.inf
        v[(u >= 0.06) & (u < 0.07)] = -0.0
        Xc[:, c] = _f32(v)
    return m, Xc


def make_rows(cfg: int, n_rows: int) -> np.ndarray:
    """``n_rows`` seeded input rows of workload ``cfg``, float32 [n_rows, F]."""
    _, rng = _streams(CONFIGS[cfg]["seed"])
    if cfg == 1:
        x = rng.random((n_rows, 8))
    elif cfg == 2:
        x = rng.standard_normal((n_rows, 28))
    elif cfg == 3:
        x = rng.uniform(-1.0, 1.0, (n_rows, 2000))
    elif cfg == 4:
        x = np.empty((n_rows, 54))
        x[:, :_CFG4_CONT] = rng.standard_normal((n_rows, _CFG4_CONT))
        x[:, _CFG4_CONT:] = rng.integers(0, 2, (n_rows, 54 - _CFG4_CONT))
    elif cfg == 5:
        x = rng.random((n_rows, 100))
    else:
        raise ValueError(f"unknown config {cfg}")
    return np.ascontiguousarray(_f32(x))


def make_config(cfg: int, n_rows: int | None = None):
    """(model, X) for workload ``cfg``; ``n_rows`` defaults to its batch size."""
    n = CONFIGS[cfg]["n_rows"] if n_rows is None else n_rows
    return make_model(cfg), make_rows(cfg, n)


def permute_nodes(model: dict, seed: int) -> dict:
    """The same ensemble with each tree's non-root nodes renumbered at random.

    Node 0 stays the root. Returns a new dict; leaf ids reported against it
    are in the new numbering (``perm[old] = new`` per tree is stored under
    ``"_perm"``).
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    off = model["tree_node_offset"]
    ld = model["leaf_dim"]
    out = {k: v for k, v in model.items()}
    feature = model["feature"].copy()
    threshold = model["threshold"].copy()
    left = model["left"].copy()
    right = model["right"].copy()
    value = model["leaf_value"].reshape(-1, ld).copy()
    perms = []
    for t in range(model["n_trees"]):
        a, b = int(off[t]), int(off[t + 1])
        n = b - a
        perm = np.concatenate([[0], 1 + rng.permutation(n - 1)]).astype(np.int32)  # old -> new
        inv = np.empty(n, np.int32)
        inv[perm] = np.arange(n, dtype=np.int32)  # new -> old
        f_old = model["feature"][a:b]
        feature[a:b] = f_old[inv]
        threshold[a:b] = model["threshold"][a:b][inv]
        lo = model["left"][a:b][inv]
        ro = model["right"][a:b][inv]
        left[a:b] = np.where(lo >= 0, perm[np.maximum(lo, 0)], -1)
        right[a:b] = np.where(ro >= 0, perm[np.maximum(ro, 0)], -1)
        value[a:b] = model["leaf_value"].reshape(-1, ld)[a:b][inv]
        perms.append(perm)
    out.update(feature=feature, threshold=threshold, left=left, right=right,
               leaf_value=value.reshape(-1), _perm=perms)
    return out


def model_stats(model: dict) -> dict:
    """Shape statistics of an ensemble: max depth, mean leaf depth, node counts."""
    off = model["tree_node_offset"]
    depths, leaf_depth_sum, n_leaves = [], 0, 0
    for t in range(model["n_trees"]):
        a, b = int(off[t]), int(off[t + 1])
        d = np.zeros(b - a, np.int64)
        stack = [0]
        while stack:
            v = stack.pop()
            if model["feature"][a + v] >= 0:
                for c in (model["left"][a + v], model["right"][a + v]):
                    d[c] = d[v] + 1
                    stack.append(int(c))
        leaf = model["feature"][a:b] < 0
        depths.append(int(d[leaf].max()))
        leaf_depth_sum += int(d[leaf].sum())
        n_leaves += int(leaf.sum())
    return {
        "max_depth": max(depths),
        "mean_leaf_depth": leaf_depth_sum / max(n_leaves, 1),
        "n_nodes": int(off[-1]),
        "n_leaves": n_leaves,
    }

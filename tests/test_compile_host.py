"""hb_compile's tensors (host-only handles, no GPU): hand-derived tables,
size formulas, and Algorithms 1-3 run over them in numpy against the oracle."""
import numpy as np
import pytest

import oracle
import paper_2010_04804_amd as hb
from paper_2010_04804_amd import synth
import emulate
import pins


def host(model, strategy="auto"):
    return hb.compile(model, strategy=strategy, device=-1)


def golden_model():
    trees, _ = pins.load_golden()
    return pins.model_from_trees(trees, 3)


def test_tree_a_gemm_tensors_match_table3_by_hand():
    # Tree A of the golden fixture: node 0 tests f0<0.5, node 1 f1<0.25,
    # node 2 f2<0.75; leaves 3,4,5,6 left to right. From Table 3's definitions:
    #   C (internal x leaf) = [[+1,+1,-1,-1], [+1,-1,0,0], [0,0,+1,-1]]
    #   D (left edges on each leaf's root path) = [2, 1, 1, 0]
    h = host(golden_model())
    k_pad, l_pad, S = h.table("gemm", "dims", np.int32)
    assert (k_pad, l_pad, S) == (64, 16, 2)
    shape = h.table("gemm", "shape", np.int32)
    ct = h.table("gemm", "ct", np.int8).reshape(S, l_pad, k_pad)[shape[0]]
    want_c = np.array([[1, 1, -1, -1], [1, -1, 0, 0], [0, 0, 1, -1]])
    assert np.array_equal(ct[:4, :3], 4 * want_c.T)
    assert not ct[4:].any() and not ct[:, 3:].any()
    bias = h.table("gemm", "bias", np.int32).reshape(S, l_pad)[shape[0]]
    D = np.array([2, 1, 1, 0])
    assert np.array_equal(bias[:4], np.arange(4) - 256 * D)
    assert np.all(bias[4:] < -(1 << 20))
    lid = h.table("gemm", "leaf_id", np.int32).reshape(2, l_pad)
    assert list(lid[0, :4]) == [3, 4, 5, 6]
    # tree B (depth-first caller numbering) leaves left to right: 2, 3, 6, 7, 8
    assert list(lid[1, :5]) == [2, 3, 6, 7, 8]
    node = h.table("gemm", "node", np.uint32).reshape(2, k_pad, 2)
    assert list(node[0, :3, 1]) == [0, 1, 2]
    assert list(node[0, :3, 0].view(np.float32)) == [0.5, 0.25, 0.75]
    assert np.all(np.isneginf(node[0, 3:, 0].view(np.float32)))


def test_tree_b_ptt_padding_by_hand():
    # Tree B has depth 3 (node 5 sits under node 4); leaves 2 and 3 are at
    # depth 2 and leaf 8 at depth 2, so each is padded into 2 perfect leaves.
    h = host(golden_model())
    assert h.info()["ptt_depth"] == 3
    lid = h.table("ptt", "leaf_id", np.int32).reshape(2, 8)
    assert list(lid[1]) == [2, 2, 3, 3, 6, 7, 8, 8]
    assert list(lid[0]) == [3, 3, 4, 4, 5, 5, 6, 6]
    node = h.table("ptt", "node", np.uint32).reshape(2, 8, 2)
    # heap slot 1 = root (f1 < 0), 2 = node 1 (f0 < -1), 3 = node 4 (f2 < 2),
    # 6 = node 5 (f0 < 1); slots 4, 5, 7 are padding below leaves
    assert list(node[1, [1, 2, 3, 6], 1]) == [1, 0, 2, 0]
    assert list(node[1, [1, 2, 3, 6], 0].view(np.float32)) == [0.0, -1.0, 2.0, 1.0]


def test_tree_b_tt_records_by_hand():
    h = host(golden_model())
    n_pad = int(h.table("tt", "dims", np.int32)[0])
    assert n_pad == 10  # 9 nodes rounded up to even
    node = h.table("tt", "node", np.uint32).reshape(2, n_pad, 2)
    lid = h.table("tt", "leaf_id", np.int32).reshape(2, n_pad)
    # breadth-first order of tree B: 0, 1, 4, 2, 3, 5, 8, 6, 7
    assert list(lid[1, :9]) == [0, 1, 4, 2, 3, 5, 8, 6, 7]
    # canonical internal nodes 0, 1, 2, 5 (caller 0, 1, 4, 5) store their right
    # child (left = right - 1); leaves 3, 4, 6, 7, 8 and padding 9 point to themselves
    right = node[1, :, 1] >> 16
    assert list(right) == [2, 4, 6, 3, 4, 8, 6, 7, 8, 9]
    thr = node[1, :, 0].view(np.float32)
    assert list(thr[[0, 1, 2, 5]]) == [0.0, -1.0, 2.0, 1.0]
    assert np.all(np.isneginf(thr[[3, 4, 6, 7, 8, 9]]))
    assert list(h.table("tt", "depth", np.int32)) == [2, 3]


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_table_sizes_follow_table4(cfg):
    m = synth.make_model(cfg)
    h = host(m)
    info = h.info()
    T, D, ld = info["n_trees"], info["max_depth"], info["leaf_dim"]
    tb = info["table_bytes"]
    S = 1 << D
    # PTT: O(2^D) per tree: node records, leaf values and ids
    assert tb["ptt"] == T * max(S, 2) * 8 + T * S * ld * 4 + T * S * 4
    # TT: O(|N|) per tree (padded to the largest tree)
    n_pad = int(h.table("tt", "dims", np.int32)[0])
    assert n_pad >= max(np.diff(m["tree_node_offset"]))
    assert tb["tt"] == T * n_pad * 8 + T * 4 + T * n_pad * ld * 4 + T * n_pad * 4
    # GEMM: C is |I| x |L| per distinct shape
    k_pad, l_pad, nshape = (int(v) for v in h.table("gemm", "dims", np.int32))
    assert h.table("gemm", "ct", np.int8).size == nshape * l_pad * k_pad
    if cfg in (1, 2, 3, 4):
        assert nshape == 1 and info["balance"] == 1.0
    else:
        assert info["balance"] > 2.0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("strategy", ["ptt", "tt", "gemm"])
def test_emulated_algorithms_match_oracle(cfg, strategy):
    m = synth.make_model(cfg)
    n = 48 if cfg in (3, 4, 5) else 200
    X = synth.make_rows(cfg, n)
    if cfg == 4:
        X = X[:24]
    h = host(m)
    ids, raw = getattr(emulate, strategy)(h, m, X)
    o_raw, _, o_ids = oracle.predict(m, X)
    assert np.array_equal(ids, o_ids)
    assert np.allclose(raw, o_raw, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("strategy", ["ptt", "tt", "gemm"])
def test_emulated_algorithms_on_tricky_ensembles(seed, strategy):
    """Random unbalanced ensembles with permuted numbering, ties, NaN, +-inf."""
    m = pins.random_small_ensemble(seed)
    X = pins.tricky_rows(np.random.Generator(np.random.PCG64(seed)), m, 300)
    h = host(m)
    ids, raw = getattr(emulate, strategy)(h, m, X)
    o_raw, _, o_ids = oracle.predict(m, X)
    assert np.array_equal(ids, o_ids)
    assert np.allclose(raw, o_raw, rtol=1e-12, atol=1e-12)


def test_selector_choices():
    assert host(synth.make_model(2)).select(1_000_000) == "ptt"
    assert host(synth.make_model(4)).select(1_000_000) == "ptt"
    assert host(synth.make_model(5)).select(1_000_000) == "tt"
    shallow = synth.perfect_forest(np.random.Generator(np.random.PCG64(0)), 4, 2, 3,
                                   lambda r, f: r.random(f.size), lambda r, n: r.random(n))
    shallow.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
    # the crossover sweep found GEMM slower than PTT at every depth and batch
    assert host(shallow).select(1) == "ptt"
    assert host(shallow).select(1000) == "ptt"
    assert host(synth.sweep_model("leafwise-d12")).select(1000) == "tt"
    assert host(synth.sweep_model("perfect-d7")).select(1) == "ptt"
    # batch-aware since the sweep with depth-11/12 models and narrow rows:
    # near-perfect trees take PTT up to its depth limit (12), unbalanced
    # trees PTT up to 256 rows (the trees-across-lanes walk) and TT above
    assert host(synth.sweep_model("perfect-d12")).select(1_000_000) == "ptt"
    assert host(synth.sweep_model("perfect-d11-n28")).select(100_000) == "ptt"
    assert host(synth.sweep_model("leafwise-d12-n28")).select(256) == "ptt"
    assert host(synth.sweep_model("leafwise-d12-n28")).select(257) == "tt"
    assert host(synth.make_model(5)).select(100) == "ptt"
    assert hb.compile(synth.make_model(2), strategy="tt", device=-1).select(10) == "tt"


@pytest.mark.parametrize("leaf_dim", [1, 2])
def test_feature_pruning_tables_and_emulation(leaf_dim):
    """Feature selection injection (Sec. 5.2): a 3000-column input whose trees
    test 37 columns compiles to tables indexed by rank among those 37; the
    exported column list is exactly the tested set, and all three algorithms
    run on the compact tables give the oracle's leaves and margins."""
    m = synth.narrow_use_model(3000, 37, 12, 5, seed=31, leaf_dim=leaf_dim)
    used = np.unique(m["feature"][m["feature"] >= 0])
    h = host(m)
    info = h.info()
    assert info["n_features"] == 3000 and info["n_used_features"] == used.size
    for s in ("ptt", "tt", "gemm"):
        assert np.array_equal(h.table(s, "features", np.int32), used)
    ptt_node = h.table("ptt", "node", np.uint32).reshape(-1, 2)
    assert ptt_node[:, 1].max() < used.size
    X = synth.narrow_use_rows(3000, 300, seed=31)
    o_raw, _, o_ids = oracle.predict(m, X)
    for s in ("ptt", "tt", "gemm"):
        ids, raw = getattr(emulate, s)(h, m, X)
        assert np.array_equal(ids, o_ids), s
        assert np.allclose(raw, o_raw, rtol=1e-12, atol=1e-12), s


def test_no_pruning_when_every_feature_is_tested():
    h = host(synth.make_model(2))
    assert h.info()["n_used_features"] == 28
    assert np.array_equal(h.table("ptt", "features", np.int32), np.arange(28))


@pytest.mark.parametrize("strategy", ["ptt", "tt", "gemm"])
@pytest.mark.parametrize("cfg", [1, 5])
def test_missing_values_default_directions(cfg, strategy):
    """Per-node default directions for NaN: the compiled tables send a node's
    missing values through a tile column that reads NaN as -inf (left) or
    through the plain column (right); emulating the algorithms on them gives
    the oracle's leaves."""
    m, X = synth.with_missing(synth.make_model(cfg), synth.make_rows(cfg, 300), seed=cfg)
    h = host(m)
    cols = h.table(strategy, "features", np.int32)
    assert ((cols >> 30) & 1).any() and ((cols >> 30) & 1 == 0).any()
    ids, raw = getattr(emulate, strategy)(h, m, X)
    o_raw, _, o_ids = oracle.predict(m, X)
    assert np.array_equal(ids, o_ids)
    assert np.allclose(raw, o_raw, rtol=1e-12, atol=1e-12)


def test_missing_values_tricky_ensembles():
    for seed in range(4):
        m = pins.random_small_ensemble(seed)
        X = pins.tricky_rows(np.random.Generator(np.random.PCG64(seed)), m, 200)
        m, _ = synth.with_missing(m, X[:1], seed=seed)
        h = host(m)
        o_raw, _, o_ids = oracle.predict(m, X)
        for s in ("ptt", "tt", "gemm"):
            ids, raw = getattr(emulate, s)(h, m, X)
            assert np.array_equal(ids, o_ids), (seed, s)


@pytest.mark.parametrize("cfg", [1, 2, 4, 5])
def test_tt_packed_tables_walk_in_bounds(cfg):
    """The row-parallel TT kernels' packed tables ("fast_node", "fast_leaf"),
    walked in numpy the way the kernel walks them, for every tree of the
    padded count (a multiple of 32): the state never leaves its tree, the
    padding trees stay at their root, and the leaf ids are the oracle's.
    Rows include negative values, which a zero record would send to child
    offset -8."""
    model = synth.make_model(cfg)
    h = hb.compile(model, device=-1)
    info = h.info()
    T = info["n_trees"]
    node = h.table("tt", "fast_node", np.uint32).reshape(-1, 2)
    leaf = h.table("tt", "fast_leaf", np.uint32).reshape(-1, 2)
    Tp = -(-T // 32) * 32
    NP = node.shape[0] // Tp
    assert node.shape[0] == Tp * NP and NP & (NP - 1) == 0 and leaf.shape == node.shape
    X = synth.make_rows(cfg, 256).astype(np.float32)
    X[::2] = -X[::2]
    cols = h.table("tt", "features", np.int32) & ((1 << 30) - 1)
    Xt = X[:, cols]
    thr = node[:, 0].view(np.float32)
    feat = (node[:, 1] & 0xFFFF).astype(np.int64)
    right = (node[:, 1] >> 16).astype(np.int64)
    base = (np.arange(Tp, dtype=np.int64) * NP)[None, :]
    rows = np.arange(X.shape[0])[:, None]
    s = np.zeros((X.shape[0], Tp), dtype=np.int64)
    for _ in range(int(h.table("tt", "depth", np.int32).max()) + 2):
        idx = base + s // 8
        f = feat[idx]
        assert (f < Xt.shape[1]).all()
        s = right[idx] - 8 * (Xt[rows, f] < thr[idx])
        assert ((s >= 0) & (s < 8 * NP) & (s % 8 == 0)).all()
    assert (s[:, T:] == 0).all()
    _, _, o_ids = oracle.predict(model, X)
    assert np.array_equal(leaf[base + s // 8, 1][:, :T].astype(np.int32), o_ids)


@pytest.mark.parametrize("strategy", ["ptt", "tt", "gemm"])
@pytest.mark.parametrize("seed", range(4))
def test_categorical_splits_tables_and_emulation(seed, strategy):
    """Categorical nodes compile to 0/1 indicator columns (one per distinct
    column, category set and default direction) that the nodes test against
    0.5; the three algorithms run on the compiled tables give the oracle's
    leaves, with NaN, negative, fractional, -0.0, +inf and out-of-range
    category values in the rows."""
    m, X = pins.random_categorical_ensemble(seed, n_rows=300)
    h = host(m)
    n_cols = h.info()["n_used_features"]
    cols = h.table(strategy, "features", np.int32)[:n_cols]
    assert ((cols >> 29) & 1).any() and ((cols >> 29) & 1 == 0).any()
    ids, raw = getattr(emulate, strategy)(h, m, X)
    o_raw, _, o_ids = oracle.predict(m, X)
    assert np.array_equal(ids, o_ids)
    assert np.allclose(raw, o_raw, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("cfg", [1, 5])
def test_categorical_on_workload_shapes(cfg):
    m0 = synth.make_model(cfg)
    m, X = synth.with_categories(m0, synth.make_rows(cfg, 200), seed=cfg, cat_cols=[0, 3], n_categories=40)
    m, X = synth.with_missing(m, X, seed=cfg + 1, p_missing=0.05)
    h = host(m)
    o_raw, _, o_ids = oracle.predict(m, X)
    for s in ("ptt", "tt", "gemm"):
        if not h.info()["feasible"][s]:
            continue
        ids, raw = getattr(emulate, s)(h, m, X)
        assert np.array_equal(ids, o_ids), s
        assert np.allclose(raw, o_raw, rtol=1e-12, atol=1e-12), s


def test_categorical_columns_are_shared():
    """Nodes with the same column, the same categories (trailing zero words
    aside) and the same default direction share one indicator column; a
    different set or direction gets its own."""
    leaf = (-1, 0.0, -1, -1, 1.0, 0)
    trees = [
        [(0, 0.0, 1, 2, 0.0, 0, (1, [1, 2])), leaf, leaf],
        [(0, 0.0, 1, 2, 0.0, 0, (2, [1, 2])), leaf, leaf],   # same set, an extra zero word
        [(0, 0.0, 1, 2, 0.0, 1, (1, [1, 2])), leaf, leaf],   # NaN left
        [(0, 0.0, 1, 2, 0.0, 0, (1, [1, 3])), leaf, leaf],   # another set
        [(0, 0.5, 1, 2, 0.0, 0), leaf, leaf],                # numeric on the same column
    ]
    m = pins.model_from_trees(trees, 2)
    h = host(m)
    info = h.info()
    assert info["n_used_features"] == 4
    table = h.table("ptt", "features", np.int32)
    cols = table[:4]
    assert cols[0] == 0 and ((cols[1:] >> 29) & 1).all()
    descs = sorted((int(table[c & ((1 << 29) - 1)]), int(table[(c & ((1 << 29) - 1)) + 1]),
                    tuple(table[(c & ((1 << 29) - 1)) + 2:(c & ((1 << 29) - 1)) + 2 + int(table[(c & ((1 << 29) - 1)) + 1])]),
                    int((c >> 30) & 1)) for c in cols[1:])
    assert descs == [(0, 1, (6,), 0), (0, 1, (6,), 1), (0, 1, (10,), 0)]
    X = np.asarray([[1, 0], [2.5, 0], [3, 0], [np.nan, 0], [-1, 0], [0.0, 0]], np.float32)
    o_raw, _, o_ids = oracle.predict(m, X)
    for s in ("ptt", "tt", "gemm"):
        ids, raw = getattr(emulate, s)(h, m, X)
        assert np.array_equal(ids, o_ids), s


def _node_depths(model, t):
    off = model["tree_node_offset"]
    a, b = int(off[t]), int(off[t + 1])
    d = np.zeros(b - a, np.int64)
    stack = [0]
    while stack:
        v = stack.pop()
        if model["feature"][a + v] >= 0:
            for c in (model["left"][a + v], model["right"][a + v]):
                d[c] = d[v] + 1
                stack.append(int(c))
    return d


def test_tt_walk_levels_on_the_leafwise_workload():
    """The row-parallel TT walk of the leaf-wise workload: a chunk of 8 trees
    walks as many levels as its deepest tree (12 for every chunk here), while a
    row needs only the depth of the leaf it reaches (5.2 on average). The
    wave's 64 rows move in lockstep, and some row reaches depth 11-12 in most
    trees, so stopping a tree once all 64 rows of a wave sit at leaves would
    save only about 7% of the levels."""
    m = synth.make_model(5)
    X = synth.make_rows(5, 4096)
    h = host(m)
    depth = h.table("tt", "depth", np.int32)
    T, TC = m["n_trees"], 8
    chunk_levels = sum(TC * int(depth[c:c + TC].max()) for c in range(0, T, TC))
    _, _, ids = oracle.predict(m, X)
    L = np.stack([_node_depths(m, t)[ids[:, t]] for t in range(T)], 1)
    useful = L.mean(0).sum()                      # levels a row needs, over all trees
    wave_tree = L.reshape(-1, 64, T).max(1).mean()  # levels a wave needs per tree
    print(f"[tt levels] walked per row {chunk_levels}, needed {useful:.1f} "
          f"({useful / chunk_levels:.3f}), per-wave tree need {wave_tree:.2f} of 12")
    assert int(depth.max()) == 12 and chunk_levels == 6048
    assert 0.42 < useful / chunk_levels < 0.45
    assert 11.0 < wave_tree < 11.4

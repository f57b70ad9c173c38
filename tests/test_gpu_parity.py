"""GPU parity: the HIP path through the C-ABI against the CPU oracle.

Leaf ids must be identical; scores must satisfy |gpu - oracle| <= 1e-5 (1 + |oracle|)
elementwise, with the oracle aggregating in double precision. Every case
prints its config, strategy and size before touching the GPU.
"""
import os

import numpy as np
import pytest

import oracle
import paper_2010_04804_amd as hb
from paper_2010_04804_amd import synth
import pins

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

STRATEGIES = ["ptt", "tt", "gemm"]
TOL = 1e-5


def say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


_handles = {}


def handle(cfg):
    if cfg not in _handles:
        _handles[cfg] = (synth.make_model(cfg), None)
        _handles[cfg] = (_handles[cfg][0], hb.compile(_handles[cfg][0], device=0))
    return _handles[cfg]


def run(h, X, strategy, leaves=True, stream=None, workspace=True):
    Xd = torch.from_numpy(X).cuda()
    s, ids = hb.predict(h, Xd, strategy=strategy, leaves=leaves, stream=stream, workspace=workspace)
    torch.cuda.synchronize()
    return s.cpu().numpy(), (ids.cpu().numpy() if ids is not None else None)


ORACLE_THREADS = min(16, os.cpu_count() or 1)


def check(model, X, scores, ids, label):
    o_raw, o_out, o_ids = oracle.predict(model, X, n_threads=ORACLE_THREADS)
    if ids is not None:
        bad = np.argwhere(ids != o_ids)
        assert bad.size == 0, f"{label}: {len(bad)} leaf ids differ, first {bad[:5].tolist()}"
    err = np.abs(scores.astype(np.float64) - o_out)
    lim = TOL * (1.0 + np.abs(o_out))
    worst = float((err / lim).max()) if err.size else 0.0
    assert np.all(err <= lim), f"{label}: score error {worst:.3g} x tolerance"
    return worst


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_config_parity(cfg, strategy):
    model, h = handle(cfg)
    n = {1: 1000, 2: 10_000, 3: 2000, 4: 3000, 5: 10_000}[cfg]
    say("config", cfg, strategy, "rows", n)
    X = synth.make_rows(cfg, n)
    scores, ids = run(h, X, strategy)
    check(model, X, scores, ids, f"cfg{cfg}/{strategy}")


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("n", [1, 2, 63, 65, 255, 257, 513])
def test_ragged_batches(strategy, n):
    model, h = handle(2)
    say("ragged", strategy, n)
    X = synth.make_rows(2, n)
    scores, ids = run(h, X, strategy)
    check(model, X, scores, ids, f"ragged{n}/{strategy}")


@pytest.mark.parametrize("workspace", [False, True])
@pytest.mark.parametrize("strategy", ["ptt", "tt"])
@pytest.mark.parametrize("cfg,n", [(2, 1024), (2, 1025), (2, 1027), (2, 4096), (2, 12288), (2, 12289), (5, 16384),
                                   (5, 16385), (4, 1025), (4, 4095), (3, 4093), (3, 20_001)])
def test_tree_parallel_boundaries(cfg, n, strategy, workspace):
    """Batch sizes around the switches between the trees-across-lanes kernel
    and the row-parallel ones (1,024 rows with a workspace; 12,288 rows for
    PTT and 16,384 for TT without), and its four-rows-per-workgroup form with
    a ragged last workgroup, also with seven outputs; config 3's 2000-feature
    rows take it at every size."""
    model, h = handle(cfg)
    say("tree-parallel", cfg, strategy, n, "workspace" if workspace else "no workspace")
    X = synth.make_rows(cfg, n)
    scores, ids = run(h, X, strategy, workspace=workspace)
    check(model, X, scores, ids, f"lanes cfg{cfg}/{n}/{strategy}/ws={workspace}")


@pytest.mark.parametrize("strategy", ["ptt", "tt"])
@pytest.mark.parametrize("cfg,n", [(2, 513), (2, 1000), (2, 4097), (2, 30_000), (2, 65_536), (4, 700), (4, 9000),
                                   (5, 600), (5, 20_001), (3, 1000)])
def test_tree_split_parity(cfg, n, strategy):
    """With a workspace (hb_predict_ws), batches of up to 65,536 rows divide
    their trees among workgroups and add the partial sums in a second kernel:
    the result meets the oracle bar and its leaf ids equal the unsplit call's."""
    model, h = handle(cfg)
    say("tree split", cfg, strategy, n)
    X = synth.make_rows(cfg, n)
    s_ws, i_ws = run(h, X, strategy)
    s_no, i_no = run(h, X, strategy, workspace=False)
    check(model, X, s_ws, i_ws, f"split cfg{cfg}/{n}/{strategy}")
    check(model, X, s_no, i_no, f"unsplit cfg{cfg}/{n}/{strategy}")
    assert np.array_equal(i_ws, i_no)


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("cfg,n", [(2, 20_000), (2, 300), (4, 20_000), (4, 300)])
def test_raw_margins(cfg, n, strategy):
    """The sigmoid and softmax workloads with the transform removed: the
    aggregated margins themselves meet the bar against the oracle's raw
    margins (a saturated sigmoid or a dominant softmax class can hide margin
    error in the transformed scores). The worst error as a fraction of the
    tolerance is printed."""
    model = dict(synth.make_model(cfg))
    model["transform"] = "none"
    h = hb.compile(model, device=0)
    X = synth.make_rows(cfg, n)
    say("raw margins", cfg, n, strategy)
    scores, ids = run(h, X, strategy)
    o_raw, o_out, o_ids = oracle.predict(model, X, n_threads=ORACLE_THREADS)
    assert np.array_equal(o_raw, o_out)  # no transform: the oracle's output is its margin
    worst = check(model, X, scores, ids, f"raw cfg{cfg}/{n}/{strategy}")
    say("worst raw-margin error / tolerance", cfg, strategy, n, f"{worst:.3g}")
    h.close()


@pytest.mark.parametrize("cfg,n", [(2, 1), (2, 2), (2, 17), (2, 100), (2, 1000), (2, 4096), (4, 1), (4, 300),
                                   (1, 33)])
def test_gemm_tree_split(cfg, n):
    """GEMM with a workspace (hb_predict_ws) on batches of up to 4,096 rows
    divides the trees, in groups of four, among 16-row tile workgroups and
    adds the partial sums in a second kernel: the oracle bar, and leaf ids
    equal to the unsplit call's (Algorithm 1, Table 3)."""
    model, h = handle(cfg)
    say("gemm tree split", cfg, n)
    nbytes = hb.workspace_bytes(h, n, "gemm")
    kernels = [p["kernel"] for p in h.plan(n, "gemm", nbytes)]
    if cfg != 1:  # config 1's depth-3 trees have no 256-leaf tiles
        assert nbytes > 0 and kernels[0].startswith("gemm_tile_kernel<") and kernels[-1].startswith("split_finish"), kernels
    X = synth.make_rows(cfg, n)
    s_ws, i_ws = run(h, X, "gemm")
    s_no, i_no = run(h, X, "gemm", workspace=False)
    check(model, X, s_ws, i_ws, f"gemm split cfg{cfg}/{n}")
    check(model, X, s_no, i_no, f"gemm unsplit cfg{cfg}/{n}")
    assert np.array_equal(i_ws, i_no)


@pytest.mark.parametrize("strategy", ["ptt", "tt"])
def test_tree_split_uses_and_reuses_the_workspace(strategy):
    """The split writes its partial sums into the caller's workspace; one
    workspace serves successive calls (the second one smaller), and a
    workspace smaller than hb_workspace_bytes still gives correct results."""
    model, h = handle(2)
    nbytes = hb.workspace_bytes(h, 4000, strategy)
    assert nbytes == 16 * 4000 * 8
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    rows = synth.make_rows(2, 8500)
    for lo, n, avail in [(0, 4000, nbytes), (4000, 1500, nbytes), (5500, 3000, nbytes // 3)]:
        say("workspace reuse", strategy, n, avail)
        X = np.ascontiguousarray(rows[lo:lo + n])
        Xd = torch.from_numpy(X).cuda()
        scores = torch.empty((n, 1), dtype=torch.float32, device="cuda")
        ids = torch.empty((n, 500), dtype=torch.int32, device="cuda")
        hb.predict_ptr(h, Xd.data_ptr(), n, scores.data_ptr(), ids.data_ptr(), strategy,
                       torch.cuda.current_stream().cuda_stream, ws.data_ptr(), avail)
        torch.cuda.synchronize()
        if n == 4000:
            assert int((ws != 0xFF).sum()) > 0, "the split did not write the workspace"
        check(model, X, scores.cpu().numpy(), ids.cpu().numpy(), f"ws {strategy}/{n}/{avail}")


@pytest.mark.parametrize("n_trees,depth,heap", [(500, 8, True), (64, 6, False), (48, 6, False), (40, 6, False),
                                                 (36, 6, False), (3500, 8, False), (64, 8, True), (40, 8, True),
                                                 (48, 6, True), (36, 5, True)])
def test_leaf_id_lines_at_any_offset(n_trees, depth, heap):
    """Leaf ids leave as whole 128-byte lines whose first tree depends on the
    output's offset within a line and on the row (tree counts with 1, 2, 4 or
    8 line phases); every offset gives the oracle's ids, and nothing outside
    the output changes. Offsets of 1 and 2 ints take the unaligned path.
    Heap-ordered perfect trees of depth <= 8 (heap=True) keep their leaf
    values apart and form ids from 8-bit leaf slots; permuted numberings keep
    16-bit ids: both with 8-tree chunks (one or several line phases per line
    tree) and with 16-tree chunks (depth 5 and 6)."""
    if n_trees == 500:
        model, h = handle(2)
    else:
        rng = np.random.Generator(np.random.PCG64(700 + n_trees + 1000 * heap))
        model = synth.perfect_forest(rng, n_trees, depth, 28, lambda r, f: r.standard_normal(f.size),
                                     lambda r, n: r.normal(0.0, 0.05, n))
        model.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
        if not heap:
            model = synth.permute_nodes(model, n_trees)
        h = hb.compile(model, device=0)
    sizes = [3001] if n_trees == 3500 else [3001, 20_000]
    if n_trees != 3500:
        ptt_kernels = [p["kernel"] for p in h.plan(20_000, "ptt")]
        assert any(k.startswith("fast_kernel<3,") for k in ptt_kernels) == heap, ptt_kernels
    for n in sizes:
        X = synth.make_rows(2, n)
        Xd = torch.from_numpy(X).cuda()
        _, _, o_ids = oracle.predict(model, X, n_threads=ORACLE_THREADS)
        for strategy in ("ptt", "tt"):
            for off in (0, 4, 12, 28, 1, 2):
                for ws in (False, True):
                    say("id lines", n_trees, n, strategy, "offset", off, "ws" if ws else "no ws")
                    buf = torch.full((n * n_trees + 64,), -7, dtype=torch.int32, device="cuda")
                    scores = torch.empty((n, 1), dtype=torch.float32, device="cuda")
                    nws = hb.workspace_bytes(h, n, strategy) if ws else 0
                    wsb = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda")
                    hb.predict_ptr(h, Xd.data_ptr(), n, scores.data_ptr(), buf.data_ptr() + 4 * off, strategy,
                                   torch.cuda.current_stream().cuda_stream, wsb.data_ptr() if nws else None, nws)
                    torch.cuda.synchronize()
                    b = buf.cpu().numpy()
                    got = b[off:off + n * n_trees].reshape(n, n_trees)
                    bad = np.argwhere(got != o_ids)
                    assert bad.size == 0, f"offset {off}/{strategy}/ws={ws}: {len(bad)} ids differ, first {bad[:4].tolist()}"
                    assert np.all(b[:off] == -7) and np.all(b[off + n * n_trees:] == -7), "write outside the output"


@pytest.mark.parametrize("kind", ["scalar", "classes", "vector", "classes12", "vector5"])
@pytest.mark.parametrize("n_trees,n", [(1, 17), (2, 16), (3, 33), (9, 40), (10, 300), (37, 1007), (64, 4099)])
def test_gemm_wide_rows(kind, n_trees, n):
    """Depth-8 trees over 1,500 features: the GEMM tables' 256-row feature
    tile does not fit in LDS, so 16-row tiles with C^T in registers take
    the batch. From 9 trees on the used columns leave room for one tile
    workgroup per CU, which runs two groups of four waves (odd tree counts
    end on a pair of one tree, and the tree split's last part of one tree
    leaves the second group without a pair); 1 to 3 trees use a few hundred
    columns and take the four-wave tiles, two per CU. One output, 3 and 12
    classes, 2- and 5-vector leaves: each output count the eight-wave kernel
    is compiled for. Rows hold ties, NaN and infinities; with and without
    the tree split."""
    rng = np.random.Generator(np.random.PCG64(4200 + n_trees + n))
    F = 1500
    K = {"scalar": 1, "classes": 3, "vector": 2, "classes12": 12, "vector5": 5}[kind]
    ld = K if kind.startswith("vector") else 1
    model = synth.perfect_forest(rng, n_trees, 8, F, lambda r, f: r.standard_normal(f.size),
                                 lambda r, k: r.standard_normal(k * ld), leaf_dim=ld)
    classes = kind.startswith("classes")
    model.update(n_outputs=K, aggregation="mean" if ld > 1 else "sum",
                 transform="softmax" if classes else "none", base_score=None,
                 tree_class=(np.arange(n_trees) % K).astype(np.int32) if classes else None)
    model = synth.permute_nodes(model, n_trees + n)
    X = np.ascontiguousarray(pins.tricky_rows(rng, model, n))
    h = hb.compile(model, device=0)
    say("gemm wide rows", kind, n_trees, n)
    for ws in (True, False):
        plan = [p["kernel"] for p in h.plan(n, "gemm", hb.workspace_bytes(h, n, "gemm") if ws else 0)]
        km = {"scalar": 1, "classes": 8, "vector": 2, "classes12": 16, "vector5": 8}[kind]
        mode = 1 if classes else 2 if ld > 1 else 0
        assert plan[0] == (f"gemm_tile2_kernel<{mode}, {km}>" if n_trees >= 9 else f"gemm_tile_kernel<{mode}>"), plan
    scores, ids = run(h, X, "gemm")
    check(model, X, scores, ids, f"gemm wide {kind}/{n_trees}/{n}")
    scores, ids = run(h, X, "gemm", workspace=False)
    check(model, X, scores, ids, f"gemm wide unsplit {kind}/{n_trees}/{n}")


def _gemm_512_model(kind):
    """Shared-shape forests that reach the GEMM kernels with 512-row
    workgroups (batches of 32,768 rows and more whose feature tile fits
    beside C^T in LDS): the headline model; a two-output model with scalar
    leaves and a class per tree; perfect trees of depth 7 and 6 (128 and 64
    leaves, the 64-node slice kernels); depth 7 with 2-vector leaves."""
    if kind == "cfg2":
        return synth.make_model(2)
    rng = np.random.Generator(np.random.PCG64({"two_class": 9400, "depth7": 9401, "depth6": 9402,
                                                "depth7_vec": 9403}[kind]))
    depth = 6 if kind == "depth6" else 7 if kind.startswith("depth7") else 8
    ld = 2 if kind == "depth7_vec" else 1
    m = synth.perfect_forest(rng, 300 if kind != "two_class" else 200, depth, 28,
                             lambda r, f: r.standard_normal(f.size), lambda r, k: r.normal(0.0, 0.05, k * ld),
                             leaf_dim=ld)
    T = m["n_trees"]
    if kind == "two_class":
        m.update(n_outputs=2, tree_class=(np.arange(T) % 2).astype(np.int32), aggregation="sum",
                 transform="softmax", base_score=np.asarray([0.1, -0.2], np.float32))
    elif kind == "depth7_vec":
        m.update(n_outputs=2, tree_class=None, aggregation="mean", transform="none", base_score=None)
    else:
        m.update(n_outputs=1, tree_class=None, aggregation="sum", transform="sigmoid", base_score=None)
    return synth.permute_nodes(m, 31 + depth)


@pytest.mark.parametrize("kind,n,kernel", [
    ("cfg2", 65_536, "gemm_pipe_kernel<0, 512>"),
    ("two_class", 40_000, "gemm_pipe_kernel<1, 512>"),
    ("depth7", 40_001, "gemm_kernel<2, true, true, 0, 512, false>"),
    ("depth6", 33_000, "gemm_kernel<1, true, true, 0, 512, false>"),
    ("depth7_vec", 32_768, "gemm_kernel<2, true, true, 2, 512, false>"),
])
def test_gemm_512_row_workgroups(kind, n, kernel):
    """GEMM with 512-row workgroups (Algorithm 1, Table 3): every row's
    scores and leaf ids against the oracle. The launch plan the library
    reports names the kernel each case is meant to reach, the headline
    workload's included (the one its GEMM throughput is measured on)."""
    m = _gemm_512_model(kind)
    h = handle(2)[1] if kind == "cfg2" else hb.compile(m, device=0)
    plan = h.plan(n, "gemm")
    assert [p["kernel"] for p in plan] == [kernel], plan
    X = synth.make_rows(2, n)
    if kind != "cfg2":
        X = np.ascontiguousarray(pins.tricky_rows(np.random.Generator(np.random.PCG64(n)), m, n))
    say("gemm 512-row", kind, n, kernel)
    scores, ids = run(h, X, "gemm", workspace=False)
    check(m, X, scores, ids, f"gemm512 {kind}/{n}")


def _vector_forest(n_features, n_trees, depth, seed):
    rng = np.random.Generator(np.random.PCG64(seed))

    def leaves(r, n):
        p = r.random(n)
        return np.stack([1.0 - p, p], axis=1)

    m = synth.perfect_forest(rng, n_trees, depth, n_features,
                             lambda r, f: r.standard_normal(f.size), leaves, leaf_dim=2)
    m.update(n_outputs=2, tree_class=None, aggregation="mean", transform="none", base_score=None)
    return m, rng


@pytest.mark.parametrize("strategy", ["ptt", "tt"])
@pytest.mark.parametrize("n_features,n", [(28, 9000), (28, 20_000), (50_000, 37)])
def test_vector_leaf_forest_routes(n_features, n, strategy):
    """Random forests with probability-vector leaves take the row-parallel
    fast kernels at large batches when the rows fit their LDS tile, the
    trees-across-lanes kernel at small ones, and the general kernel reading
    features from global memory when a single row does not fit in LDS."""
    m, rng = _vector_forest(n_features, 100, 7, 21)
    X = np.ascontiguousarray(rng.standard_normal((n, n_features)).astype(np.float32))
    say("vector forest", strategy, n_features, n)
    h = hb.compile(m, device=0)
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"vecRF F{n_features} n{n}/{strategy}")


@pytest.mark.parametrize("ld", [2, 3, 5, 16])
@pytest.mark.parametrize("leafwise", [False, True])
def test_vector_leaves_row_parallel(ld, leafwise):
    """Vector leaves in the row-parallel fast kernels (leaf vectors read from
    the leaf-value table), with and without the tree split, with leaf ids, for
    perfect trees (PTT and TT) and leaf-wise trees (TT), 1 to 16 values."""
    rng = np.random.Generator(np.random.PCG64(9100 + ld + 50 * leafwise))
    T = 70
    if leafwise:
        m = synth.leafwise_forest(rng, T, 90, 10, 0.7, 24, lambda r, f: r.standard_normal(f.size),
                                  lambda r, k: r.standard_normal(k))
        m["leaf_dim"] = ld
        m["leaf_value"] = rng.standard_normal(m["leaf_value"].size * ld).astype(np.float32)
    else:
        m = synth.perfect_forest(rng, T, 7, 24, lambda r, f: r.standard_normal(f.size),
                                 lambda r, k: r.standard_normal(k * ld), leaf_dim=ld)
    m.update(n_outputs=ld, tree_class=None, aggregation="mean", transform="softmax" if ld > 2 else "none",
             base_score=rng.standard_normal(ld).astype(np.float32))
    m = synth.permute_nodes(m, ld)
    h = hb.compile(m, device=0)
    for n in (5000, 40_001):
        X = np.ascontiguousarray(pins.tricky_rows(rng, m, n))
        for strategy in (("tt",) if leafwise else ("ptt", "tt")):
            if not h.info()["feasible"][strategy]:
                continue
            for ws in (False, True):
                say("vector leaves", ld, "leafwise" if leafwise else "perfect", n, strategy, ws)
                scores, ids = run(h, X, strategy, workspace=ws)
                check(m, X, scores, ids, f"vec{ld}/{leafwise}/{n}/{strategy}/ws={ws}")


@pytest.mark.parametrize("strategy", STRATEGIES)
def test_rf_vector_workload(strategy):
    """The narrow binary random forest that the workload table reports beside
    the five (2-vector leaves, 28 features) at 70,001 rows."""
    m = synth.rf_vector_model()
    h = hb.compile(m, device=0)
    X = synth.rf_vector_rows(70_001)
    say("rf vector workload", strategy)
    scores, ids = run(h, X, strategy, workspace=False)
    check(m, X, scores, ids, f"rf2/{strategy}")


def test_two_class_scalar_leaves_row_parallel():
    """Two outputs with scalar leaves and a class per tree take the
    two-accumulator fast kernels (1024-row workgroups) like 2-vector leaves."""
    rng = np.random.Generator(np.random.PCG64(9300))
    m = synth.perfect_forest(rng, 90, 8, 20, lambda r, f: r.standard_normal(f.size), lambda r, k: r.standard_normal(k))
    m.update(n_outputs=2, tree_class=(rng.random(90) < 0.5).astype(np.int32), aggregation="sum",
             transform="softmax", base_score=None)
    h = hb.compile(m, device=0)
    for n in (70_001, 65_536):  # 65,536 rows with a workspace: 1024-row workgroups with the tree split
        X = np.ascontiguousarray(pins.tricky_rows(rng, m, n))
        for strategy in ("ptt", "tt"):
            for ws in (False, True):
                say("two classes", n, strategy, ws)
                scores, ids = run(h, X, strategy, workspace=ws)
                check(m, X, scores, ids, f"2cls/{n}/{strategy}/ws={ws}")


@pytest.mark.parametrize("missing", [False, True])
def test_tt_widest_workgroups(missing):
    """TreeTraversal in 1024-row workgroups (batches of 65,536 rows and more
    with a narrow feature tile), with a ragged last workgroup, and with
    default directions for missing values."""
    model, h = handle(2)
    n = 70_001
    X = synth.make_rows(2, n)
    if missing:
        model, X = synth.with_missing(model, X, seed=77)
        h = hb.compile(model, device=0)
    say("tt 1024-row workgroups", n, "missing" if missing else "")
    scores, ids = run(h, X, "tt", workspace=False)
    check(model, X, scores, ids, f"tt1024 missing={missing}")


def _random_model(seed):
    """A seeded random ensemble: perfect or leaf-wise trees, 1 to 700 trees,
    depth 1 to 12, 1 to 300 features, scalar leaves with 1 to 9 output
    columns or vector leaves of 2 to 5 values, any aggregation and transform,
    numbering permuted; plus a batch size and rows that include ties."""
    rng = np.random.Generator(np.random.PCG64(9000 + seed))
    T = int(rng.choice([1, 3, 31, 64, 65, 130, 257, 700]))
    F = int(rng.choice([1, 2, 7, 28, 64, 150, 300]))
    thr = lambda r, f: r.standard_normal(f.size)
    if rng.random() < 0.5:
        depth = int(rng.integers(1, 13))
        ld = int(rng.choice([1, 1, 1, 2, 5]))
        m = synth.perfect_forest(rng, T, depth, F, thr, lambda r, n: r.standard_normal(n * ld), leaf_dim=ld)
    else:
        ld = 1
        max_depth = int(rng.integers(2, 12))
        n_leaves = int(rng.integers(2, min(200, 2 ** max_depth) + 1))
        m = synth.leafwise_forest(rng, T, n_leaves, max_depth, 0.7, F, thr, lambda r, n: r.standard_normal(n))
    K = ld if ld > 1 else int(rng.choice([1, 1, 3, 9]))
    m.update(n_outputs=K, aggregation=str(rng.choice(["sum", "mean"])),
             transform="softmax" if K > 1 and rng.random() < 0.5 else str(rng.choice(["none", "sigmoid"])),
             base_score=rng.standard_normal(K).astype(np.float32) if rng.random() < 0.3 else None,
             tree_class=rng.integers(0, K, T).astype(np.int32) if ld == 1 and K > 1 else None)
    m = synth.permute_nodes(m, seed)
    n = int(rng.choice([1, 5, 700, 3000, 40_000]))
    X = pins.tricky_rows(rng, m, n) if rng.random() < 0.5 else rng.standard_normal((n, F)).astype(np.float32)
    return m, np.ascontiguousarray(X)


@pytest.mark.parametrize("seed", range(24))
def test_random_ensembles(seed):
    """Seeded random shapes through every feasible strategy, with and without
    a workspace, with and without leaf ids."""
    m, X = _random_model(seed)
    h = hb.compile(m, device=0)
    info = h.info()
    o_raw, o_out, o_ids = oracle.predict(m, X, n_threads=ORACLE_THREADS)
    for strategy in ("ptt", "tt", "gemm"):
        if not info["feasible"][strategy]:
            continue
        for ws in (False, True):
            say("random", seed, strategy, "ws" if ws else "no ws", m["n_trees"], X.shape)
            scores, ids = run(h, X, strategy, workspace=ws, leaves=ws)
            if ids is not None:
                assert np.array_equal(ids, o_ids), f"random{seed}/{strategy}/ws={ws}: leaf ids differ"
            err = np.abs(scores.astype(np.float64) - o_out)
            assert np.all(err <= TOL * (1.0 + np.abs(o_out))), f"random{seed}/{strategy}/ws={ws}: scores"


def _layout_forest(n_trees, depth, leaf_dim, seed, n_features=12):
    rng = np.random.Generator(np.random.PCG64(seed))
    m = synth.perfect_forest(rng, n_trees, depth, n_features, lambda r, f: r.standard_normal(f.size),
                             lambda r, n: r.standard_normal(n * leaf_dim), leaf_dim=leaf_dim)
    m.update(n_outputs=leaf_dim, tree_class=None, aggregation="mean" if leaf_dim > 1 else "sum",
             transform="none", base_score=None)
    return m, rng


@pytest.mark.parametrize("strategy", ["ptt", "tt"])
@pytest.mark.parametrize("n", [37, 3000])
@pytest.mark.parametrize("n_trees,depth,leaf_dim", [(70, 0, 1), (300, 1, 1), (300, 5, 1), (100, 1, 2), (130, 4, 3),
                                                    (65, 3, 9)])
def test_lanes_layouts(n_trees, depth, leaf_dim, n, strategy):
    """The trees-across-lanes kernel's layouts at their edges: node records
    interleaved by 64 trees with a partial last group and a second round of
    trees per lane (300 trees), the 32-byte last-level record at depth 1 and
    with two leaf values, packed leaf records of 4 and 16 words (3 and 9
    values), single-leaf trees (no last level); one row per workgroup (37
    rows, and 9 values at any size) and four."""
    m, rng = _layout_forest(n_trees, depth, leaf_dim, seed=500 + 7 * depth + leaf_dim)
    X = np.ascontiguousarray(rng.standard_normal((n, 12)).astype(np.float32))
    say("lanes layouts", strategy, n_trees, depth, leaf_dim, n)
    h = hb.compile(m, device=0)
    scores, ids = run(h, X, strategy, workspace=False)
    check(m, X, scores, ids, f"lanes T{n_trees} D{depth} ld{leaf_dim} n{n}/{strategy}")


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("used,leaf_dim,n", [(40, 1, 700), (40, 1, 20_000), (40, 1, 40_000), (40, 2, 9000),
                                             (120, 1, 30_000), (200, 1, 20_001)])
def test_pruned_wide_inputs(used, leaf_dim, n, strategy):
    """2000-column rows whose trees test 40 (or 200) columns: the kernels
    stage only those (gathered through the compiled column list), which puts
    these batches on the row-parallel fast kernel (128, 256 and 512 rows)
    instead of the wide-row path; small batches and vector leaves take the
    other kernels."""
    m = synth.narrow_use_model(2000, used, 64, 8, seed=41, leaf_dim=leaf_dim)
    X = synth.narrow_use_rows(2000, n, seed=41)
    say("pruned", strategy, used, leaf_dim, n)
    h = hb.compile(m, device=0)
    assert h.info()["n_used_features"] == used
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"pruned ld{leaf_dim} n{n}/{strategy}")


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("cfg,n", [(2, 1000), (2, 12_000), (2, 40_000), (3, 2000), (4, 3000), (4, 40_000),
                                   (5, 20_000)])
def test_missing_values_parity(cfg, n, strategy):
    """Per-node default directions for NaN (half the nodes send missing values
    left, 10% of the inputs missing) on every kernel path: tree-parallel,
    row-parallel fast shapes, general, GEMM."""
    model, _ = handle(cfg)
    m, X = synth.with_missing(model, synth.make_rows(cfg, n), seed=cfg + n)
    say("missing", cfg, n, strategy)
    h = hb.compile(m, device=0)
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"missing cfg{cfg}/{n}/{strategy}")


@pytest.mark.parametrize("strategy", STRATEGIES)
def test_hand_traced_default_left(strategy):
    trees, rows = pins.load_golden("hand_traced_default_left.txt")
    m = pins.model_from_trees(trees, 3)
    X = np.asarray([r[0] for r in rows], np.float32)
    say("hand-traced default-left", strategy)
    scores, ids = run(hb.compile(m, device=0), X, strategy)
    assert np.array_equal(ids, np.asarray([r[1] for r in rows], np.int32))
    assert np.allclose(scores[:, 0], [r[2] for r in rows], rtol=1e-6, atol=0)


@pytest.mark.parametrize("strategy", STRATEGIES)
def test_hand_traced_categorical(strategy):
    trees, rows = pins.load_golden("hand_traced_categorical.txt")
    m = pins.model_from_trees(trees, 3)
    X = np.asarray([r[0] for r in rows], np.float32)
    say("hand-traced categorical", strategy)
    scores, ids = run(hb.compile(m, device=0), X, strategy)
    assert np.array_equal(ids, np.asarray([r[1] for r in rows], np.int32))
    assert np.allclose(scores[:, 0], [r[2] for r in rows], rtol=1e-6, atol=0)


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("cfg,n", [(1, 1000), (2, 1000), (2, 12_000), (2, 40_000), (3, 2000), (3, 8000),
                                   (4, 3000), (5, 20_000)])
def test_categorical_parity(cfg, n, strategy):
    """Categorical nodes on four columns (40 categories: sets of two words,
    some with a third all-zero word; rows with fractional, negative, -0.0,
    +inf, out-of-range and missing values, nodes sending missing values
    left or right) on every kernel path: tree-parallel, split, row-parallel
    fast shapes, rows across lanes, general (the 7-class model's 66,000
    distinct sets exceed every feature tile), GEMM."""
    model, _ = handle(cfg)
    m, X = synth.with_categories(model, synth.make_rows(cfg, n), seed=cfg + n, cat_cols=[0, 3, 5, 7],
                                 n_categories=40)
    m, X = synth.with_missing(m, X, seed=cfg + n + 1, p_missing=0.03)
    say("categorical", cfg, n, strategy)
    h = hb.compile(m, device=0)
    if not h.info()["feasible"][strategy]:
        pytest.skip("strategy infeasible (too many indicator columns for TT's 16-bit feature ids)")
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"categorical cfg{cfg}/{n}/{strategy}")


@pytest.mark.parametrize("cfg,n,strategy,kernel", [
    (2, 40_000, "ptt", "fast_kernel<"), (2, 40_000, "tt", "fast_kernel<"), (2, 40_000, "gemm", "gemm_tile_kernel<"),
    (5, 20_000, "tt", "rows_kernel<"), (1, 20_000, "ptt", "fast_kernel<"), (2, 3000, "gemm", "gemm_tile_kernel<")])
def test_categorical_few_sets_on_the_fast_kernels(cfg, n, strategy, kernel):
    """Categorical nodes on one column of 4 categories (at most 16 distinct
    sets, so a few indicator columns): the row-parallel fast kernels (PTT
    with leaf values in global memory, TT with leaf records in global
    memory), the rows-across-lanes kernel and the GEMM tile kernel (with and
    without the tree split) stage the indicators in their LDS tiles."""
    model, _ = handle(cfg)
    m, X = synth.with_categories(model, synth.make_rows(cfg, n), seed=cfg + n, cat_cols=[1], n_categories=4)
    m, X = synth.with_missing(m, X, seed=cfg + n + 2, p_missing=0.03)
    h = hb.compile(m, device=0)
    assert h.info()["n_used_features"] <= 2 * model["n_features"] + 2 * 16  # plain and NaN-left columns, sets
    plan = [p["kernel"] for p in h.plan(n, strategy, hb.workspace_bytes(h, n, strategy))]
    say("categorical few sets", cfg, n, strategy, plan)
    assert plan[0].startswith(kernel), plan
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"categorical few sets cfg{cfg}/{n}/{strategy}")


def _band_model(F, K, ld, n_trees, seed, depth=8):
    """Perfect trees over F N(0,1) features: one output (K = 1), K classes
    with tree t in class t mod K (softmax), or vector leaves of ld class
    probabilities (ld > 1, averaged)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if ld > 1:
        def leaves(r, n):
            p = r.random((n, ld))
            return p / p.sum(1, keepdims=True)
    else:
        leaves = lambda r, n: r.normal(0, .05, n)
    m = synth.perfect_forest(rng, n_trees, depth, F, lambda r, f: r.normal(0, 1, f.size), leaves, leaf_dim=ld)
    m.update(n_outputs=max(K, ld), tree_class=(np.arange(n_trees) % K).astype(np.int32) if K > 1 else None,
             aggregation="mean" if ld > 1 else "sum", transform="softmax" if K > 1 else "sigmoid", base_score=None)
    return m


@pytest.mark.parametrize("F,K,ld,n_trees,n,kernel", [
    (54, 7, 1, 70, 65_536, "gemm_band_kernel<1, 8>"),     # the 7-class model's shape
    (60, 1, 1, 37, 49_153, "gemm_band_kernel<0, 1>"),     # ragged last band
    (60, 10, 1, 41, 52_000, "gemm_band_kernel<1, 16>"),
    (60, 1, 2, 33, 50_001, "gemm_band_kernel<2, 2>"),
    (48, 1, 1, 5, 49_152, "gemm_band_kernel<0, 1>"),      # fewer trees than waves
    (60, 1, 5, 23, 49_999, "gemm_band_kernel<2, 8>"),     # 5-vector leaves
    (60, 1, 10, 17, 50_113, "gemm_band_kernel<2, 16>"),   # 10-vector leaves
])
def test_gemm_band_kernel(F, K, ld, n_trees, n, kernel):
    """Batches of three 64-row bands per CU and more, with rows too wide for
    the 512-row pipelined kernel, take the band kernel: every row against the
    oracle, at ragged batch sizes, with one output, 7 or 10 classes and
    2-, 5- and 10-vector leaves (every instantiation of the kernel)."""
    m = _band_model(F, K, ld, n_trees, seed=F * 100 + n_trees)
    h = hb.compile(m, device=0)
    plan = [p["kernel"] for p in h.plan(n, "gemm")]
    say("gemm band", F, K, ld, n_trees, n, plan)
    assert plan == [kernel], plan
    X = np.random.Generator(np.random.PCG64(n)).normal(0, 1, (n, F)).astype(np.float32)
    scores, ids = run(h, X, "gemm", workspace=False)
    check(m, X, scores, ids, f"band F{F} K{K} ld{ld} T{n_trees} n{n}")


def test_gemm_band_kernel_with_column_list():
    """Missing values and categorical splits on the band kernel (its feature
    tile goes through the column list)."""
    m = _band_model(24, 1, 1, 64, seed=5)
    X = np.random.Generator(np.random.PCG64(6)).normal(0, 1, (50_000, 24)).astype(np.float32)
    m, X = synth.with_categories(m, X, seed=7, cat_cols=[2], n_categories=2)
    m, X = synth.with_missing(m, X, seed=8, p_missing=0.05)
    h = hb.compile(m, device=0)
    plan = [p["kernel"] for p in h.plan(50_000, "gemm")]
    say("gemm band with column list", plan, h.info()["n_used_features"])
    assert plan == ["gemm_band_kernel<0, 1>"], plan
    scores, ids = run(h, X, "gemm", workspace=False)
    check(m, X, scores, ids, "band with column list")


@pytest.mark.parametrize("strategy", STRATEGIES)
def test_empty_batch_enqueues_nothing(strategy):
    model, h = handle(1)
    say("empty", strategy)
    X = torch.empty((0, 8), dtype=torch.float32, device="cuda")
    s, ids = hb.predict(h, X, strategy=strategy)
    torch.cuda.synchronize()
    assert s.shape == (0, 1) and ids.shape == (0, 10)


@pytest.mark.parametrize("strategy", STRATEGIES)
@pytest.mark.parametrize("seed", range(4))
def test_tricky_ensembles(strategy, seed):
    """Unbalanced trees, permuted numbering, ties, NaN and +-inf inputs."""
    m = pins.random_small_ensemble(seed)
    X = pins.tricky_rows(np.random.Generator(np.random.PCG64(seed)), m, 700)
    say("tricky", strategy, seed)
    h = hb.compile(m, device=0)
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"tricky{seed}/{strategy}")


@pytest.mark.parametrize("strategy", STRATEGIES)
def test_permuted_numbering_and_mixed_aggregations(strategy):
    base = synth.make_model(3)
    m = synth.permute_nodes(base, 9)
    m["base_score"] = np.asarray([0.25, -0.5], np.float32)
    X = synth.make_rows(3, 700)
    say("permuted cfg3", strategy)
    h = hb.compile(m, device=0)
    scores, ids = run(h, X, strategy)
    check(m, X, scores, ids, f"perm/{strategy}")
    gb = synth.make_model(4)
    gb["transform"] = "sigmoid"
    gb["base_score"] = np.linspace(-1, 1, 7).astype(np.float32)
    X4 = synth.make_rows(4, 600)
    h4 = hb.compile(gb, device=0)
    scores, ids = run(h4, X4, strategy)
    check(gb, X4, scores, ids, f"sigmoid7/{strategy}")


@pytest.mark.parametrize("strategy", STRATEGIES)
def test_scores_only_and_determinism(strategy):
    model, h = handle(5)
    X = synth.make_rows(5, 4096)
    say("determinism", strategy)
    s1, i1 = run(h, X, strategy)
    s2, i2 = run(h, X, strategy)
    s3, i3 = run(h, X, strategy, leaves=False)
    assert i3 is None
    assert np.array_equal(i1, i2)
    assert np.array_equal(s1.view(np.uint32), s2.view(np.uint32))
    assert np.array_equal(s1.view(np.uint32), s3.view(np.uint32))


def test_strategies_agree_bitwise_on_leaf_ids():
    model, h = handle(4)
    X = synth.make_rows(4, 1500)
    say("cross-strategy cfg4")
    out = {s: run(h, X, s) for s in STRATEGIES}
    for s in STRATEGIES[1:]:
        assert np.array_equal(out[s][1], out["ptt"][1])


def test_non_default_stream():
    model, h = handle(2)
    X = synth.make_rows(2, 5000)
    say("side stream")
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        Xd = torch.from_numpy(X).to("cuda", non_blocking=False)
        s, ids = hb.predict(h, Xd, strategy="auto")
    st.synchronize()
    check(model, X, s.cpu().numpy(), ids.cpu().numpy(), "stream")


@pytest.mark.parametrize("strategy,n,use_ws", [("ptt", 100, False), ("ptt", 20_000, False), ("tt", 3000, False),
                                              ("gemm", 600, False), ("ptt", 2000, True), ("tt", 3000, True)])
def test_graph_capture_replays_match_eager(strategy, n, use_ws):
    """hb_predict (or hb_predict_ws with a workspace) captured into a HIP
    graph: every replay, with eager work and synchronisations between
    replays, equals the eager call bit for bit."""
    model, h = handle(2)
    say("graph capture", strategy, n, "workspace" if use_ws else "")
    X = torch.from_numpy(synth.make_rows(2, n)).cuda()
    s_ref, i_ref = hb.predict(h, X, strategy=strategy, workspace=use_ws)
    torch.cuda.synchronize()
    scores = torch.empty_like(s_ref)
    ids = torch.empty_like(i_ref)
    nws = hb.workspace_bytes(h, n, strategy) if use_ws else 0
    assert nws > 0 or not use_ws
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda")
    ws_ptr = ws.data_ptr() if nws else None
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):  # warm up on the capture stream
        hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), ids.data_ptr(), strategy, side.cuda_stream,
                       ws_ptr, nws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), ids.data_ptr(), strategy, side.cuda_stream,
                       ws_ptr, nws)
    for rep in range(4):
        scores.fill_(float("nan"))
        ids.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(scores.view(torch.int32), s_ref.view(torch.int32)), f"replay {rep} scores"
        assert torch.equal(ids, i_ref), f"replay {rep} leaf ids"
        junk = torch.randn(1 << 16, device="cuda").sum()  # eager work between replays
        del junk
    check(model, X.cpu().numpy(), scores.cpu().numpy(), ids.cpu().numpy(), f"graph/{strategy}/{n}")


@pytest.mark.parametrize("cfg", [2, 5])
def test_full_size_every_row(cfg):
    """A 1,000,000-row workload in the benchmark's launch configuration (AUTO,
    leaf ids, no workspace): every row's scores and leaf ids against the
    oracle, compared in 65,536-row chunks."""
    model, h = handle(cfg)
    n = 1_000_000
    X = synth.make_rows(cfg, n)
    say("full size every row", cfg, n)
    Xd = torch.from_numpy(X).cuda()
    s, ids = hb.predict(h, Xd, strategy="auto", workspace=False)
    torch.cuda.synchronize()
    worst = 0.0
    for lo in range(0, n, 65_536):
        hi = min(n, lo + 65_536)
        worst = max(worst, check(model, X[lo:hi], s[lo:hi].cpu().numpy(), ids[lo:hi].cpu().numpy(),
                                 f"cfg{cfg}-1M rows {lo}..{hi}"))
    say("worst score error / tolerance", worst)
    if cfg == 2:  # every score is a probability
        sc = s.cpu().numpy()
        assert np.all((sc >= 0) & (sc <= 1))


def test_full_size_wide_forest_every_row():
    """The 2000-feature random forest (workload 3) at its benchmark size,
    100,000 rows, in the benchmark's launch configuration (AUTO, leaf ids, no
    workspace: rows across lanes, 16 rows per workgroup): every row's class
    probabilities and leaf ids against the oracle."""
    model, h = handle(3)
    n = 100_000
    X = synth.make_rows(3, n)
    assert [p["kernel"] for p in h.plan(n, "auto")] == ["rows_kernel<true, 2, true, 16, true>"], h.plan(n, "auto")
    say("full size every row", 3, n)
    Xd = torch.from_numpy(X).cuda()
    s, ids = hb.predict(h, Xd, strategy="auto", workspace=False)
    torch.cuda.synchronize()
    for lo in range(0, n, 25_000):
        check(model, X[lo:lo + 25_000], s[lo:lo + 25_000].cpu().numpy(), ids[lo:lo + 25_000].cpu().numpy(),
              f"cfg3-100K rows {lo}..")


def _wide_model(kind, n_trees, depth, leafwise, seed):
    """Trees over 2000 features, too wide for the row-parallel tile: scalar
    leaves with one output, scalar leaves with two classes (tree t to class
    t mod 2), or 2-vector leaves averaged."""
    rng = np.random.Generator(np.random.PCG64(seed))
    F = 2000
    ld = 2 if kind == "vector" else 1
    thr = lambda r, f: r.uniform(-1.0, 1.0, f.size)
    leaves = (lambda r, n: np.stack([1 - r.random(n), r.random(n)], 1)) if ld == 2 else (lambda r, n: r.normal(0, .1, n))
    if leafwise:
        model = synth.leafwise_forest(rng, n_trees, 64, depth, 0.7, F, thr, lambda r, n: r.normal(0, .1, n))
        if ld == 2:  # probability pairs at the leaves
            p = np.random.Generator(np.random.PCG64(seed + 1)).random(model["feature"].size).astype(np.float32)
            model["leaf_value"] = np.stack([1 - p, p], 1).reshape(-1)
    else:
        model = synth.perfect_forest(rng, n_trees, depth, F, thr, leaves, leaf_dim=ld)
    model.update(n_outputs=2 if kind != "scalar" else 1, leaf_dim=ld,
                 tree_class=(np.arange(n_trees) % 2).astype(np.int32) if kind == "classes" else None,
                 aggregation="mean" if kind == "vector" else "sum",
                 transform="softmax" if kind == "classes" else "none", base_score=None)
    return model


@pytest.mark.parametrize("strategy", ["ptt", "tt"])
@pytest.mark.parametrize("kind,n_trees,depth,leafwise,n", [
    ("vector", 500, 8, False, 4096), ("vector", 37, 6, False, 4111), ("scalar", 61, 7, False, 4100),
    ("classes", 130, 5, False, 5003), ("scalar", 90, 10, True, 4099), ("vector", 41, 9, True, 4500)])
def test_rows_across_lanes(kind, n_trees, depth, leafwise, n, strategy):
    """Rows too wide for the row-parallel tile, at batches of a workgroup per
    CU or more, take rows_kernel (16 rows per workgroup, each wave walking
    four trees for all 16 rows): tree counts that do not fill a pass,
    ragged row tiles, scalar, two-class and vector leaves, perfect and
    leaf-wise trees, on PTT and TT, and leaf ids at an unaligned offset."""
    model = _wide_model(kind, n_trees, depth, leafwise, 900 + n_trees)
    h = hb.compile(model, device=0)
    if not h.info()["feasible"][strategy]:
        pytest.skip("strategy infeasible")
    kernels = [p["kernel"] for p in h.plan(n, strategy)]
    assert kernels[0].startswith("rows_kernel<"), kernels
    X = np.random.Generator(np.random.PCG64(n)).uniform(-1, 1, (n, 2000)).astype(np.float32)
    say("rows across lanes", kind, n_trees, depth, leafwise, n, strategy)
    scores, ids = run(h, X, strategy, workspace=False)
    check(model, X, scores, ids, f"rows {kind}/{n_trees}/{strategy}/{n}")
    # leaf ids one int past a 16-byte boundary: one int32 store per id
    Xd = torch.from_numpy(X).cuda()
    buf = torch.full((n * n_trees + 8,), -7, dtype=torch.int32, device="cuda")
    sc = torch.empty((n, model["n_outputs"]), dtype=torch.float32, device="cuda")
    hb.predict_ptr(h, Xd.data_ptr(), n, sc.data_ptr(), buf.data_ptr() + 4, strategy,
                   torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    b = buf.cpu().numpy()
    assert b[0] == -7 and np.all(b[1 + n * n_trees:] == -7)
    assert np.array_equal(b[1:1 + n * n_trees].reshape(n, n_trees), ids)
    h.close()


def test_full_size_multiclass_sampled():
    """The 7-class model at 1,000,000 rows (14 GB of leaf ids on the device):
    every output of a seeded sample of 40,000 rows, the first and last
    included, and every softmax row summing to one."""
    model, h = handle(4)
    n = 1_000_000
    X = synth.make_rows(4, n)
    say("full size cfg4 1M sampled")
    Xd = torch.from_numpy(X).cuda()
    s, ids = hb.predict(h, Xd, strategy="auto", workspace=False)
    torch.cuda.synchronize()
    rows = np.sort(np.random.Generator(np.random.PCG64(1)).choice(n, 40_000, replace=False))
    rows[0], rows[-1] = 0, n - 1
    rows_t = torch.from_numpy(rows).cuda()
    check(model, X[rows], s[rows_t].cpu().numpy(), ids[rows_t].cpu().numpy(), "cfg4-1M")
    tot = s.double().sum(dim=1).cpu().numpy()
    assert np.all(np.abs(tot - 1.0) < 1e-5)


def test_invalid_arguments_raise():
    model, h = handle(1)
    say("invalid args")
    with pytest.raises(hb.HBError):
        hb.predict_ptr(h, 0, 10, 0, None)
    with pytest.raises(hb.HBError):
        hb.predict_ptr(h, 1, -1, 1, None)
    with pytest.raises(hb.HBError):
        hb.predict_ptr(h, 1, 1, 1, None, strategy=7)


def _shape_model(kind, size, F, T, K, ld, seed, spread=1):
    """Perfect trees of depth `size` or leaf-wise trees of `size` leaves (depth
    <= 14) over F N(0,1) features, each feature index times `spread` (so that
    the input has F * spread columns); K > 1: tree t in class t mod K
    (softmax); ld > 1: probability vectors averaged."""
    rng = np.random.Generator(np.random.PCG64(seed))
    thr = lambda r, f: r.normal(0, 1, f.size)
    if ld > 1:
        def leaves(r, n):
            p = r.random((n, ld))
            return p / p.sum(1, keepdims=True)
    else:
        leaves = lambda r, n: r.normal(0, .05, n)
    if kind == "perfect":
        m = synth.perfect_forest(rng, T, size, F, thr, leaves, leaf_dim=ld)
    else:
        m = synth.leafwise_forest(rng, T, size, 14, 0.7, F, thr, lambda r, n: r.normal(0, .05, n))
        if ld > 1:
            m["leaf_value"] = leaves(np.random.Generator(np.random.PCG64(seed + 1)), m["feature"].size).reshape(-1)
            m["leaf_dim"] = ld
    if spread > 1:
        m["feature"] = np.where(m["feature"] >= 0, m["feature"] * spread, m["feature"]).astype(m["feature"].dtype)
        m["n_features"] = F * spread
    m.update(n_outputs=max(K, ld), tree_class=(np.arange(T) % K).astype(np.int32) if K > 1 else None,
             aggregation="mean" if ld > 1 else "sum", transform="softmax" if K > 1 or ld > 1 else "none",
             base_score=None)
    return m


@pytest.mark.parametrize("kind,size,F,spread,T,K,ld,n,strategy,expect", [
    # PTT deeper than the row-parallel kernels hold, at batches past the tree-parallel kernel
    ("perfect", 11, 28, 1, 24, 1, 1, 20_000, "ptt", "traverse_kernel<true, true, 1, false, false>"),
    ("perfect", 11, 28, 1, 24, 3, 1, 20_000, "ptt", "traverse_kernel<true, true, 8, false, false>"),
    ("perfect", 11, 28, 1, 24, 1, 2, 20_000, "ptt", "traverse_kernel<true, true, 2, true, false>"),
    # pruned inputs: the column list is applied while the feature tile is staged
    ("perfect", 11, 28, 3, 24, 1, 1, 20_001, "ptt", "traverse_kernel<true, true, 1, false, false>"),
    # TT trees of more than 2,048 nodes
    ("leafwise", 1500, 28, 1, 12, 1, 1, 20_000, "tt", "traverse_kernel<false, true, 1, false, false>"),
    ("leafwise", 1500, 28, 1, 12, 1, 3, 20_000, "tt", "traverse_kernel<false, true, 8, true, false>"),
    ("leafwise", 1500, 28, 3, 12, 2, 1, 20_001, "tt", "traverse_kernel<false, true, 2, false, false>"),
    # rows wider than LDS (over 40,960 staged features): features read from
    # global memory, whole or through the column list
    ("perfect", 12, 45_000, 1, 24, 1, 1, 300, "ptt", "traverse_kernel<true, false, 1, false, false>"),
    ("perfect", 12, 60_000, 1, 18, 1, 1, 301, "ptt", "traverse_kernel<true, false, 1, false, true>"),
    # more than about 2,300 used columns: 8 rows per workgroup instead of 16
    ("perfect", 6, 4000, 1, 120, 1, 1, 8_000, "ptt", "rows_kernel<true, 1, false, 8, false>"),
    ("perfect", 6, 4000, 1, 120, 1, 2, 8_001, "ptt", "rows_kernel<true, 2, true, 8, false>"),
    ("leafwise", 40, 4000, 1, 120, 2, 1, 8_002, "tt", "rows_kernel<false, 2, false, 8, false>"),
    # several outputs on the tree-parallel kernel, one and four rows per workgroup
    ("perfect", 7, 28, 1, 90, 2, 1, 700, "ptt", "lanes_kernel<true, 2, false, 1>"),
    ("perfect", 7, 28, 1, 90, 2, 1, 3000, "ptt", "lanes_kernel<true, 2, false, 4>"),
    ("leafwise", 60, 28, 1, 90, 5, 1, 3000, "tt", "lanes_kernel<false, 8, false, 4>"),
    ("leafwise", 60, 28, 1, 90, 12, 1, 3000, "tt", "lanes_kernel<false, 16, false, 1>"),
    ("perfect", 7, 28, 1, 90, 1, 12, 3000, "ptt", "lanes_kernel<true, 16, true, 1>"),
    ("leafwise", 60, 28, 1, 90, 1, 2, 3000, "tt", "lanes_kernel<false, 2, true, 4>"),
])
def test_general_and_wide_kernel_paths(kind, size, F, spread, T, K, ld, n, strategy, expect):
    """Kernels the workloads do not reach: the general traversal kernel (trees
    beyond the row-parallel kernels, rows wider than LDS), the
    rows-across-lanes kernel with 8 rows per workgroup, and the tree-parallel
    kernel with several outputs; each case asserts the launch plan and
    compares every row with the oracle."""
    m = _shape_model(kind, size, F, T, K, ld, seed=size * 1000 + F + T, spread=spread)
    h = hb.compile(m, device=0)
    assert h.info()["feasible"][strategy]
    plan = [p["kernel"] for p in h.plan(n, strategy)]
    say("kernel path", kind, size, F, spread, T, K, ld, n, strategy, plan)
    assert plan == [expect], plan
    X = np.random.Generator(np.random.PCG64(n + F)).normal(0, 1, (n, F * spread)).astype(np.float32)
    scores, ids = run(h, X, strategy, workspace=False)
    check(m, X, scores, ids, f"path {kind}{size} F{F}x{spread} T{T} K{K} ld{ld} n{n} {strategy}")


@pytest.mark.parametrize("K,permuted,n,expect", [
    (7, False, 20_003, "fast_kernel<3, 8, 16, "),
    (7, True, 20_003, "fast_kernel<0, 8, 16, "),
    (2, False, 20_003, "fast_kernel<3, 8, 2, "),
    (2, True, 20_003, "fast_kernel<0, 8, 2, "),
    # batches wide enough for 1024-row workgroups (root records in scalar registers)
    (2, False, 70_001, "fast_kernel<3, 8, 2, 1024, "),
    (2, True, 70_001, "fast_kernel<0, 8, 2, 1024, "),
])
def test_class_trees_on_both_ptt_layouts(K, permuted, n, expect):
    """One output column per tree class (softmax over K): heap-ordered perfect
    trees keep their leaf values apart and add each held value to its tree's
    column (mode 3); a permuted numbering keeps the leaf records in the
    blocks (mode 0). Every row is compared with the oracle, leaf ids and
    scores, at a batch past the tree-parallel kernel's range."""
    rng = np.random.Generator(np.random.PCG64(900 + K + 10 * permuted))
    T = 20 * K
    model = synth.perfect_forest(rng, T, 8, 28, lambda r, f: r.standard_normal(f.size),
                                 lambda r, n: r.normal(0.0, 0.05, n))
    model.update(n_outputs=K, tree_class=(np.arange(T) % K).astype(np.int32), aggregation="sum",
                 transform="softmax", base_score=None)
    if permuted:
        model = synth.permute_nodes(model, T)
    h = hb.compile(model, device=0)
    plan = [p["kernel"] for p in h.plan(n, "ptt")]
    say("class trees", K, "permuted" if permuted else "heap", n, plan)
    assert plan[0].startswith(expect), plan
    X = synth.make_rows(2, n)
    scores, ids = run(h, X, "ptt", workspace=False)
    check(model, X, scores, ids, f"class trees K={K} permuted={permuted}")

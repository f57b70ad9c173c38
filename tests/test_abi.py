"""The C-ABI library loads, exports every declared symbol, and reports errors
(CPU only: host-only handles, no compute calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2010_04804_amd as hb
from paper_2010_04804_amd import synth
import pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"^[\w \*]*?\b(hb_\w+)\s*\(", src, flags=re.M))
    return sorted(names)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(hb.LIB_PATH)
    names = declared_functions()
    assert {"hb_compile", "hb_predict", "hb_query", "hb_destroy", "hb_last_error",
            "hb_table", "hb_select_strategy"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_library_exports_only_the_c_abi():
    """Built with hidden visibility and a version script: the dynamic symbol
    table holds the declared hb_* functions and nothing else."""
    import subprocess

    out = subprocess.run(["nm", "-D", "--defined-only", hb.LIB_PATH], capture_output=True, text=True, check=True)
    syms = sorted(line.split()[-1] for line in out.stdout.splitlines() if line.strip())
    assert syms == declared_functions(), syms


def test_plan_needs_a_device_handle():
    h = hb.compile(synth.make_model(1), device=-1)
    with pytest.raises(hb.HBError) as e:
        h.plan(1000, "ptt")
    assert e.value.code == -1 and "host-only" in str(e.value)


def test_host_only_handle_cannot_predict():
    h = hb.compile(synth.make_model(1), device=-1)
    with pytest.raises(hb.HBError) as e:
        hb.predict_ptr(h, 1, 10, 1, None)
    assert e.value.code == -1 and "host-only" in str(e.value)


def test_query_fields():
    info = hb.compile(synth.make_model(2), device=-1).info()
    assert info["n_trees"] == 500 and info["max_depth"] == 8 and info["n_features"] == 28
    assert info["n_internal"] == 500 * 255 and info["n_leaves"] == 500 * 256
    assert info["feasible"] == {"auto": True, "gemm": True, "tt": True, "ptt": True}
    assert info["device"] == -1 and info["gemm_shapes"] == 1


def _expect(model, code, match, strategy="auto"):
    with pytest.raises(hb.HBError) as e:
        hb.compile(model, strategy=strategy, device=-1)
    assert e.value.code == code, str(e.value)
    assert re.search(match, str(e.value)), str(e.value)


def test_invalid_models_are_rejected():
    cyc = pins.model_from_trees([[(0, 0.5, 1, 1, 0), (0, 0.5, 0, 0, 0)]], 1)
    _expect(cyc, -2, "reached twice")
    out_of_range = pins.model_from_trees([[(0, 0.5, 1, 5, 0), (-1, 0, -1, -1, 1.0)]], 1)
    _expect(out_of_range, -2, "child out of range")
    unreachable = pins.model_from_trees([[(-1, 0, -1, -1, 1.0), (-1, 0, -1, -1, 2.0)]], 1)
    _expect(unreachable, -2, "unreachable")
    nan_thr = pins.model_from_trees([[(0, np.nan, 1, 2, 0), (-1, 0, -1, -1, 1), (-1, 0, -1, -1, 2)]], 1)
    _expect(nan_thr, -2, "NaN threshold")
    bad_feat = pins.model_from_trees([[(3, 0.5, 1, 2, 0), (-1, 0, -1, -1, 1), (-1, 0, -1, -1, 2)]], 2)
    _expect(bad_feat, -2, "feature out of range")
    bad_class = pins.model_from_trees([[(-1, 0, -1, -1, 1.0)]], 1, n_outputs=2, tree_class=[2])
    _expect(bad_class, -2, "tree_class")
    bad_ld = dict(pins.model_from_trees([[(-1, 0, -1, -1, 1.0)]], 1, n_outputs=3), leaf_dim=2)
    _expect(bad_ld, -1, "leaf_dim")
    too_many = dict(pins.model_from_trees([[(-1, 0, -1, -1, 1.0)]], 1), n_outputs=17)
    _expect(too_many, -1, "n_outputs")
    # rejected before any per-tree array is read
    too_many_trees = dict(pins.model_from_trees([[(-1, 0, -1, -1, 1.0)]], 1), n_trees=(1 << 24) + 1)
    _expect(too_many_trees, -1, "n_trees")


def test_forced_infeasible_strategy_is_unsupported():
    rng = np.random.Generator(np.random.PCG64(0))
    big = synth.perfect_forest(rng, 1, 9, 4, lambda r, f: r.random(f.size), lambda r, n: r.random(n))
    big.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
    _expect(big, -3, "infeasible", strategy="gemm")       # 512 leaves > 256
    deep = synth.leafwise_forest(rng, 1, 20, 19, 1.0, 4, lambda r, f: r.random(f.size),
                                 lambda r, n: r.random(n))
    deep.update(n_outputs=1, tree_class=None, aggregation="sum", transform="none", base_score=None)
    _expect(deep, -3, "infeasible", strategy="ptt")       # depth 19 > 12
    h = hb.compile(deep, device=-1)
    assert h.info()["feasible"]["ptt"] is False and h.select(10) == "tt"


def test_destroy_twice_via_close_is_safe():
    h = hb.compile(synth.make_model(1), device=-1)
    h.close()
    h.close()
    with pytest.raises(RuntimeError):
        h.info()


def test_default_left_validation():
    trees, rows = pins.load_golden("hand_traced_default_left.txt")
    m = pins.model_from_trees(trees, 3)
    hb.compile(m, device=-1).close()
    bad = dict(m, default_left=np.where(m["default_left"] > 0, 2, 0).astype(np.uint8))
    with pytest.raises(hb.HBError) as e:
        hb.compile(bad, device=-1)
    assert e.value.code == -2  # HB_ERR_INVALID_MODEL
    ninf = dict(m, threshold=m["threshold"].copy())
    ninf["threshold"][0] = -np.inf  # tree A's root sends missing values left
    with pytest.raises(hb.HBError) as e:
        hb.compile(ninf, device=-1)
    assert e.value.code == -3  # HB_ERR_UNSUPPORTED


def test_workspace_bytes_and_errors():
    lib = hb.load_library()
    h = hb.compile(synth.make_model(2), device=-1)  # 500 trees: 16 groups of 32
    assert hb.workspace_bytes(h, 1000, "ptt") == 16 * 1000 * 1 * 8
    assert hb.workspace_bytes(h, 65536, "tt") == 16 * 65536 * 8
    assert hb.workspace_bytes(h, 65537, "ptt") == 0  # large batches never split
    assert hb.workspace_bytes(h, 0, "ptt") == 0
    # GEMM splits its 16-row tiles in groups of 4 trees, up to 4,096 rows
    assert hb.workspace_bytes(h, 1000, "gemm") == 125 * 1000 * 8
    assert hb.workspace_bytes(h, 4097, "gemm") == 0
    assert lib.hb_workspace_bytes(h.ptr, -1, 0) == -1
    assert lib.hb_workspace_bytes(None, 10, 0) == -1
    assert lib.hb_workspace_bytes(h.ptr, 10, 9) == -1
    one = hb.compile(synth.make_model(1), device=-1)
    info = one.info()
    groups = (info["n_trees"] + 31) // 32
    want = groups * 100 * info["n_outputs"] * 8 if groups >= 2 else 0
    assert hb.workspace_bytes(one, 100, "tt") == want
    for ws, nbytes, match in [(None, 64, "needs a workspace"), (8, -1, "needs a workspace"),
                              (12, 64, "8-byte aligned")]:
        rc = lib.hb_predict_ws(h.ptr, 1, 10, 1, None, 0, None, ws, nbytes)
        assert rc == -1 and match in lib.hb_last_error().decode()
    # a valid workspace on a host-only handle reaches the device check
    assert lib.hb_predict_ws(h.ptr, 1, 10, 1, None, 0, None, 64, 64) == -1
    assert "host-only" in lib.hb_last_error().decode()


def test_scratch_entry_point_rejects_sizes_beyond_the_maximum():
    """hb_predict_scratch checks scratch_bytes before anything else (no GPU
    is touched): outside [0, HB_SCRATCH_BYTES] is an argument error; a
    host-only handle is rejected as by hb_predict."""
    h = hb.compile(synth.make_model(1), device=-1)
    for bad in (-1, hb.SCRATCH_BYTES + 1):
        with pytest.raises(hb.HBError) as e:
            hb.predict_scratch_ptr(h, 1, 10, 1, None, "ptt", None, bad)
        assert e.value.code == -1 and "HB_SCRATCH_BYTES" in str(e.value)
    with pytest.raises(hb.HBError) as e:
        hb.predict_scratch_ptr(h, 1, 10, 1, None, "ptt", None, 1024)
    assert e.value.code == -1 and "host-only" in str(e.value)
    src = open(os.path.join(ROOT, "include", "hb.h")).read()
    assert f"#define HB_SCRATCH_BYTES ((int64_t)32 << 20)" in src and hb.SCRATCH_BYTES == 32 << 20


def test_categorical_validation():
    trees, rows = pins.load_golden("hand_traced_categorical.txt")
    m = pins.model_from_trees(trees, 3)
    hb.compile(m, device=-1).close()
    # a categorical node's threshold is not read: NaN, or -inf with NaN left, are accepted
    thr = m["threshold"].copy()
    thr[0] = np.nan  # tree A's root, categorical, NaN left
    hb.compile(dict(m, threshold=thr), device=-1).close()
    thr[0] = -np.inf
    hb.compile(dict(m, threshold=thr), device=-1).close()
    co = m["cat_offset"]
    _expect(dict(m, cat_offset=co + 1), -2, r"cat_offset\[0\]")
    dec = co.copy()
    dec[2] = dec[1] - 1
    _expect(dict(m, cat_offset=dec), -2, "must not decrease")
    wide = co.copy()
    wide[1:] += 65536  # node 0 of tree A: 65,537 words
    _expect(dict(m, cat_offset=wide, cat_bits=np.zeros(int(wide[-1]), np.uint32)), -2, "category words")
    # an empty range everywhere is a numeric model
    h = hb.compile(dict(m, cat_offset=np.zeros_like(co), cat_bits=None), device=-1)
    h0 = hb.compile(dict(m, cat_offset=None, cat_bits=None), device=-1)
    for s in ("ptt", "tt", "gemm"):
        assert np.array_equal(h.table(s, "features", np.int32), h0.table(s, "features", np.int32))
        assert np.array_equal(h.table(s, "node", np.uint8), h0.table(s, "node", np.uint8))
    h.close()
    h0.close()

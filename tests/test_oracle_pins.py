"""The oracle against the pins in tests/pins.py (CPU only)."""
import numpy as np
import pytest

import oracle
from paper_2010_04804_amd import synth
import pins


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


def test_golden_hand_traced(lib):
    pins.pin_golden(lib)


def test_brute_force_paths(lib):
    pins.pin_brute_force(lib)


def test_gemm_closed_form_and_ptt_heap(lib):
    pins.pin_gemm_closed_form(lib)


def test_categorical_splits(lib):
    pins.pin_categorical(lib)


def test_closed_forms(lib):
    pins.pin_closed_forms(lib)


def test_sklearn_library_walk(lib):
    if not pins.pin_sklearn(lib):
        pytest.skip("scikit-learn not importable")


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_configs_one_leaf_per_tree_and_brute_force_sample(lib, cfg):
    """On every workload: each reported id is a leaf, and a sample of (row, tree)
    pairs agrees with brute-force path enumeration."""
    m = synth.make_model(cfg)
    X = synth.make_rows(cfg, 64)
    _, _, ids = oracle.predict(m, X, lib=lib)
    off = m["tree_node_offset"]
    T = m["n_trees"]
    nodes = off[:-1][None, :] + ids
    assert np.all(ids >= 0) and np.all(ids < (off[1:] - off[:-1])[None, :])
    assert np.all(m["feature"][nodes] < 0), "a reported id is not a leaf"
    rng = np.random.Generator(np.random.PCG64(cfg))
    for r, t in zip(rng.integers(0, 64, 40), rng.integers(0, T, 40)):
        assert ids[r, t] == pins.brute_force_leaf(m, int(t), X[r])


def test_thread_count_does_not_change_results(lib):
    m = synth.make_model(5)
    X = synth.make_rows(5, 257)
    a = oracle.predict(m, X, lib=lib, n_threads=1)
    b = oracle.predict(m, X, lib=lib, n_threads=7)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def test_permuted_numbering_reports_permuted_ids(lib):
    m = synth.make_model(5)
    p = synth.permute_nodes(m, 3)
    X = synth.make_rows(5, 100)
    r0, _, i0 = oracle.predict(m, X, lib=lib)
    r1, _, i1 = oracle.predict(p, X, lib=lib)
    want = np.stack([p["_perm"][t][i0[:, t]] for t in range(m["n_trees"])], axis=1)
    assert np.array_equal(i1, want)
    assert np.array_equal(r0, r1)


def test_ill_formed_trees_are_errors(lib):
    cyc = pins.model_from_trees([[(0, 0.5, 1, 1, 0), (0, 0.5, 0, 0, 0)]], 1)
    with pytest.raises(ValueError, match="cycle"):
        oracle.predict(cyc, np.zeros((1, 1), np.float32), lib=lib)
    bad = pins.model_from_trees([[(0, 0.5, 1, 5, 0), (-1, 0, -1, -1, 1.0)]], 1)
    with pytest.raises(ValueError, match="child"):
        oracle.predict(bad, np.ones((1, 1), np.float32), lib=lib)

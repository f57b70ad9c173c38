"""Test infrastructure only: the CPU oracle for batched tree-ensemble scoring.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package; the product library never does. The arithmetic lives in
``oracle.c`` (a plain node-by-node walk with double-precision aggregation, see
its header for the passages of the paper it follows); this module only builds
it with gcc, loads it and marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

AGG = {"sum": 0, "mean": 1}
POST = {"none": 0, "sigmoid": 1, "softmax": 2}
ERRORS = {-1: "invalid argument", -2: "cycle", -3: "child out of range", -4: "feature out of range"}

_lib = None


def build(out: str = _LIB, extra_flags=()) -> str:
    """Compile oracle.c with gcc into ``out`` (a shared library)."""
    cmd = ["gcc", "-O2", "-std=c99", "-D_POSIX_C_SOURCE=200809L", "-shared", "-fPIC",
           *extra_flags, "-o", out, _SRC, "-lpthread", "-lm"]
    subprocess.run(cmd, check=True)
    return out


def load(path: str = _LIB):
    """Load a built oracle library (building the default one if absent)."""
    global _lib
    if path == _LIB and _lib is not None:
        return _lib
    if not os.path.exists(path):
        if path != _LIB:
            raise FileNotFoundError(path)
        build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.oracle_predict.restype = ctypes.c_int
    lib.oracle_predict.argtypes = [i32, i32, i32, i32, P, P, P, P, P, P, P, i32, i32, P, P, P, P, P,
                                   i64, P, P, P, i32]
    if path == _LIB:
        _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def predict(model: dict, X: np.ndarray, leaves: bool = True, n_threads: int | None = None,
            lib=None):
    """Score ``X`` against ``model``.

    Returns ``(raw, scores, leaf_ids)``: float64 ``[n, K]`` aggregated margins
    before the transform, float64 ``[n, K]`` after it, and int32 ``[n, T]``
    caller-local leaf ids (``None`` when ``leaves`` is false).
    """
    lib = lib or load()
    X = np.ascontiguousarray(X, dtype=np.float32)
    n = X.shape[0]
    T, F, K = int(model["n_trees"]), int(model["n_features"]), int(model["n_outputs"])
    if X.ndim != 2 or X.shape[1] != F:
        raise ValueError(f"X must be [n, {F}]")
    arr = {
        "off": np.ascontiguousarray(model["tree_node_offset"], np.int64),
        "feature": np.ascontiguousarray(model["feature"], np.int32),
        "threshold": np.ascontiguousarray(model["threshold"], np.float32),
        "left": np.ascontiguousarray(model["left"], np.int32),
        "right": np.ascontiguousarray(model["right"], np.int32),
        "value": np.ascontiguousarray(model["leaf_value"], np.float32),
    }
    tc = model.get("tree_class")
    tc = None if tc is None else np.ascontiguousarray(tc, np.int32)
    bs = model.get("base_score")
    bs = None if bs is None else np.ascontiguousarray(bs, np.float32)
    dl = model.get("default_left")
    dl = None if dl is None else np.ascontiguousarray(dl, np.uint8)
    co = model.get("cat_offset")
    co = None if co is None else np.ascontiguousarray(co, np.int64)
    cb = model.get("cat_bits")
    cb = None if cb is None else np.ascontiguousarray(cb, np.uint32)
    if co is not None and (cb is None or cb.size == 0):
        cb = np.zeros(1, np.uint32)
    raw = np.empty((n, K), np.float64)
    out = np.empty((n, K), np.float64)
    ids = np.empty((n, T), np.int32) if leaves else None
    if n_threads is None:
        n_threads = os.cpu_count() or 1
    rc = lib.oracle_predict(T, F, K, int(model["leaf_dim"]), _ptr(arr["off"]), _ptr(arr["feature"]),
                            _ptr(arr["threshold"]), _ptr(arr["left"]), _ptr(arr["right"]),
                            _ptr(arr["value"]), _ptr(tc), AGG[model["aggregation"]],
                            POST[model["transform"]], _ptr(bs), _ptr(dl), _ptr(co), _ptr(cb), _ptr(X), n,
                            _ptr(raw), _ptr(out),
                            _ptr(ids), int(n_threads))
    if rc != 0:
        raise ValueError(f"oracle: {ERRORS.get(rc, rc)}")
    return raw, out, ids

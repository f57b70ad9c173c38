"""Batched tree-ensemble inference on MI355X: Python binding of libhb.

This module only marshals arguments into the C-ABI declared in
``include/hb.h`` (``hb_compile``, ``hb_predict``, ``hb_predict_ws``,
``hb_predict_scratch``, ``hb_workspace_bytes``, ``hb_query``, ``hb_table``, ``hb_select_strategy``,
``hb_plan``, ``hb_destroy``, ``hb_last_error``). Every step of
scoring runs in the library's HIP kernels; PyTorch only supplies device
memory and the current stream. If ``libhb.so`` has not been built, importing
works but every call raises.

Models are dicts in the caller form described in :mod:`.synth`.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = ["compile", "predict", "predict_ptr", "predict_scratch_ptr", "workspace_bytes", "SCRATCH_BYTES", "Handle", "HBError", "STRATEGY", "load_library",
           "LIB_PATH"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhb.so")

STRATEGY = {"auto": 0, "gemm": 1, "tt": 2, "ptt": 3}
STRATEGY_NAME = {v: k for k, v in STRATEGY.items()}
AGG = {"sum": 0, "mean": 1}
POST = {"none": 0, "sigmoid": 1, "softmax": 2}
ERR = {-1: "INVALID_ARG", -2: "INVALID_MODEL", -3: "UNSUPPORTED", -4: "OOM", -5: "HIP"}

_P = ctypes.c_void_p


class hb_ensemble_desc(ctypes.Structure):
    _fields_ = [
        ("n_trees", ctypes.c_int32), ("n_features", ctypes.c_int32),
        ("n_outputs", ctypes.c_int32), ("leaf_dim", ctypes.c_int32),
        ("tree_node_offset", _P), ("feature", _P), ("threshold", _P), ("left", _P),
        ("right", _P), ("leaf_value", _P), ("tree_class", _P),
        ("aggregation", ctypes.c_int32), ("transform", ctypes.c_int32), ("base_score", _P),
        ("default_left", _P), ("cat_offset", _P), ("cat_bits", _P),
    ]


class hb_info(ctypes.Structure):
    _fields_ = [
        ("n_trees", ctypes.c_int32), ("n_features", ctypes.c_int32),
        ("n_outputs", ctypes.c_int32), ("leaf_dim", ctypes.c_int32),
        ("max_depth", ctypes.c_int32), ("device", ctypes.c_int32),
        ("n_nodes", ctypes.c_int64), ("n_internal", ctypes.c_int64), ("n_leaves", ctypes.c_int64),
        ("balance", ctypes.c_double), ("default_strategy", ctypes.c_int32),
        ("feasible", ctypes.c_int32 * 4), ("table_bytes", ctypes.c_int64 * 4),
        ("gemm_shapes", ctypes.c_int32), ("ptt_depth", ctypes.c_int32),
        ("n_used_features", ctypes.c_int32),
    ]


class HBError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"hb error {code} ({ERR.get(code, '?')}): {msg}")
        self.code = code


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libhb.so; raises if it is missing (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run __graft_entry__.build() "
                           "(or python -m paper_2010_04804_amd.build)")
    lib = ctypes.CDLL(path)
    lib.hb_compile.restype = ctypes.c_int
    lib.hb_compile.argtypes = [ctypes.POINTER(hb_ensemble_desc), ctypes.c_int, ctypes.c_int,
                               ctypes.POINTER(_P)]
    lib.hb_predict.restype = ctypes.c_int
    lib.hb_predict.argtypes = [_P, _P, ctypes.c_int64, _P, _P, ctypes.c_int, _P]
    lib.hb_predict_ws.restype = ctypes.c_int
    lib.hb_predict_ws.argtypes = [_P, _P, ctypes.c_int64, _P, _P, ctypes.c_int, _P, _P, ctypes.c_int64]
    lib.hb_predict_scratch.restype = ctypes.c_int
    lib.hb_predict_scratch.argtypes = [_P, _P, ctypes.c_int64, _P, _P, ctypes.c_int, _P, ctypes.c_int64]
    lib.hb_workspace_bytes.restype = ctypes.c_int64
    lib.hb_workspace_bytes.argtypes = [_P, ctypes.c_int64, ctypes.c_int]
    lib.hb_select_strategy.restype = ctypes.c_int
    lib.hb_select_strategy.argtypes = [_P, ctypes.c_int64]
    lib.hb_query.restype = ctypes.c_int
    lib.hb_query.argtypes = [_P, ctypes.POINTER(hb_info)]
    lib.hb_table.restype = ctypes.c_int
    lib.hb_table.argtypes = [_P, ctypes.c_int, ctypes.c_char_p, ctypes.POINTER(_P),
                             ctypes.POINTER(ctypes.c_int64)]
    lib.hb_plan.restype = ctypes.c_int
    lib.hb_plan.argtypes = [_P, ctypes.c_int64, ctypes.c_int, ctypes.c_int64, ctypes.c_char_p, ctypes.c_int64]
    lib.hb_destroy.restype = None
    lib.hb_destroy.argtypes = [_P]
    lib.hb_last_error.restype = ctypes.c_char_p
    lib.hb_last_error.argtypes = []
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        raise HBError(rc, load_library().hb_last_error().decode())
    return rc


def _strategy(s) -> int:
    return STRATEGY[s] if isinstance(s, str) else int(s)


class Handle:
    """A compiled ensemble (owns the library handle)."""

    def __init__(self, ptr: int, device: int):
        self._ptr = ptr
        self.device = device

    @property
    def ptr(self):
        if not self._ptr:
            raise RuntimeError("handle already destroyed")
        return self._ptr

    def info(self) -> dict:
        inf = hb_info()
        _check(load_library().hb_query(self.ptr, ctypes.byref(inf)))
        out = {name: getattr(inf, name) for name, _ in hb_info._fields_}
        out["feasible"] = {STRATEGY_NAME[i]: bool(inf.feasible[i]) for i in range(4)}
        out["table_bytes"] = {STRATEGY_NAME[i]: int(inf.table_bytes[i]) for i in range(4)}
        return out

    def select(self, n_rows: int) -> str:
        rc = load_library().hb_select_strategy(self.ptr, int(n_rows))
        if rc < 0:
            _check(rc)
        return STRATEGY_NAME[rc]

    def plan(self, n_rows: int, strategy="auto", workspace_bytes: int = 0) -> list:
        """The kernels hb_predict_ws would launch for this batch (hb_plan):
        one dict per launch with the kernel's template name, grid, block and
        dynamic LDS bytes."""
        buf = ctypes.create_string_buffer(4096)
        _check(load_library().hb_plan(self.ptr, int(n_rows), _strategy(strategy), int(workspace_bytes), buf, 4096))
        out = []
        for part in filter(None, buf.value.decode().split("; ")):
            name, rest = part.split(" grid=(")
            grid, rest = rest.split(") block=")
            block, lds = rest.split(" lds=")
            out.append({"kernel": name, "grid": tuple(int(g) for g in grid.split(",")), "block": int(block),
                        "lds": int(lds)})
        return out

    def table(self, strategy, name: str, dtype) -> np.ndarray:
        """A copy of one compiled tensor (see hb_table in include/hb.h)."""
        data, nbytes = _P(), ctypes.c_int64()
        _check(load_library().hb_table(self.ptr, _strategy(strategy), name.encode(),
                                       ctypes.byref(data), ctypes.byref(nbytes)))
        buf = (ctypes.c_char * nbytes.value).from_address(data.value) if nbytes.value else b""
        return np.frombuffer(bytes(buf), dtype=dtype).copy()

    def close(self):
        if self._ptr:
            load_library().hb_destroy(self._ptr)
            self._ptr = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _arr(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def compile(model: dict, strategy="auto", device: int = 0) -> Handle:
    """Compile a caller-form model dict. ``device=-1`` builds a host-only handle."""
    lib = load_library()
    keep = {
        "off": _arr(model["tree_node_offset"], np.int64),
        "feature": _arr(model["feature"], np.int32),
        "threshold": _arr(model["threshold"], np.float32),
        "left": _arr(model["left"], np.int32),
        "right": _arr(model["right"], np.int32),
        "value": _arr(model["leaf_value"], np.float32),
        "tree_class": _arr(model.get("tree_class"), np.int32),
        "base": _arr(model.get("base_score"), np.float32),
        "default_left": _arr(model.get("default_left"), np.uint8),
        "cat_offset": _arr(model.get("cat_offset"), np.int64),
        "cat_bits": _arr(model.get("cat_bits"), np.uint32),
    }
    if keep["cat_offset"] is not None and (keep["cat_bits"] is None or keep["cat_bits"].size == 0):
        keep["cat_bits"] = np.zeros(1, np.uint32)

    def p(a):
        return None if a is None else a.ctypes.data

    d = hb_ensemble_desc(
        int(model["n_trees"]), int(model["n_features"]), int(model["n_outputs"]),
        int(model["leaf_dim"]), p(keep["off"]), p(keep["feature"]), p(keep["threshold"]),
        p(keep["left"]), p(keep["right"]), p(keep["value"]), p(keep["tree_class"]),
        AGG[model["aggregation"]], POST[model["transform"]], p(keep["base"]), p(keep["default_left"]),
        p(keep["cat_offset"]), p(keep["cat_bits"]))
    h = _P()
    _check(lib.hb_compile(ctypes.byref(d), _strategy(strategy), int(device), ctypes.byref(h)))
    return Handle(h.value, device)


def workspace_bytes(h: Handle, n_rows: int, strategy="auto") -> int:
    """Device workspace bytes that let a batch of ``n_rows`` split its trees."""
    v = load_library().hb_workspace_bytes(h.ptr, int(n_rows), _strategy(strategy))
    _check(int(v) if v < 0 else 0)
    return int(v)


def predict_ptr(h: Handle, x_ptr: int, n_rows: int, scores_ptr: int, ids_ptr: int | None,
                strategy="auto", stream: int | None = None, ws_ptr: int | None = None, ws_bytes: int = 0):
    """hb_predict (hb_predict_ws with a workspace) on raw device pointers
    (no allocation, no synchronisation)."""
    if ws_ptr:
        _check(load_library().hb_predict_ws(h.ptr, x_ptr, int(n_rows), scores_ptr, ids_ptr or None,
                                            _strategy(strategy), stream or None, ws_ptr, int(ws_bytes)))
    else:
        _check(load_library().hb_predict(h.ptr, x_ptr, int(n_rows), scores_ptr, ids_ptr or None,
                                         _strategy(strategy), stream or None))


SCRATCH_BYTES = 32 << 20  # HB_SCRATCH_BYTES of include/hb.h


def predict_scratch_ptr(h: Handle, x_ptr: int, n_rows: int, scores_ptr: int, ids_ptr: int | None,
                        strategy="auto", stream: int | None = None, scratch_bytes: int = 0):
    """hb_predict_scratch on raw device pointers: hb_predict_ws with the
    library's static device scratch (up to ``scratch_bytes`` of it) as the
    workspace; allocates nothing."""
    _check(load_library().hb_predict_scratch(h.ptr, x_ptr, int(n_rows), scores_ptr, ids_ptr or None,
                                             _strategy(strategy), stream or None, int(scratch_bytes)))


def predict(h: Handle, X, strategy="auto", leaves: bool = True, out=None, stream=None,
            workspace: bool = True):
    """Score a float32 CUDA tensor ``X`` [n, F].

    Returns ``(scores [n, K] float32, leaf_ids [n, T] int32 or None)`` as torch
    tensors on X's device, enqueued on ``stream`` (default: torch's current
    stream) without synchronising. With ``workspace`` (the default) a small
    batch gets a torch-allocated workspace so that its trees can be split
    across workgroups (hb_predict_ws); ``workspace=False`` calls hb_predict.
    """
    import torch

    if not (isinstance(X, torch.Tensor) and X.is_cuda and X.dtype == torch.float32):
        raise TypeError("X must be a float32 CUDA tensor")
    if X.dim() != 2:
        raise ValueError("X must be 2-D")
    X = X.contiguous()
    info = h.info()
    n = X.shape[0]
    if X.shape[1] != info["n_features"]:
        raise ValueError(f"X has {X.shape[1]} columns, model expects {info['n_features']}")
    if out is None:
        scores = torch.empty((n, info["n_outputs"]), dtype=torch.float32, device=X.device)
        ids = torch.empty((n, info["n_trees"]), dtype=torch.int32, device=X.device) if leaves else None
    else:
        scores, ids = out
        _check_out(scores, (n, info["n_outputs"]), torch.float32, X.device, "scores")
        if ids is not None:
            _check_out(ids, (n, info["n_trees"]), torch.int32, X.device, "leaf ids")
    current = torch.cuda.current_stream(X.device)
    ext = None
    if stream is None:
        stream = current.cuda_stream
    elif stream != current.cuda_stream:
        # X's copy and the output allocations were enqueued on the current
        # stream: the kernel on `stream` waits for them
        ext = torch.cuda.ExternalStream(stream, device=X.device)
        ext.wait_stream(current)
    nws = workspace_bytes(h, n, strategy) if workspace else 0
    ws = torch.empty(nws, dtype=torch.uint8, device=X.device) if nws else None
    predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), ids.data_ptr() if ids is not None else None,
                strategy, stream, ws.data_ptr() if ws is not None else None, nws)
    if ext is not None:
        # torch's allocator must not reuse these buffers before `stream` is done with them
        for t in (X, scores, ids, ws):
            if t is not None:
                t.record_stream(ext)
    return scores, ids


def _check_out(t, shape, dtype, device, what):
    """An out= buffer must be exactly what the kernels write: no bigger check
    is possible past this point, and a smaller buffer would be overrun."""
    import torch

    if not isinstance(t, torch.Tensor) or t.dtype != dtype or tuple(t.shape) != tuple(shape) \
            or t.device != device or not t.is_contiguous():
        raise ValueError(f"out {what} must be a contiguous {dtype} tensor of shape {tuple(shape)} on {device}")

"""CPU oracle for classification-tree evaluation: TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package.  The GPU library never calls it and shares no code with it.

The arithmetic lives in ``dtree_oracle.c`` (a plain serial walk, Section 3.1 problem
statement with the comparison ``x < t`` -> left).  This module compiles it with gcc and
wraps it with ctypes.  ``procedures.py`` holds models of the paper's Procedures 4 and 5
(pointer jumping over a ``path`` array), used as additional pins.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dtree_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ORACLE_NODE_DTYPE = np.dtype(
    [("feature", "<i4"), ("threshold", "<f4"), ("left", "<i4"), ("cls", "<i4")], align=False
)

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (IEEE comparisons: no fast-math, no FTZ)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fno-fast-math",
               "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp, _SRC]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        lib.oracle_tree_leaves.argtypes = [p, i32, i32, p, i64, i64, p]
        lib.oracle_tree_classes.argtypes = [p, i32, i32, p, i64, i64, p]
        lib.oracle_forest_classes.argtypes = [p, p, i32, i32, i32, p, i64, i64, p]
        for f in (lib.oracle_tree_leaves, lib.oracle_tree_classes, lib.oracle_forest_classes):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


class OracleError(RuntimeError):
    pass


def _nodes(nodes) -> np.ndarray:
    arr = np.ascontiguousarray(nodes)
    if arr.dtype != ORACLE_NODE_DTYPE:
        arr = np.ascontiguousarray(arr.astype(ORACLE_NODE_DTYPE))
    return arr


def _rows(x: np.ndarray, n_features: int):
    x = np.asarray(x)
    if x.dtype != np.float32 or x.ndim != 2:
        raise TypeError("features must be a 2-D float32 array")
    if x.strides[1] != 4 or x.strides[0] % 4 != 0:
        x = np.ascontiguousarray(x)
    ld = x.strides[0] // 4 if x.shape[0] > 1 else max(x.shape[1], n_features)
    if x.shape[1] < n_features:
        raise ValueError("fewer columns than the tree's feature count")
    return x, ld


def _fan_out(call, x: np.ndarray, ld: int, out: np.ndarray, threads: int, name: str):
    """Run ``call(x_ptr, n, ld, out_ptr)`` over contiguous row chunks on ``threads`` host
    threads (ctypes releases the GIL during the call).  threads == 1 is one serial call."""
    n = x.shape[0]
    bounds = np.linspace(0, n, max(1, min(threads, n)) + 1).astype(np.int64) if n else [0, 0]

    def part(k):
        lo, hi = int(bounds[k]), int(bounds[k + 1])
        return call(x.ctypes.data + lo * ld * 4, hi - lo, ld, out.ctypes.data + lo * 4)

    if len(bounds) <= 2:
        rcs = [part(0)]
    else:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(len(bounds) - 1) as pool:
            rcs = list(pool.map(part, range(len(bounds) - 1)))
    if any(rc != 0 for rc in rcs):
        raise OracleError("%s failed: %s" % (name, rcs))
    return out


def tree_leaves(nodes, x: np.ndarray, n_features: int, threads: int = 1) -> np.ndarray:
    """Index of the leaf each row reaches (int32[N])."""
    nd = _nodes(nodes)
    x, ld = _rows(x, n_features)
    out = np.empty(x.shape[0], dtype=np.int32)
    f = _load().oracle_tree_leaves
    return _fan_out(lambda xp, n, ld_, op: f(nd.ctypes.data, len(nd), n_features, xp, n, ld_, op),
                    x, ld, out, threads, "oracle_tree_leaves")


def tree_classes(nodes, x: np.ndarray, n_features: int, threads: int = 1) -> np.ndarray:
    """Class label of each row (int32[N])."""
    nd = _nodes(nodes)
    x, ld = _rows(x, n_features)
    out = np.empty(x.shape[0], dtype=np.int32)
    f = _load().oracle_tree_classes
    return _fan_out(lambda xp, n, ld_, op: f(nd.ctypes.data, len(nd), n_features, xp, n, ld_, op),
                    x, ld, out, threads, "oracle_tree_classes")


def forest_classes(nodes, offsets, x: np.ndarray, n_features: int, n_classes: int,
                   threads: int = 1) -> np.ndarray:
    """Majority-vote label of each row (int32[N]); ties go to the smallest class id."""
    nd = _nodes(nodes)
    off = np.ascontiguousarray(offsets, dtype=np.int32)
    x, ld = _rows(x, n_features)
    out = np.empty(x.shape[0], dtype=np.int32)
    f = _load().oracle_forest_classes
    return _fan_out(lambda xp, n, ld_, op: f(nd.ctypes.data, off.ctypes.data, len(off) - 1,
                                             n_features, n_classes, xp, n, ld_, op),
                    x, ld, out, threads, "oracle_forest_classes")

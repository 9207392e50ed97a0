"""Tree-structure helpers for the tests (parents, depths, root-to-leaf path conditions).

These read the breadth-first node array (Procedure 1 layout: right child = left + 1,
cls < 0 marks a decision node) and never evaluate a record by walking from the root, so
they can check walkers independently.
"""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def parents(nodes):
    """parent[i] and side[i] (0 = left child, 1 = right child); root has parent -1."""
    n = len(nodes)
    par = np.full(n, -1, dtype=np.int64)
    side = np.zeros(n, dtype=np.int64)
    for i in range(n):
        if nodes["cls"][i] < 0:
            l = int(nodes["left"][i])
            par[l], side[l] = i, 0
            par[l + 1], side[l + 1] = i, 1
    return par, side


def depths(nodes):
    par, _ = parents(nodes)
    d = np.zeros(len(nodes), dtype=np.int64)
    for i in range(1, len(nodes)):       # breadth-first: parent index < child index
        d[i] = d[par[i]] + 1
    return d


def leaf_conditions(nodes):
    """For every leaf, the list of (node, side) pairs on its root path."""
    par, side = parents(nodes)
    out = {}
    for i in np.nonzero(nodes["cls"] >= 0)[0]:
        conds = []
        v = int(i)
        while par[v] >= 0:
            conds.append((int(par[v]), int(side[v])))
            v = int(par[v])
        out[int(i)] = conds[::-1]
    return out


def satisfied(nodes, x, conds):
    """Boolean per row: every predicate on the path holds (left: x<t, right: not x<t)."""
    ok = np.ones(x.shape[0], dtype=bool)
    for node, s in conds:
        lt = x[:, nodes["feature"][node]] < nodes["threshold"][node]
        ok &= lt if s == 0 else ~lt
    return ok


def certificate(nodes, x, leaf):
    """Check, from the leaf upwards, that each row's leaf is consistent with its features.

    Returns a boolean per row.  O(depth) vectorised numpy per row.
    """
    par, side = parents(nodes)
    leaf = np.asarray(leaf, dtype=np.int64)
    ok = nodes["cls"][leaf] >= 0
    v = leaf.copy()
    rows = np.arange(x.shape[0])
    for _ in range(len(nodes)):
        p = par[v]
        live = p >= 0
        if not live.any():
            break
        pv = np.where(live, p, 0)
        lt = x[rows, nodes["feature"][pv]] < nodes["threshold"][pv]
        want_left = side[v] == 0
        ok &= ~live | (lt == want_left)
        v = np.where(live, p, v)
    return ok


def load_hand_trees():
    from paper_1111_1373_amd.workloads import NODE_DTYPE
    with open(os.path.join(GOLDEN, "hand_trees.json")) as fh:
        doc = json.load(fh)
    out = []
    for t in doc["trees"]:
        nodes = np.zeros(len(t["nodes"]), dtype=NODE_DTYPE)
        for i, n in enumerate(t["nodes"]):
            thr = float.fromhex(n["threshold"])
            assert np.isnan(thr) or float(np.float32(thr)) == thr
            nodes[i] = (n["feature"], np.float32(thr), n["left"], n["cls"])
        xs = np.array([[float.fromhex(v) for v in c["x"]] for c in t["cases"]], dtype=np.float64)
        x32 = xs.astype(np.float32)
        assert np.array_equal(np.isnan(xs), np.isnan(x32))
        assert np.array_equal(x32[~np.isnan(x32)].astype(np.float64), xs[~np.isnan(xs)])
        out.append(dict(name=t["name"], nodes=nodes, n_features=t["n_features"],
                        n_classes=t["n_classes"], x=x32,
                        leaf=np.array([c["leaf"] for c in t["cases"]], dtype=np.int32),
                        cls=np.array([c["cls"] for c in t["cases"]], dtype=np.int32)))
    return out


def special_pool():
    f32 = np.float32
    return np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, -1.0,
                     np.float32(np.ldexp(1.0, -149)), -np.float32(np.ldexp(1.0, -149)),
                     np.finfo(np.float32).max, -np.finfo(np.float32).max, 0.5], dtype=f32)


def boundary_values(nodes, feature):
    """Every threshold on ``feature``, its float neighbours, and the special values."""
    f32 = np.float32
    vals = list(special_pool())
    internal = nodes["cls"] < 0
    for t in nodes["threshold"][internal & (nodes["feature"] == feature)]:
        t = f32(t)
        with np.errstate(over="ignore"):
            vals += [t, np.nextafter(t, f32(np.inf)), np.nextafter(t, f32(-np.inf))]
    arr = np.array(vals, dtype=f32)
    # unique by bit pattern (keeps -0.0 and NaN)
    _, idx = np.unique(arr.view(np.uint32), return_index=True)
    return arr[np.sort(idx)]


def widen(xn: np.ndarray, x_type: str) -> np.ndarray:
    """Exact fp32 values of narrow records (the definition the GPU path must match):
    binary16 and uint8 by numpy's exact casts, bfloat16 bits by placing them in the upper
    half of a binary32."""
    if x_type in ("f16", "u8"):
        return xn.astype(np.float32)
    if x_type == "bf16":
        return (xn.astype(np.uint32) << np.uint32(16)).view(np.float32)
    raise ValueError(x_type)


def narrow_specials(x_type: str) -> np.ndarray:
    """Stored values that stress the widening: signed zeros, subnormals, extremes, infinities
    and NaN of each type (as the type's storage: float16, uint16 bits or uint8)."""
    if x_type == "f16":
        return np.array([0.0, -0.0, 2.0 ** -24, -(2.0 ** -24), 2.0 ** -14, 1023 * 2.0 ** -24,
                         65504.0, -65504.0, np.inf, -np.inf, np.nan, 1.0, 0.5, 0.099976],
                        dtype=np.float16)
    if x_type == "bf16":
        return np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x0080, 0x7F7F, 0xFF7F,
                         0x7F80, 0xFF80, 0x7FC0, 0x3F80, 0x3F00, 0x3DCD], dtype=np.uint16)
    if x_type == "u8":
        return np.array([0, 1, 2, 127, 128, 254, 255], dtype=np.uint8)
    raise ValueError(x_type)

"""Seeded synthetic workloads: trees in breadth-first node-array form and fp32 feature matrices.

This module only draws random numbers and lays them out; it evaluates nothing.  Both the
GPU path and the CPU oracle consume what it produces, so it must stay free of the
method's arithmetic (no comparisons of features against thresholds, no walks).

Node arrays follow the breadth-first encoding of Procedure 1 (Section 3.1): node ``i``
stores ``(feature, threshold, left, cls)``; the right child is ``left + 1``; ``cls = -1``
marks an internal (decision) node.  Features are 0-based (the paper counts from 1).

The five configurations C1..C5 are the evaluation workloads of this implementation (C0 is
the shape of the paper's own experiment, for context):

    C0  N=65,536     F=19  U[0,1)  15 decision nodes, depth 11 (the paper's shape), 7 classes

    C1  N=65,536     F=8   U[0,1)  complete depth-4 tree,  4 classes
    C2  N=262,144    F=16  U[0,1)  complete depth-8 tree,  8 classes (512x512 image)
    C3  N=2,073,600  F=32  N(0,1)  random tree, p_split=0.85, depth<=16, <=1,023 internal, 16 classes
    C4  N=16,777,216 F=64  U[0,1)  complete depth-12 tree, 32 classes
    C5  N=4,194,304  F=32  U[0,1)  forest of 32 complete depth-10 trees, 8 classes

C1 and C2 stand in for the paper's image-segmentation workload (Section 4.1), whose
records and trained tree are not available: they keep its shape (a 256x256 or 512x512
image of independent records) with synthetic i.i.d. features.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

NODE_DTYPE = np.dtype(
    [("feature", "<i4"), ("threshold", "<f4"), ("left", "<i4"), ("cls", "<i4")], align=False
)
assert NODE_DTYPE.itemsize == 16

SEED_BASE = 137300


@dataclasses.dataclass
class TreeWorkload:
    name: str
    nodes: np.ndarray          # NODE_DTYPE, one tree (or all trees concatenated for a forest)
    n_features: int
    n_classes: int
    n_samples: int
    feature_dist: str          # "uniform" or "normal"
    seed: int
    tree_offsets: Optional[np.ndarray] = None   # forest only: int32[n_trees + 1]

    @property
    def is_forest(self) -> bool:
        return self.tree_offsets is not None

    def features(self, n: Optional[int] = None, start: int = 0) -> np.ndarray:
        """Row-major fp32 matrix of ``n`` rows (default: all), rows ``start .. start+n``.

        Rows are generated in fixed blocks so that any slice is identical to the same rows
        of the full matrix.
        """
        n = self.n_samples - start if n is None else n
        return feature_rows(self.seed, self.n_features, self.feature_dist, start, n)


# ----------------------------------------------------------------------------------------
# random streams

def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    tree_ss, feat_ss = ss.spawn(2)
    return tree_ss, feat_ss


def uniform_f32(rng: np.random.Generator, shape) -> np.ndarray:
    """U[0,1) on the 24-bit grid k * 2**-24 (numpy's float32 generator)."""
    return rng.random(shape, dtype=np.float32)


def normal_f32(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(shape, dtype=np.float32)


_BLOCK_ROWS = 1 << 16


def feature_rows(seed: int, n_features: int, dist: str, start: int, n: int) -> np.ndarray:
    """Rows ``start .. start+n`` of the feature matrix of a workload.

    The matrix is produced in blocks of 65,536 rows, each from its own child seed, so a
    slice can be produced without generating the rows before it.
    """
    if n < 0 or start < 0:
        raise ValueError("negative row range")
    out = np.empty((n, n_features), dtype=np.float32)
    if n == 0:
        return out
    _, feat_ss = _streams(seed)
    b0 = start // _BLOCK_ROWS
    b1 = (start + n - 1) // _BLOCK_ROWS
    for b in range(b0, b1 + 1):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
            entropy=feat_ss.entropy, spawn_key=feat_ss.spawn_key + (b,))))
        if dist == "uniform":
            blk = uniform_f32(rng, (_BLOCK_ROWS, n_features))
        elif dist == "normal":
            blk = normal_f32(rng, (_BLOCK_ROWS, n_features))
        else:
            raise ValueError(dist)
        lo = max(start, b * _BLOCK_ROWS)
        hi = min(start + n, (b + 1) * _BLOCK_ROWS)
        out[lo - start:hi - start] = blk[lo - b * _BLOCK_ROWS:hi - b * _BLOCK_ROWS]
    return out


# ----------------------------------------------------------------------------------------
# trees

def complete_tree(rng: np.random.Generator, depth: int, n_features: int, n_classes: int,
                  threshold_dist: str = "uniform") -> np.ndarray:
    """Complete binary tree of the given depth in breadth-first (heap) order.

    Internal node i has children 2i+1 and 2i+2, which is exactly what Procedure 1 assigns
    to a complete tree.  Depth counts edges, so there are 2**depth - 1 internal nodes and
    2**depth leaves.
    """
    n_int = (1 << depth) - 1
    n_leaf = 1 << depth
    nodes = np.zeros(n_int + n_leaf, dtype=NODE_DTYPE)
    feats = rng.integers(0, n_features, size=n_int, dtype=np.int32)
    if threshold_dist == "uniform":
        thr = uniform_f32(rng, n_int)
    else:
        thr = normal_f32(rng, n_int)
    cls = rng.integers(0, n_classes, size=n_leaf, dtype=np.int32)
    idx = np.arange(n_int, dtype=np.int32)
    nodes["feature"][:n_int] = feats
    nodes["threshold"][:n_int] = thr
    nodes["left"][:n_int] = 2 * idx + 1
    nodes["cls"][:n_int] = -1
    nodes["feature"][n_int:] = 0
    nodes["threshold"][n_int:] = 0.0
    nodes["left"][n_int:] = -1
    nodes["cls"][n_int:] = cls
    return nodes


def grown_tree(rng: np.random.Generator, p_split: float, max_depth: int, max_internal: int,
               n_features: int, n_classes: int, threshold_dist: str = "normal") -> np.ndarray:
    """Random full binary tree grown breadth-first.

    Nodes are created in breadth-first order, so creation order is the Procedure 1 index.
    The root always splits; any other node at depth d splits iff d < max_depth, the
    internal-node cap is not yet reached, and a uniform draw is below ``p_split``.  Once
    the cap is reached every remaining frontier node becomes a leaf.  Per node the draws
    are: split uniform (float64), then feature and threshold (internal) or class (leaf).
    """
    feature: List[int] = []
    threshold: List[float] = []
    left: List[int] = []
    cls: List[int] = []
    depth_of: List[int] = [0]
    # node 0 exists; queue holds indices awaiting a decision
    queue = [0]
    n_created = 1
    n_internal = 0
    feature.append(0); threshold.append(0.0); left.append(-1); cls.append(-1)
    head = 0
    while head < len(queue):
        i = queue[head]; head += 1
        d = depth_of[i]
        u = rng.random()
        split = (i == 0 or u < p_split) and d < max_depth and n_internal < max_internal
        if split:
            n_internal += 1
            feature[i] = int(rng.integers(0, n_features))
            if threshold_dist == "normal":
                threshold[i] = float(normal_f32(rng, 1)[0])
            else:
                threshold[i] = float(uniform_f32(rng, 1)[0])
            left[i] = n_created
            cls[i] = -1
            for _ in range(2):
                feature.append(0); threshold.append(0.0); left.append(-1); cls.append(-1)
                depth_of.append(d + 1)
                queue.append(n_created)
                n_created += 1
        else:
            cls[i] = int(rng.integers(0, n_classes))
            left[i] = -1
    nodes = np.zeros(n_created, dtype=NODE_DTYPE)
    nodes["feature"] = feature
    nodes["threshold"] = np.asarray(threshold, dtype=np.float32)
    nodes["left"] = left
    nodes["cls"] = cls
    return nodes


def random_full_tree(rng: np.random.Generator, n_internal: int, n_features: int,
                     n_classes: int, threshold_values: Optional[np.ndarray] = None) -> np.ndarray:
    """Random full binary tree with exactly ``n_internal`` internal nodes (any shape).

    Shapes come from repeatedly splitting a uniformly chosen leaf; the result is then
    renumbered breadth-first as Procedure 1 does.  ``threshold_values``, if given, is the
    pool thresholds are drawn from (to force ties and special values in tests).
    """
    # build with explicit children first
    kids = {0: None}
    leaves = [0]
    nxt = 1
    for _ in range(n_internal):
        k = int(rng.integers(0, len(leaves)))
        v = leaves.pop(k)
        kids[v] = (nxt, nxt + 1)
        kids[nxt] = None
        kids[nxt + 1] = None
        leaves += [nxt, nxt + 1]
        nxt += 2
    # breadth-first renumbering (Procedure 1)
    order = []
    q = [0]
    h = 0
    while h < len(q):
        v = q[h]; h += 1
        order.append(v)
        if kids[v] is not None:
            q += list(kids[v])
    new_id = {v: i for i, v in enumerate(order)}
    nodes = np.zeros(len(order), dtype=NODE_DTYPE)
    for v in order:
        i = new_id[v]
        if kids[v] is None:
            nodes[i] = (0, 0.0, -1, int(rng.integers(0, n_classes)))
        else:
            if threshold_values is None:
                t = float(uniform_f32(rng, 1)[0])
            else:
                t = float(threshold_values[int(rng.integers(0, len(threshold_values)))])
            nodes[i] = (int(rng.integers(0, n_features)), t, new_id[kids[v][0]], -1)
    return nodes


def _bfs_nodes(kids, rng, n_features, n_classes, threshold_draw):
    order, q, h = [], [0], 0
    while h < len(q):
        v = q[h]; h += 1
        order.append(v)
        if kids[v] is not None:
            q += list(kids[v])
    new_id = {v: i for i, v in enumerate(order)}
    nodes = np.zeros(len(order), dtype=NODE_DTYPE)
    for v in order:
        i = new_id[v]
        if kids[v] is None:
            nodes[i] = (0, 0.0, -1, int(rng.integers(0, n_classes)))
        else:
            nodes[i] = (int(rng.integers(0, n_features)), threshold_draw(), new_id[kids[v][0]], -1)
    return nodes


def paper_shape_tree(rng: np.random.Generator, n_internal: int = 15, depth: int = 11,
                     n_features: int = 19, n_classes: int = 7,
                     spine_p: Optional[float] = None) -> np.ndarray:
    """Random full binary tree with the shape of the paper's experimental tree
    (Section 4.1: 31 nodes, 16 leaves, depth 11): a root-to-leaf spine of ``depth``
    decision nodes, whose turns are random, plus ``n_internal - depth`` splits of random
    leaves above the bottom level, so the depth stays ``depth``.  With ``spine_p`` the
    spine's thresholds are drawn so that about that fraction of U[0,1) records reaching a
    spine node follow the spine (otherwise every threshold is U[0,1))."""
    if n_internal < depth:
        raise ValueError("need at least `depth` decision nodes")
    kids = {0: None}
    dep = {0: 0}
    spine_right = {}
    nxt = 1
    v = 0
    for _ in range(depth):                       # the spine
        kids[v] = (nxt, nxt + 1)
        for c in (nxt, nxt + 1):
            kids[c] = None
            dep[c] = dep[v] + 1
        turn = int(rng.integers(0, 2))
        spine_right[v] = turn == 1
        v = nxt + turn
        nxt += 2
    for _ in range(n_internal - depth):          # side splits that keep the depth
        leaves = [u for u, k in kids.items() if k is None and dep[u] < depth - 1]
        u = leaves[int(rng.integers(0, len(leaves)))]
        kids[u] = (nxt, nxt + 1)
        for c in (nxt, nxt + 1):
            kids[c] = None
            dep[c] = dep[u] + 1
        nxt += 2
    if spine_p is None:
        return _bfs_nodes(kids, rng, n_features, n_classes,
                          lambda: float(uniform_f32(rng, 1)[0]))
    order, q, h = [], [0], 0
    while h < len(q):
        u = q[h]; h += 1
        order.append(u)
        if kids[u] is not None:
            q += list(kids[u])
    new_id = {u: i for i, u in enumerate(order)}
    nodes = np.zeros(len(order), dtype=NODE_DTYPE)
    for u in order:
        i = new_id[u]
        if kids[u] is None:
            nodes[i] = (0, 0.0, -1, int(rng.integers(0, n_classes)))
            continue
        t = float(uniform_f32(rng, 1)[0])
        if u in spine_right:
            w = t * (1.0 - spine_p)
            t = w if spine_right[u] else 1.0 - w
        nodes[i] = (int(rng.integers(0, n_features)), np.float32(t), new_id[kids[u][0]], -1)
    return nodes


def chain_tree(rng: np.random.Generator, n_internal: int, n_features: int, n_classes: int,
               p_exit: float = 0.05) -> np.ndarray:
    """Chain ("caterpillar") tree: every decision node has one leaf child and one decision
    child, the side of the leaf chosen at random, so the depth is ``n_internal``.  For
    U[0,1) features each node sends about ``p_exit`` of the records that reach it to its
    leaf: the threshold is drawn from [0, 2 p_exit) when the chain continues to the right
    and from [1 - 2 p_exit, 1) when it continues to the left."""
    kids = {0: None}
    v, nxt = 0, 1
    cont_right = {}
    for _ in range(n_internal):
        kids[v] = (nxt, nxt + 1)
        kids[nxt] = None
        kids[nxt + 1] = None
        right = bool(rng.integers(0, 2))
        cont_right[v] = right
        v = nxt + 1 if right else nxt
        nxt += 2
    order, q, h = [], [0], 0
    while h < len(q):
        u = q[h]; h += 1
        order.append(u)
        if kids[u] is not None:
            q += list(kids[u])
    new_id = {u: i for i, u in enumerate(order)}
    nodes = np.zeros(len(order), dtype=NODE_DTYPE)
    for u in order:
        i = new_id[u]
        if kids[u] is None:
            nodes[i] = (0, 0.0, -1, int(rng.integers(0, n_classes)))
        else:
            w = float(uniform_f32(rng, 1)[0]) * 2 * p_exit
            t = w if cont_right[u] else 1.0 - w
            nodes[i] = (int(rng.integers(0, n_features)), np.float32(t), new_id[kids[u][0]], -1)
    return nodes


def coherent_rows(seed: int, height: int, width: int, n_features: int) -> np.ndarray:
    """Image-like records: the pixels of a ``height`` x ``width`` raster in row-major
    order, each feature a smooth random field (a sum of four plane waves of 1 to 8 cycles
    across the image plus 2% pixel noise) mapped through the normal CDF, so that every
    feature is spread over [0, 1) while neighbouring pixels have close values."""
    from scipy.special import ndtr

    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    yy, xx = np.meshgrid(np.arange(height, dtype=np.float32) / height,
                         np.arange(width, dtype=np.float32) / width, indexing="ij")
    out = np.empty((height * width, n_features), dtype=np.float32)
    for f in range(n_features):
        g = np.zeros((height, width), dtype=np.float32)
        for _ in range(4):
            fx, fy = rng.uniform(1, 8, size=2) * rng.choice([-1, 1], size=2)
            ph = rng.uniform(0, 2 * np.pi)
            g += np.cos(np.float32(2 * np.pi) * (np.float32(fx) * xx + np.float32(fy) * yy) +
                        np.float32(ph))
        g = g / np.float32(np.sqrt(2.0)) + np.float32(0.02 * 2) * rng.standard_normal(
            g.shape, dtype=np.float32)
        out[:, f] = np.minimum(ndtr(g.reshape(-1)).astype(np.float32), np.float32(1 - 2 ** -24))
    return out


GEOMETRIES = ("complete10", "grown", "random1023", "paper15", "chain64")
ORDERS = ("iid", "coherent", "sorted")


def sweep_tree(geometry: str, n_features: int = 32, n_classes: int = 8) -> np.ndarray:
    """Tree of one geometry of the sweep over tree shapes and record arrangements (the
    further work of Section 6): a complete depth-10 tree; a breadth-first grown tree
    (p = 0.85, depth <= 16, <= 1,023 decision nodes); a random full tree of 1,023 decision
    nodes (random leaf splits); the paper's 15-node, depth-11 shape (about 80% of the
    records reaching a spine node follow the spine); a 64-deep chain."""
    seed = SEED_BASE + 100 + GEOMETRIES.index(geometry)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    F, C = n_features, n_classes
    if geometry == "complete10":
        return complete_tree(rng, 10, F, C)
    if geometry == "grown":
        return grown_tree(rng, 0.85, 16, 1023, F, C, "uniform")
    if geometry == "random1023":
        return random_full_tree(rng, 1023, F, C)
    if geometry == "paper15":
        return paper_shape_tree(rng, 15, 11, F, C, spine_p=0.8)
    if geometry == "chain64":
        return chain_tree(rng, 64, F, C)
    raise ValueError(geometry)


def sweep_rows(order: str, height: int = 2048, width: int = 2048, n_features: int = 32,
               sort_feature: int = 0) -> np.ndarray:
    """height x width records of one arrangement: i.i.d. U[0,1); image-like coherent
    fields (``coherent_rows``); or the i.i.d. records sorted by attribute
    ``sort_feature``."""
    n = height * width
    if order == "coherent":
        return coherent_rows(SEED_BASE + 200, height, width, n_features)
    x = feature_rows(SEED_BASE + 300, n_features, "uniform", 0, n)
    if order == "sorted":
        return np.ascontiguousarray(x[np.argsort(x[:, sort_feature], kind="stable")])
    if order != "iid":
        raise ValueError(order)
    return x


def sweep_case(geometry: str, order: str, height: int = 2048, width: int = 2048,
               n_features: int = 32, n_classes: int = 8):
    """(nodes, records) of one geometry x order case; "sorted" sorts by the root's
    attribute."""
    nodes = sweep_tree(geometry, n_features, n_classes)
    return nodes, sweep_rows(order, height, width, n_features, int(nodes["feature"][0]))


def config(k: int, n_samples: Optional[int] = None) -> TreeWorkload:
    """Workload C0..C5 (``k`` in 0..5).  ``n_samples`` may shrink the sample count.

    C0 is the shape of the paper's own experiment (Section 4.1: 65,536 records of 19
    attributes, a 31-node tree of depth 11, 7 classes), with synthetic records and tree."""
    seed = SEED_BASE + k
    tree_ss, _ = _streams(seed)
    rng = np.random.Generator(np.random.PCG64(tree_ss))
    if k == 0:
        w = TreeWorkload("C0", paper_shape_tree(rng, 15, 11, 19, 7, spine_p=0.8), 19, 7, 65_536,
                         "uniform", seed)
    elif k == 1:
        w = TreeWorkload("C1", complete_tree(rng, 4, 8, 4), 8, 4, 65_536, "uniform", seed)
    elif k == 2:
        w = TreeWorkload("C2", complete_tree(rng, 8, 16, 8), 16, 8, 262_144, "uniform", seed)
    elif k == 3:
        s = seed
        while True:
            nodes = grown_tree(rng, 0.85, 16, 1023, 32, 16, "normal")
            if int((nodes["cls"] < 0).sum()) >= 512:
                break
            s += 1
            rng = np.random.Generator(np.random.PCG64(_streams(s)[0]))
        w = TreeWorkload("C3", nodes, 32, 16, 2_073_600, "normal", seed)
    elif k == 4:
        w = TreeWorkload("C4", complete_tree(rng, 12, 64, 32), 64, 32, 16_777_216, "uniform", seed)
    elif k == 5:
        trees = []
        for t_ss in tree_ss.spawn(32):
            trng = np.random.Generator(np.random.PCG64(t_ss))
            trees.append(complete_tree(trng, 10, 32, 8))
        offsets = np.zeros(33, dtype=np.int32)
        offsets[1:] = np.cumsum([len(t) for t in trees])
        w = TreeWorkload("C5", np.concatenate(trees), 32, 8, 4_194_304, "uniform", seed,
                         tree_offsets=offsets)
    else:
        raise ValueError("config index must be 0..5")
    if n_samples is not None:
        w.n_samples = int(n_samples)
    return w


# ----------------------------------------------------------------------------------------
# narrower record types

NARROW_TYPES = ("f16", "bf16", "u8")


def _u8_affine(dist: str):
    """(scale, offset) of the 8-bit quantisation q = clip(floor(scale * x + offset), 0, 255)."""
    return (256.0, 0.0) if dist == "uniform" else (32.0, 128.0)


def narrow_records(x: np.ndarray, x_type: str, dist: str = "uniform") -> np.ndarray:
    """The fp32 records ``x`` stored as ``x_type``.

    f16: IEEE binary16, round to nearest even (numpy's cast).  bf16: the upper half of the
    binary32 after round to nearest even, as uint16 bit patterns (inputs must not be NaN).
    u8: the 8-bit quantisation of ``_u8_affine(dist)`` (ordered discrete values 0..255).
    """
    if x_type == "f16":
        with np.errstate(over="ignore"):     # beyond 65504 rounds to infinity
            return x.astype(np.float16)
    if x_type == "bf16":
        bits = x.view(np.uint32)
        rounded = bits + np.uint32(0x7FFF) + ((bits >> np.uint32(16)) & np.uint32(1))
        return (rounded >> np.uint32(16)).astype(np.uint16)
    if x_type == "u8":
        a, b = _u8_affine(dist)
        return np.clip(np.floor(x * np.float32(a) + np.float32(b)), 0, 255).astype(np.uint8)
    raise ValueError(x_type)


def narrow_tree(nodes: np.ndarray, x_type: str, dist: str = "uniform") -> np.ndarray:
    """A tree for records of ``x_type``: for u8 the thresholds are mapped by the same affine
    quantisation as the records (so the splits fall on the 8-bit grid's scale); for the
    floating-point types the tree is unchanged."""
    if x_type != "u8":
        return nodes
    a, b = _u8_affine(dist)
    out = nodes.copy()
    internal = out["cls"] < 0
    out["threshold"][internal] = (out["threshold"][internal] * np.float32(a) +
                                  np.float32(b)).astype(np.float32)
    return out


CONFIG_DESCRIPTIONS = {
    0: "C0: N=65,536 x F=19 fp32 U[0,1); the paper's tree shape (15 internal, depth 11), 7 classes",
    1: "C1: N=65,536 x F=8 fp32 U[0,1); complete depth-4 tree (15 internal), 4 classes",
    2: "C2: N=262,144 (512x512) x F=16 fp32 U[0,1); complete depth-8 tree (255 internal), 8 classes",
    3: "C3: N=2,073,600 (1920x1080) x F=32 fp32 N(0,1); random tree p=0.85, depth<=16, <=1,023 internal, 16 classes",
    4: "C4: N=16,777,216 x F=64 fp32 U[0,1); complete depth-12 tree (4,095 internal), 32 classes",
    5: "C5: N=4,194,304 x F=32 fp32 U[0,1); forest of 32 complete depth-10 trees, 8 classes, majority vote",
}

"""Pins of the CPU oracle against truths other than itself (CPU only).

Each test fixes the oracle to something the paper or mathematics determines: hand-worked
trees, brute force over leaf regions, a textbook search routine, a library tree
evaluator, the partition property, closed forms, and the paper's own speculative
procedures (Sections 3.3 and 3.4) modelled step by step.
"""
import numpy as np
import pytest

import oracle
from oracle import procedures
from paper_1111_1373_amd import workloads as W
from tests import treeutil as TU


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ---------------------------------------------------------------- hand-worked trees

@pytest.mark.parametrize("tree", TU.load_hand_trees(), ids=lambda t: t["name"])
def test_hand_worked_trees(tree):
    leaf = oracle.tree_leaves(tree["nodes"], tree["x"], tree["n_features"])
    cls = oracle.tree_classes(tree["nodes"], tree["x"], tree["n_features"])
    np.testing.assert_array_equal(leaf, tree["leaf"])
    np.testing.assert_array_equal(cls, tree["cls"])


def test_hand_fixture_is_consistent():
    # the fixture's expected classes are the classes of its expected leaves
    for t in TU.load_hand_trees():
        np.testing.assert_array_equal(t["nodes"]["cls"][t["leaf"]], t["cls"])


# ---------------------------------------------------------------- brute force

def _brute_force_leaf(nodes, x):
    conds = TU.leaf_conditions(nodes)
    hits = np.zeros(x.shape[0], dtype=np.int64)
    which = np.full(x.shape[0], -1, dtype=np.int64)
    for leaf, c in conds.items():
        ok = TU.satisfied(nodes, x, c)
        hits += ok
        which[ok] = leaf
    return hits, which


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_exhaustive_boundaries(seed):
    """Exactly one leaf's path conjunction holds, and it is the oracle's leaf, over the
    full Cartesian product of every feature's boundary values."""
    r = rng(1000 + seed)
    n_int = int(r.integers(1, 8))
    F = int(r.integers(1, 3))
    pool = np.concatenate([TU.special_pool(), W.uniform_f32(r, 4)])
    pool = pool[~np.isneginf(pool)]
    nodes = W.random_full_tree(r, n_int, F, 5, threshold_values=pool)
    axes = [TU.boundary_values(nodes, f) for f in range(F)]
    grid = np.stack(np.meshgrid(*axes, indexing="ij"), axis=-1).reshape(-1, F)
    hits, which = _brute_force_leaf(nodes, grid)
    assert (hits == 1).all()
    np.testing.assert_array_equal(oracle.tree_leaves(nodes, grid, F), which)


@pytest.mark.parametrize("seed", range(8))
def test_brute_force_random_trees(seed):
    r = rng(2000 + seed)
    n_int = int(r.integers(1, 16))
    F = int(r.integers(1, 4))
    nodes = W.random_full_tree(r, n_int, F, 7)
    x = W.uniform_f32(r, (4000, F))
    # plant exact ties with thresholds and special values
    internal = np.nonzero(nodes["cls"] < 0)[0]
    for k in range(0, 4000, 7):
        i = internal[k % len(internal)]
        x[k, nodes["feature"][i]] = nodes["threshold"][i]
    sp = TU.special_pool()
    for k in range(3, 4000, 11):
        x[k, k % F] = sp[k % len(sp)]
    hits, which = _brute_force_leaf(nodes, x)
    assert (hits == 1).all()
    np.testing.assert_array_equal(oracle.tree_leaves(nodes, x, F), which)


# ---------------------------------------------------------------- textbook / library

def _bst(sorted_t, depth):
    """Complete BST of the given depth over sorted thresholds (in-order), breadth-first
    (heap) layout, single feature; leaf class = in-order leaf rank."""
    n_int = (1 << depth) - 1
    nodes = np.zeros(2 * n_int + 1, dtype=W.NODE_DTYPE)
    counter = {"t": 0, "leaf": 0}

    def inorder(h, d):
        if d == depth:
            nodes[h] = (0, 0.0, -1, counter["leaf"]); counter["leaf"] += 1
            return
        inorder(2 * h + 1, d + 1)
        nodes[h] = (0, sorted_t[counter["t"]], 2 * h + 1, -1); counter["t"] += 1
        inorder(2 * h + 2, d + 1)

    inorder(0, 0)
    return nodes


@pytest.mark.parametrize("depth", [1, 3, 6])
def test_bst_equals_searchsorted_right(depth):
    """Single-feature BST: in-order leaf rank == #thresholds <= x (upper bound).  Pins the
    comparison direction (ties go right) and the right = left + 1 layout."""
    r = rng(3000 + depth)
    n_int = (1 << depth) - 1
    t = np.sort(np.unique(W.uniform_f32(r, 4 * n_int)))[:n_int]
    if depth == 6:
        t[-1] = np.inf          # +inf threshold: only x=+inf/NaN pass it
        t[0] = -0.0
        t = np.sort(t)
    nodes = _bst(t, depth)
    x = np.concatenate([W.uniform_f32(r, 2000), t, np.nextafter(t, np.float32(np.inf)),
                        np.nextafter(t, np.float32(-np.inf)), TU.special_pool()]).astype(np.float32)
    got = oracle.tree_classes(nodes, x[:, None], 1)
    want = np.searchsorted(t, x, side="right")
    np.testing.assert_array_equal(got, want)


def _to_sklearn(nodes, n_features):
    from sklearn.tree._tree import NODE_DTYPE as SK, Tree
    n = len(nodes)
    sk = np.zeros(n, dtype=SK)
    internal = nodes["cls"] < 0
    sk["left_child"] = np.where(internal, nodes["left"], -1)
    sk["right_child"] = np.where(internal, nodes["left"] + 1, -1)
    sk["feature"] = np.where(internal, nodes["feature"], -2)
    # sklearn sends x <= thr left; x < t (fp32 x) == x <= the double just below t
    thr = np.nextafter(nodes["threshold"].astype(np.float64), -np.inf)
    sk["threshold"] = np.where(internal, thr, -2.0)
    sk["missing_go_to_left"] = 0            # NaN goes right, as NaN < t is false
    sk["n_node_samples"] = 1
    sk["weighted_n_node_samples"] = 1.0
    tree = Tree(n_features, np.array([1], dtype=np.intp), 1)
    depth = int(TU.depths(nodes).max())
    tree.__setstate__({"max_depth": depth, "node_count": n, "nodes": sk,
                       "values": np.zeros((n, 1, 1))})
    return tree


@pytest.mark.parametrize("seed", range(6))
def test_matches_sklearn_tree_apply(seed):
    """scikit-learn's tree evaluator (an independent implementation) on random trees."""
    r = rng(4000 + seed)
    F = int(r.integers(1, 9))
    pool = np.concatenate([TU.special_pool(), W.uniform_f32(r, 64)])
    pool = pool[~np.isneginf(pool)]     # no double lies below -inf for sklearn's <=
    nodes = W.random_full_tree(r, int(r.integers(1, 200)), F, 9, threshold_values=pool)
    x = W.uniform_f32(r, (20000, F))
    x[r.random(x.shape) < 0.05] = pool[r.integers(0, len(pool), size=1)[0]]
    m = r.random(x.shape) < 0.05
    x[m] = pool[r.integers(0, len(pool), size=int(m.sum()))]
    sk = _to_sklearn(nodes, F)
    np.testing.assert_array_equal(oracle.tree_leaves(nodes, x, F), sk.apply(x))


# ---------------------------------------------------------------- closed forms

def test_stump_closed_form():
    r = rng(5)
    nodes = np.zeros(3, dtype=W.NODE_DTYPE)
    nodes[0] = (1, np.float32(0.375), 1, -1)
    nodes[1] = (0, 0.0, -1, 4)
    nodes[2] = (0, 0.0, -1, 9)
    x = W.uniform_f32(r, (5000, 2))
    x[::13, 1] = np.float32(0.375)
    x[::17, 1] = np.nan
    want = np.where(x[:, 1] < np.float32(0.375), 4, 9)
    np.testing.assert_array_equal(oracle.tree_classes(nodes, x, 2), want)


@pytest.mark.parametrize("depth", [1, 4, 9])
def test_complete_tree_heap_formula(depth):
    """Complete tree in heap order: leaf = 2^D - 1 + sum_k b_k 2^(D-1-k), where b_k is the
    branch bit taken at level k (computed level by level with heap arithmetic, not the
    stored child pointers)."""
    r = rng(6000 + depth)
    F = 5
    nodes = W.complete_tree(r, depth, F, 3)
    x = W.uniform_f32(r, (20000, F))
    h = np.zeros(x.shape[0], dtype=np.int64)
    acc = np.zeros(x.shape[0], dtype=np.int64)
    rows = np.arange(x.shape[0])
    for k in range(depth):
        b = ~(x[rows, nodes["feature"][h]] < nodes["threshold"][h])
        acc += b.astype(np.int64) << (depth - 1 - k)
        h = 2 * h + 1 + b
    np.testing.assert_array_equal(oracle.tree_leaves(nodes, x, F), (1 << depth) - 1 + acc)


# ---------------------------------------------------------------- partition invariant

@pytest.mark.parametrize("k", [1, 2, 3])
def test_partition_invariant_configs(k):
    """Every record lands in exactly one leaf, and the leaf's path predicates hold
    (checked from the leaf upwards)."""
    w = W.config(k, n_samples={1: 65536, 2: 65536, 3: 65536}[k])
    x = w.features()
    leaf = oracle.tree_leaves(w.nodes, x, w.n_features)
    assert TU.certificate(w.nodes, x, leaf).all()
    assert np.bincount(leaf, minlength=len(w.nodes)).sum() == x.shape[0]
    if k in (1, 2):
        hits, which = _brute_force_leaf(w.nodes, x[:8192])
        assert (hits == 1).all()
        np.testing.assert_array_equal(leaf[:8192], which)


def test_certificate_detects_a_planted_mistake():
    """The certificate check itself must fail when one leaf is wrong."""
    w = W.config(1, n_samples=4096)
    x = w.features()
    leaf = oracle.tree_leaves(w.nodes, x, w.n_features)
    bad = leaf.copy()
    leaves = np.nonzero(w.nodes["cls"] >= 0)[0]
    bad[100] = leaves[(np.searchsorted(leaves, bad[100]) + 1) % len(leaves)]
    ok = TU.certificate(w.nodes, x, bad)
    assert not ok[100] and ok[:100].all() and ok[101:].all()


# ---------------------------------------------------------------- forest vote

def _const_tree(c):
    n = np.zeros(1, dtype=W.NODE_DTYPE)
    n[0] = (0, 0.0, -1, c)
    return n


def _forest(trees):
    off = np.zeros(len(trees) + 1, dtype=np.int32)
    off[1:] = np.cumsum([len(t) for t in trees])
    return np.concatenate(trees), off


@pytest.mark.parametrize("votes,want", [
    ([2, 1, 2], 2), ([1, 2], 1), ([0, 3, 3, 5, 5], 3), ([7], 7), ([4, 4, 0, 0], 0),
    ([6, 5, 6, 5, 5], 5),
])
def test_forest_vote_hand_cases(votes, want):
    nodes, off = _forest([_const_tree(c) for c in votes])
    x = np.zeros((3, 2), dtype=np.float32)
    np.testing.assert_array_equal(oracle.forest_classes(nodes, off, x, 2, 8), [want] * 3)


def test_forest_identical_trees_equal_single_tree():
    r = rng(7)
    t = W.complete_tree(r, 5, 6, 8)
    nodes, off = _forest([t] * 32)
    x = W.uniform_f32(r, (3000, 6))
    np.testing.assert_array_equal(oracle.forest_classes(nodes, off, x, 6, 8),
                                  oracle.tree_classes(t, x, 6))


def test_forest_vote_matches_bincount_argmax():
    """Vote by counting each tree's class (numpy argmax returns the first maximum, which
    is the smallest class id)."""
    w = W.config(5, n_samples=2000)
    x = w.features()
    per_tree = np.stack([
        oracle.tree_classes(w.nodes[w.tree_offsets[k]:w.tree_offsets[k + 1]], x, w.n_features)
        for k in range(len(w.tree_offsets) - 1)])
    counts = np.stack([(per_tree == c).sum(axis=0) for c in range(w.n_classes)])
    want = np.argmax(counts, axis=0)
    np.testing.assert_array_equal(
        oracle.forest_classes(w.nodes, w.tree_offsets, x, w.n_features, w.n_classes), want)


# ---------------------------------------------------------------- paper procedures

@pytest.mark.parametrize("seed", range(10))
def test_procedures_4_and_5_reach_the_oracle_leaf(seed):
    r = rng(8000 + seed)
    F = int(r.integers(1, 4))
    pool = np.concatenate([TU.special_pool(), W.uniform_f32(r, 6)])
    nodes = W.random_full_tree(r, int(r.integers(1, 31)), F, 6, threshold_values=pool)
    x = W.uniform_f32(r, (600, F))
    m = r.random(x.shape) < 0.2
    x[m] = pool[r.integers(0, len(pool), size=int(m.sum()))]
    want = oracle.tree_leaves(nodes, x, F)
    leaf4, rounds = procedures.procedure4(nodes, x)
    np.testing.assert_array_equal(leaf4, want)
    # Theta(log2 d) synchronous rounds for a path of d edges (Section 3.3)
    d = TU.depths(nodes)[want]
    np.testing.assert_array_equal(rounds, [int(v - 1).bit_length() if v > 0 else 0 for v in d])
    for hops in (1, 2, 3):
        np.testing.assert_array_equal(procedures.procedure5(nodes, x, hops=hops), want)
    np.testing.assert_array_equal(procedures.procedure5_async(nodes, x[:60], r), want[:60])


# ---------------------------------------------------------------- generators

def test_generator_uniform_grid():
    x = W.config(1).features(10000)
    assert x.max() < 1.0 and x.min() >= 0.0
    s = x.astype(np.float64) * 2 ** 24
    assert np.array_equal(s, np.floor(s))


def test_generator_slices_are_consistent():
    w = W.config(2)
    full = w.features(200000)
    np.testing.assert_array_equal(w.features(1000, start=65000), full[65000:66000])


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4, 5])
def test_generator_trees_are_valid(k):
    w = W.config(k, n_samples=16)
    offs = w.tree_offsets if w.is_forest else np.array([0, len(w.nodes)])
    for a, b in zip(offs[:-1], offs[1:]):
        nodes = w.nodes[a:b]
        internal = nodes["cls"] < 0
        n_int = int(internal.sum())
        assert len(nodes) == 2 * n_int + 1                       # full binary
        assert (nodes["cls"][~internal] < w.n_classes).all()
        assert (nodes["feature"][internal] < w.n_features).all()
        lefts = nodes["left"][internal]
        assert np.array_equal(lefts, 1 + 2 * np.arange(n_int))   # Procedure 1 numbering
        d = TU.depths(nodes)
        if k == 3:
            assert 512 <= n_int <= 1023 and d.max() <= 16
        elif k == 0:
            assert d.max() == 11 and n_int == 15          # the paper's 31-node tree shape
        else:
            depth = {1: 4, 2: 8, 4: 12, 5: 10}[k]
            assert d.max() == depth and n_int == (1 << depth) - 1


# ------------------------------------------------------------- sweep generators

def _depths(nodes):
    d = np.zeros(len(nodes), dtype=np.int64)
    for i in range(len(nodes)):
        if nodes["cls"][i] < 0:
            d[nodes["left"][i]] = d[nodes["left"][i] + 1] = d[i] + 1
    return d


@pytest.mark.parametrize("geometry", W.GEOMETRIES)
def test_sweep_trees_are_valid_and_shaped(geometry):
    from paper_1111_1373_amd import dtree as dt
    nodes = W.sweep_tree(geometry)
    info = dt.tree_check(nodes, 32, 8)
    want = {"complete10": (1023, 10), "paper15": (15, 11), "chain64": (64, 64)}
    if geometry in want:
        assert (info["n_internal"], info["depth"]) == want[geometry]
    else:
        assert info["n_internal"] <= 1023 and info["depth"] <= (16 if geometry == "grown" else 1023)
    assert info["depth"] == _depths(nodes).max()


def test_chain_tree_every_decision_node_has_a_leaf_child():
    """Each decision node above the deepest one has one leaf and one decision child; the
    deepest has two leaves."""
    nodes = W.sweep_tree("chain64")
    d = _depths(nodes)
    inner = np.flatnonzero(nodes["cls"] < 0)
    for i in inner:
        l = nodes["left"][i]
        leaf_kids = int(nodes["cls"][l] >= 0) + int(nodes["cls"][l + 1] >= 0)
        assert leaf_kids == (2 if d[i] == d.max() - 1 else 1)


def test_sweep_rows():
    xc = W.sweep_rows("coherent", 128, 128, 4)
    xi = W.sweep_rows("iid", 128, 128, 4)
    xs = W.sweep_rows("sorted", 128, 128, 4, sort_feature=2)
    for x in (xc, xi, xs):
        assert x.shape == (128 * 128, 4) and x.dtype == np.float32
        assert x.min() >= 0 and x.max() < 1
    assert (np.diff(xs[:, 2]) >= 0).all()
    np.testing.assert_array_equal(np.sort(xs, axis=0), np.sort(xi, axis=0))
    # neighbouring pixels of the coherent raster are close, the i.i.d. records are not
    assert np.abs(np.diff(xc, axis=0)).mean() < 0.1 < 0.3 < np.abs(np.diff(xi, axis=0)).mean()


# ------------------------------------------------------- threaded row-chunk wrapper

def _python_walk(nodes, x):
    """Leaf of every row by the plain root-to-leaf walk (Section 2.1's evaluation), one
    row at a time in Python: independent of the C oracle and of its row chunking."""
    out = np.empty(x.shape[0], dtype=np.int32)
    for s in range(x.shape[0]):
        i = 0
        while nodes["cls"][i] < 0:
            i = nodes["left"][i] if x[s, nodes["feature"][i]] < nodes["threshold"][i] \
                else nodes["left"][i] + 1
        out[s] = i
    return out


@pytest.mark.parametrize("threads", [2, 3, 16])
@pytest.mark.parametrize("n", [0, 1, 2, 5, 17, 1001])
def test_threaded_wrapper_equals_serial_call(threads, n):
    """The oracle split over contiguous row chunks on several host threads returns the
    serial call's result for every row: uneven splits (n not a multiple of the thread
    count), more threads than rows, no rows, a one-row matrix, and rows with ld > F."""
    r = rng(9100 + 31 * threads + n)
    F = 6
    nodes = W.random_full_tree(r, 40, F, 5)
    wide = W.uniform_f32(r, (n, F + 3))
    forest_trees = [W.random_full_tree(r, int(r.integers(1, 30)), F, 5) for _ in range(7)]
    fnodes, foff = _forest(forest_trees)
    for x in (np.ascontiguousarray(wide[:, :F]), wide[:, :F]):      # ld == F, ld == F + 3
        if n > 1:
            assert x.strides[0] // 4 in (F, F + 3)
        leaves = oracle.tree_leaves(nodes, x, F, threads=threads)
        np.testing.assert_array_equal(leaves, oracle.tree_leaves(nodes, x, F))
        np.testing.assert_array_equal(leaves, _python_walk(nodes, x))
        np.testing.assert_array_equal(oracle.tree_classes(nodes, x, F, threads=threads),
                                      nodes["cls"][_python_walk(nodes, x)])
        np.testing.assert_array_equal(
            oracle.forest_classes(fnodes, foff, x, F, 5, threads=threads),
            oracle.forest_classes(fnodes, foff, x, F, 5))


def test_threaded_wrapper_row_chunks_cover_every_row_once():
    """Each row is written by exactly one chunk: a row whose features send it to a
    distinct leaf per position shows up in the right place at every thread count."""
    F = 1
    depth = 7
    t = np.arange(1, 1 << depth, dtype=np.float32)           # thresholds 1 .. 127
    nodes = np.zeros(2 * len(t) + 1, dtype=W.NODE_DTYPE)
    counter = {"t": 0, "leaf": 0}

    def inorder(h, d):
        if d == depth:
            nodes[h] = (0, 0.0, -1, counter["leaf"]); counter["leaf"] += 1
            return
        inorder(2 * h + 1, d + 1)
        nodes[h] = (0, t[counter["t"]], 2 * h + 1, -1); counter["t"] += 1
        inorder(2 * h + 2, d + 1)

    inorder(0, 0)
    for n in (1, 7, 100, 128):
        x = (np.arange(n, dtype=np.float32) % 128)[:, None]
        for threads in (1, 2, 3, 16, 200):
            got = oracle.tree_classes(nodes, x, F, threads=threads)
            np.testing.assert_array_equal(got, np.arange(n) % 128)

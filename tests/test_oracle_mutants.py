"""The oracle pins must catch plausible mistakes in the oracle (CPU only).

Each case compiles a copy of the oracle source with one planted mistake into a temporary
directory and checks that at least one pin rejects it.  The real oracle is untouched.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_1111_1373_amd import workloads as W
from tests import treeutil as TU

SRC = open(os.path.join(os.path.dirname(oracle.__file__), "dtree_oracle.c")).read()

MUTANTS = {
    "le_instead_of_lt": ("if (x < n->threshold)", "if (x <= n->threshold)"),
    "gt_swapped": ("if (x < n->threshold)", "if (!(x > n->threshold))"),
    "children_swapped": ("int32_t left_child = n->left;", "int32_t left_child = n->left + 1;"),
    "right_is_left_plus_2": ("int32_t right_child = n->left + 1;", "int32_t right_child = n->left + 2 < n_nodes ? n->left + 2 : n->left;"),
    "ties_to_larger_class": ("if (votes[c] > votes[best])", "if (votes[c] >= votes[best])"),
    "feature_off_by_one": ("float x = row[n->feature];", "float x = row[n->feature > 0 ? n->feature - 1 : 0];"),
}


def _compile(tmp_path, name, src):
    c = tmp_path / (name + ".c")
    so = tmp_path / (name + ".so")
    c.write_text(src)
    subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-o", str(so), str(c)], check=True)
    lib = ctypes.CDLL(str(so))
    p, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.oracle_tree_leaves.argtypes = [p, i32, i32, p, i64, i64, p]
    lib.oracle_forest_classes.argtypes = [p, p, i32, i32, i32, p, i64, i64, p]
    return lib


def _leaves(lib, nodes, x, F):
    x = np.ascontiguousarray(x, dtype=np.float32)
    nodes = np.ascontiguousarray(nodes)
    out = np.empty(x.shape[0], dtype=np.int32)
    rc = lib.oracle_tree_leaves(nodes.ctypes.data, len(nodes), F, x.ctypes.data, x.shape[0],
                                x.shape[1], out.ctypes.data)
    return out if rc == 0 else None


def _pins_pass(lib):
    """A cheap subset of the pins: hand-worked trees, brute force, forest ties."""
    for t in TU.load_hand_trees():
        got = _leaves(lib, t["nodes"], t["x"], t["n_features"])
        if got is None or not np.array_equal(got, t["leaf"]):
            return False
    r = np.random.Generator(np.random.PCG64(99))
    for _ in range(4):
        F = 3
        nodes = W.random_full_tree(r, 9, F, 5)
        x = W.uniform_f32(r, (3000, F))
        got = _leaves(lib, nodes, x, F)
        hits = np.zeros(len(x), dtype=int); which = np.full(len(x), -1)
        for leaf, c in TU.leaf_conditions(nodes).items():
            ok = TU.satisfied(nodes, x, c); hits += ok; which[ok] = leaf
        if got is None or not np.array_equal(got, which):
            return False
    trees = []
    for c in (1, 2):
        n = np.zeros(1, dtype=W.NODE_DTYPE); n[0] = (0, 0.0, -1, c); trees.append(n)
    nodes = np.concatenate(trees); off = np.array([0, 1, 2], dtype=np.int32)
    x = np.zeros((2, 1), dtype=np.float32); out = np.empty(2, dtype=np.int32)
    lib.oracle_forest_classes(nodes.ctypes.data, off.ctypes.data, 2, 1, 4, x.ctypes.data, 2, 1,
                              out.ctypes.data)
    return bool((out == 1).all())


def test_unmodified_source_passes(tmp_path):
    assert _pins_pass(_compile(tmp_path, "orig", SRC))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    assert SRC.count(old) == 1
    assert not _pins_pass(_compile(tmp_path, name, SRC.replace(old, new)))

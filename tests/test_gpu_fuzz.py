"""Seeded random GPU parity cases: tree shape, feature count, classes, record type,
layout, decomposition, window depths and output kind all drawn at random (and random
forests of 1 to 255 trees), each case checked element by element against the oracle on
the (widened) records."""
import numpy as np
import pytest

import oracle
from paper_1111_1373_amd import workloads as W
from tests import treeutil as TU

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dt():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1111_1373_amd import dtree   # raises ImportError if the library is missing
    return dtree


def _gpu(xn, x_type):
    t = torch.from_numpy(np.ascontiguousarray(xn))
    if x_type == "bf16":
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.cuda()


@pytest.mark.parametrize("seed", range(40))
def test_random_case(dt, seed):
    r = np.random.Generator(np.random.PCG64(9000 + seed))
    F = int(r.choice([1, 2, 3, 4, 5, 7, 8, 12, 16, 19, 31, 32, 33, 48, 64, 65, 100, 128, 200, 256]))
    C = int(r.choice([1, 2, 7, 32, 255, 256, 300]))
    n_int = int(r.choice([0, 1, 2, 5, 15, 63, 200, 1000, 3000]))
    x_type = str(r.choice(["f32", "f32", "f16", "bf16", "u8"]))
    N = int(r.integers(1, 9000))
    pool = np.concatenate([TU.special_pool(), W.uniform_f32(r, 16),
                           np.float32([0.5, 1, 2, 100, 127.5, 200, 255, 256])])
    if n_int == 0:
        nodes = np.zeros(1, dtype=W.NODE_DTYPE)
        nodes[0] = (0, 0.0, -1, int(r.integers(0, C)))
    else:
        nodes = W.random_full_tree(r, n_int, F, C, threshold_values=pool)
    x = W.uniform_f32(r, (N, F + 2))
    if x_type == "u8":
        x = x * np.float32(256)
    m = r.random(x.shape) < 0.05
    x[m] = pool[r.integers(0, len(pool), size=int(m.sum()))]
    if x_type == "f32":
        xn = x
    elif x_type == "u8":
        xn = np.clip(np.nan_to_num(x, nan=0.0), 0, 255).astype(np.uint8)
    elif x_type == "f16":
        xn = W.narrow_records(x, "f16")            # NaN and overflow to infinity included
    else:
        xn = W.narrow_records(np.nan_to_num(x, nan=0.5, posinf=1e30, neginf=-1e30), "bf16")
    xw = xn if x_type == "f32" else TU.widen(xn, x_type)
    layout = str(r.choice(["dense", "strided", "offset"]))
    if layout == "dense":
        host = np.ascontiguousarray(xn[:, :F])
        xd = _gpu(host, x_type)
    elif layout == "strided":
        xd = _gpu(xn, x_type)[:, :F]
    else:
        flat = _gpu(np.concatenate([xn.reshape(-1)[:1], np.ascontiguousarray(xn[:, :F]).reshape(-1)]),
                    x_type)
        xd = flat[1:].view(N, F)
    want_leaf = oracle.tree_leaves(nodes, np.ascontiguousarray(xw[:, :F]), F)
    want_cls = nodes["cls"][want_leaf]
    dd = int(r.integers(0, 17))
    sd = int(r.integers(0, 7))
    t = dt.Tree(nodes, F, C, data_window_depth=dd, spec_window_depth=sd,
                path_hops=int(r.integers(0, 9)), waves_per_cu=int(r.choice([0, 0, 1, 3, 8, 32])))
    algos = ["data", "speculative"] + (["path"] if x_type == "f32" else [])
    for algo in algos:
        for out_kind in ("leaf_i32", "class_i32", "class_u8"):
            if out_kind == "class_u8" and C > 256:
                continue
            got = t.classify(xd, algo=algo, out_kind=out_kind).cpu().numpy().astype(np.int64)
            want = want_leaf if out_kind == "leaf_i32" else want_cls
            np.testing.assert_array_equal(
                got, want, err_msg="seed %d F=%d C=%d n_int=%d %s %s dd=%d sd=%d %s %s"
                % (seed, F, C, n_int, x_type, layout, dd, sd, algo, out_kind))


@pytest.mark.parametrize("seed", range(30))
def test_random_forest(dt, seed):
    """Random forests: 1 to 255 trees of any shape (single leaves included), 1 to 64
    classes, feature counts up to 256, dense or strided records with special values, and
    random data and speculative window depths and wavefront targets, so that the tables
    take every exit encoding, LDS chunking and in-place path; the majority vote against
    the oracle's."""
    r = np.random.Generator(np.random.PCG64(9500 + seed))
    F = int(r.choice([1, 3, 8, 19, 32, 33, 64, 100, 256]))
    C = int(r.choice([1, 2, 8, 9, 16, 17, 64]))
    n_trees = int(r.choice([1, 2, 3, 5, 31, 64, 255]))
    pool = np.concatenate([TU.special_pool(), W.uniform_f32(r, 16)])
    sizes = [0, 1, 3, 15, 63, 255] + ([1023] if n_trees < 64 else [])
    trees = []
    for _ in range(n_trees):
        n_int = int(r.choice(sizes))
        if n_int == 0:
            leaf = np.zeros(1, dtype=W.NODE_DTYPE)
            leaf[0] = (0, 0.0, -1, int(r.integers(0, C)))
            trees.append(leaf)
        else:
            trees.append(W.random_full_tree(r, n_int, F, C, threshold_values=pool))
    off = np.zeros(n_trees + 1, dtype=np.int32)
    off[1:] = np.cumsum([len(t) for t in trees])
    nodes = np.concatenate(trees)
    N = int(r.integers(1, 6000))
    x = W.uniform_f32(r, (N, F + 1))
    m = r.random(x.shape) < 0.05
    x[m] = pool[r.integers(0, len(pool), size=int(m.sum()))]
    dense = np.ascontiguousarray(x[:, :F])
    strided = bool(r.integers(0, 2))
    xd = torch.from_numpy(x).cuda()[:, :F] if strided else torch.from_numpy(dense).cuda()
    dd = int(r.choice([0, 0, 1, 3, 6, 10, 16]))
    sd = int(r.choice([0, 2, 4]))
    waves = int(r.choice([0, 0, 1, 5, 16]))
    f = dt.Forest(nodes, off, F, C, data_window_depth=dd, spec_window_depth=sd, waves_per_cu=waves)
    want = oracle.forest_classes(nodes, off, dense, F, C)
    for algo in ("data", "speculative"):
        for out_kind in ("class_i32", "class_u8"):
            got = f.classify(xd, algo=algo, out_kind=out_kind).cpu().numpy().astype(np.int64)
            np.testing.assert_array_equal(
                got, want, err_msg="seed %d F=%d C=%d trees=%d strided=%d dd=%d sd=%d waves=%d %s %s"
                % (seed, F, C, n_trees, strided, dd, sd, waves, algo, out_kind))

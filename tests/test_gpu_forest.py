"""GPU parity of the forest majority vote (both decompositions) against the CPU oracle."""
import numpy as np
import pytest

import oracle
from paper_1111_1373_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

ALGOS = ["data", "speculative"]


@pytest.fixture(scope="module")
def dt():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1111_1373_amd import dtree
    return dtree


def _forest(trees):
    off = np.zeros(len(trees) + 1, dtype=np.int32)
    off[1:] = np.cumsum([len(t) for t in trees])
    return np.concatenate(trees), off


def _check(dt, nodes, off, x, F, C, algos=ALGOS, xd=None):
    want = oracle.forest_classes(nodes, off, x, F, C)
    f = dt.Forest(nodes, off, F, C)
    xd = torch.from_numpy(np.ascontiguousarray(x)).cuda() if xd is None else xd
    for algo in algos:
        got = f.classify(xd, algo=algo, out_kind="class_i32").cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=algo)
        if C <= 256:
            got8 = f.classify(xd, algo=algo, out_kind="class_u8").cpu().numpy()
            np.testing.assert_array_equal(got8.astype(np.int32), want, err_msg=algo + "/u8")


def test_config5_full_size(dt):
    w = W.config(5)
    x = w.features()
    print("C5", x.shape, flush=True)
    _check(dt, w.nodes, w.tree_offsets, x, w.n_features, w.n_classes)


@pytest.mark.parametrize("votes", [[2, 1, 2], [1, 2], [0, 3, 3, 5, 5], [7], [4, 4, 0, 0],
                                   [6, 5, 6, 5, 5], list(range(8)) * 4])
def test_vote_ties(dt, votes):
    trees = []
    for c in votes:
        n = np.zeros(1, dtype=W.NODE_DTYPE)
        n[0] = (0, 0.0, -1, c)
        trees.append(n)
    nodes, off = _forest(trees)
    x = W.uniform_f32(np.random.Generator(np.random.PCG64(0)), (300, 4))
    _check(dt, nodes, off, x, 4, 8)


@pytest.mark.parametrize("C", [1, 2, 5, 8, 9, 16, 17, 33, 64])
def test_class_counts(dt, C):
    r = np.random.Generator(np.random.PCG64(C))
    trees = [W.complete_tree(r, int(r.integers(1, 7)), 12, C) for _ in range(int(r.integers(3, 20)))]
    nodes, off = _forest(trees)
    x = W.uniform_f32(r, (5000, 12))
    _check(dt, nodes, off, x, 12, C)


@pytest.mark.parametrize("n_trees", [1, 2, 31, 255])
def test_tree_counts_and_shapes(dt, n_trees):
    r = np.random.Generator(np.random.PCG64(100 + n_trees))
    trees = [W.random_full_tree(r, int(r.integers(0, 60)), 19, 7) for _ in range(n_trees)]
    nodes, off = _forest(trees)
    x = W.uniform_f32(r, (3001, 19))        # F = 19: general (non-vectorised) staging
    _check(dt, nodes, off, x, 19, 7)


@pytest.mark.parametrize("F", [20, 100, 200])
@pytest.mark.parametrize("spec_depth", [2, 4])
def test_row_widths_and_window_depths(dt, F, spec_depth):
    """Rows of 20, 100 and 200 features (vector and scalar loads; 16- and 8-wavefront
    workgroups) with several tree chunks per pass, both speculative window depths."""
    r = np.random.Generator(np.random.PCG64(F * 10 + spec_depth))
    trees = [W.complete_tree(r, int(r.integers(6, 10)), F, 11) for _ in range(40)]
    nodes, off = _forest(trees)
    x = W.uniform_f32(r, (6001, F))
    want = oracle.forest_classes(nodes, off, x, F, 11)
    f = dt.Forest(nodes, off, F, 11, spec_window_depth=spec_depth)
    xd = torch.from_numpy(x).cuda()
    for algo in ALGOS:
        got = f.classify(xd, algo=algo, out_kind="class_i32").cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=algo)


def test_large_trees_read_tables_in_place(dt):
    """Trees whose tables do not fit the LDS: the forest reads them from global memory."""
    r = np.random.Generator(np.random.PCG64(7))
    trees = [W.random_full_tree(r, 8191, 16, 10) for _ in range(3)]
    nodes, off = _forest(trees)
    x = W.uniform_f32(r, (4000, 16))
    _check(dt, nodes, off, x, 16, 10)


@pytest.mark.parametrize("n_internal", [1024, 1025, 32768, 32769])
def test_exit_codes_at_the_int16_limit(dt, n_internal):
    """Exit codes are packed into the windows' bottom slots when every code of the forest
    fits 11 bits, else stored as int16 when they fit 16, else as int32.  A chain cut into
    one-node windows has window ids 0 .. n_internal - 1: the largest is 1023 (packed) for
    1,024 decision nodes, 1024 (int16) for 1,025, 32767 (int16) for 32,768 and 32768
    (int32) for 32,769.  Exits are rare (one record in 10,000 per node), so most records
    travel the whole chain of 1,024 and a few percent past window 32,767."""
    r = np.random.Generator(np.random.PCG64(11))
    chain = W.chain_tree(r, n_internal, 8, 5, p_exit=1e-4)
    nodes, off = _forest([chain, W.complete_tree(r, 6, 8, 5)])
    x = W.uniform_f32(r, (3000, 8))
    want = oracle.forest_classes(nodes, off, x, 8, 5)
    f = dt.Forest(nodes, off, 8, 5, data_window_depth=1)
    got = f.classify(torch.from_numpy(x).cuda(), algo="data", out_kind="class_i32").cpu().numpy()
    np.testing.assert_array_equal(got, want)
    # some records reach the last window (its decision node is at depth n_internal - 1, and
    # the chain's breadth-first ids put its leaves at 2 (n_internal - 1) + 1 and + 2)
    assert (oracle.tree_leaves(chain, x, 8) >= 2 * (n_internal - 1) + 1).sum() > 10


@pytest.mark.parametrize("F", [4, 32, 64, 65])
def test_special_values_ties_and_near_ties(dt, F):
    """Records on and around the thresholds of a forest: a quarter of every record's values
    sit on a threshold or on one of its float neighbours up to 40 steps away, and a few
    are NaN, -0/+0, infinities or denormals, which also appear among the thresholds."""
    from tests import treeutil as TU
    r = np.random.Generator(np.random.PCG64(1373 + F))
    pool = np.concatenate([TU.special_pool(), W.uniform_f32(r, 8), -W.uniform_f32(r, 4),
                           np.float32([3e-39, -3e-39, 1e30, -1e30])])
    trees = [W.random_full_tree(r, int(r.integers(1, 120)), F, 6, threshold_values=pool)
             for _ in range(9)]
    nodes, off = _forest(trees)
    internal = nodes["cls"] < 0
    th = nodes["threshold"][internal]
    n = 20000
    x = W.uniform_f32(r, (n, F))
    # every record: a quarter of its entries on a threshold or a float neighbour of one
    pick = r.random((n, F)) < 0.25
    base = th[r.integers(0, len(th), size=int(pick.sum()))]
    steps = r.integers(-40, 41, size=base.shape)
    toward = np.where(steps > 0, np.float32(np.inf), np.float32(-np.inf)).astype(np.float32)
    near = base.copy()
    with np.errstate(over="ignore", invalid="ignore"):
        for i in range(1, 41):
            m = np.abs(steps) >= i
            near[m] = np.nextafter(near[m], toward[m])
    x[pick] = near
    special = r.random((n, F)) < 0.03
    x[special] = pool[r.integers(0, len(pool), size=int(special.sum()))]
    _check(dt, nodes, off, x, F, 6)


@pytest.mark.parametrize("waves", [1, 3, 8, 12, 15, 16])
def test_workgroup_shapes_and_chunkings(dt, waves):
    """Other wavefront counts give other chunk budgets: one to many trees per LDS chunk,
    walked in groups of four, three, two or one."""
    w = W.config(5, n_samples=9000)
    x = w.features()
    want = oracle.forest_classes(w.nodes, w.tree_offsets, x, w.n_features, w.n_classes)
    f = dt.Forest(w.nodes, w.tree_offsets, w.n_features, w.n_classes, waves_per_cu=waves)
    xd = torch.from_numpy(x).cuda()
    for algo in ALGOS:
        got = f.classify(xd, algo=algo, out_kind="class_i32").cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=algo)


@pytest.mark.parametrize("n", [1, 63, 65, 130, 1000, 70000])
def test_ragged_sizes_and_strides(dt, n):
    w = W.config(5, n_samples=n)
    x = w.features()
    _check(dt, w.nodes, w.tree_offsets, x, w.n_features, w.n_classes)
    padded = torch.zeros((n, w.n_features + 3), dtype=torch.float32, device="cuda")
    padded[:, :w.n_features] = torch.from_numpy(x).cuda()
    _check(dt, w.nodes, w.tree_offsets, x, w.n_features, w.n_classes,
           xd=padded[:, :w.n_features])


def test_forest_argument_errors(dt):
    w = W.config(5, n_samples=10)
    f = dt.Forest(w.nodes, w.tree_offsets, w.n_features, w.n_classes)
    x = torch.from_numpy(w.features()).cuda()
    with pytest.raises(dt.DTreeError):
        f.classify(x, out_kind="leaf_i32")
    out = torch.empty(10, dtype=torch.uint8, device="cuda")
    assert dt._lib.dt_forest_classify(f._h, x.data_ptr(), 10, 31, out.data_ptr(), 0, 0, None) == dt.DT_ERR_INVALID_ARG
    assert dt._lib.dt_forest_classify(f._h, x.data_ptr(), 0, 32, out.data_ptr(), 0, 0, None) == dt.DT_OK
    # the path-array kernel is a single-tree decomposition
    assert dt._lib.dt_forest_classify(f._h, x.data_ptr(), 10, 32, out.data_ptr(), 0, 2, None) == dt.DT_ERR_UNSUPPORTED
    assert dt._lib.dt_forest_classify(f._h, x.data_ptr(), 10, 32, out.data_ptr(), 0, 3, None) == dt.DT_ERR_INVALID_ARG

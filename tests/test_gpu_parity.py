"""GPU parity: every decomposition against the CPU oracle, element by element, bit-exact.

Labels and leaf indices are integers decided by exact fp32 comparisons, so the tolerance
is zero.  Runs through the C ABI (``paper_1111_1373_amd.dtree`` -> ``libdtree.so``).
"""
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


# data: Procedure 3; speculative: Procedures 4-5 with the predicate mask; path: Procedures
# 4-5 with the path array and pointer jumping as printed.
ALGOS = ["data", "speculative", "path"]


def _gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _check_all_outputs(dt, tree, nodes, x_np, x_dev, F, algos=ALGOS):
    want_cls = oracle.tree_classes(nodes, x_np, F)
    want_leaf = oracle.tree_leaves(nodes, x_np, F)
    for algo in algos:
        got_leaf = tree.classify(x_dev, algo=algo, out_kind="leaf_i32").cpu().numpy()
        np.testing.assert_array_equal(got_leaf, want_leaf, err_msg="leaf/" + algo)
        got_i32 = tree.classify(x_dev, algo=algo, out_kind="class_i32").cpu().numpy()
        np.testing.assert_array_equal(got_i32, want_cls, err_msg="i32/" + algo)
        if tree.n_classes <= 256:
            got_u8 = tree.classify(x_dev, algo=algo, out_kind="class_u8").cpu().numpy()
            np.testing.assert_array_equal(got_u8.astype(np.int32), want_cls, err_msg="u8/" + algo)


# ------------------------------------------------------------------ hand-worked trees

@pytest.mark.parametrize("tree", TU.load_hand_trees(), ids=lambda t: t["name"])
def test_hand_trees(dt, tree):
    for dd in range(1, max(1, int(TU.depths(tree["nodes"]).max())) + 1):
        for sd in range(1, 7):
            t = dt.Tree(tree["nodes"], tree["n_features"], tree["n_classes"],
                        data_window_depth=dd, spec_window_depth=sd)
            x = _gpu(tree["x"])
            for algo in ALGOS:
                got = t.classify(x, algo=algo, out_kind="leaf_i32").cpu().numpy()
                np.testing.assert_array_equal(got, tree["leaf"], err_msg="%s dd=%d sd=%d" % (algo, dd, sd))
                got = t.classify(x, algo=algo, out_kind="class_i32").cpu().numpy()
                np.testing.assert_array_equal(got, tree["cls"])


# ------------------------------------------------------------------ configurations

@pytest.mark.parametrize("k", [0, 1, 2, 3])
def test_config_full_size(dt, k):
    w = W.config(k)
    x = w.features()
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    print("config", w.name, t.info, flush=True)
    _check_all_outputs(dt, t, w.nodes, x, _gpu(x), w.n_features)


@pytest.mark.parametrize("k", [1, 2, 3])
@pytest.mark.parametrize("sd", [1, 2, 3, 4, 5, 6])
def test_config_every_spec_window_depth(dt, k, sd):
    w = W.config(k, n_samples=20_000)
    x = w.features()
    t = dt.Tree(w.nodes, w.n_features, w.n_classes, spec_window_depth=sd,
                data_window_depth=sd)
    want = oracle.tree_leaves(w.nodes, x, w.n_features)
    xd = _gpu(x)
    for algo in ALGOS:
        got = t.classify(xd, algo=algo, out_kind="leaf_i32").cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=algo)


def test_config4_full_size(dt):
    """The largest single-tree workload at its full size (4 GiB of features)."""
    w = W.config(4)
    x = w.features()
    print("C4 features generated", x.shape, flush=True)
    want = oracle.tree_classes(w.nodes, x, w.n_features)
    print("C4 oracle done", flush=True)
    xd = _gpu(x)
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    for algo in ALGOS:
        got = t.classify(xd, algo=algo, out_kind="class_u8").cpu().numpy()
        np.testing.assert_array_equal(got.astype(np.int32), want, err_msg=algo)
        print("C4", algo, "ok", flush=True)
    # leaf indices on a sample of rows (the oracle computes them one by one)
    idx = np.random.Generator(np.random.PCG64(4)).integers(0, x.shape[0], size=200_000)
    want_leaf = oracle.tree_leaves(w.nodes, x[idx], w.n_features)
    for algo in ALGOS:
        got = t.classify(xd, algo=algo, out_kind="leaf_i32")[torch.from_numpy(idx).cuda()]
        np.testing.assert_array_equal(got.cpu().numpy(), want_leaf, err_msg=algo)


@pytest.mark.parametrize("sd", [3, 4, 5, 6])
def test_config4_tree_every_wide_spec_window_depth(dt, sd):
    """The C4 tree (complete depth 12, 4,095 decision nodes) with the wide speculative
    windows: at depth 6 it is cut into 1 + 64 full 63-slot windows (subtree blocking,
    Section 3.4 and the windows of Section 6).  200,000 seeded rows of the C4 records with
    exact ties planted on every path level and NaN features."""
    w = W.config(4, n_samples=200_000)
    x = w.features()
    F = w.n_features
    r = np.random.Generator(np.random.PCG64(4000 + sd))
    # ties: set the feature a row tests at some level of its own path to that threshold
    leaf = oracle.tree_leaves(w.nodes, x, F)
    rows = r.choice(x.shape[0], size=20_000, replace=False)
    for s in rows:
        i = 0
        level = int(r.integers(0, 12))
        for _ in range(level):
            i = w.nodes["left"][i] + int(not (x[s, w.nodes["feature"][i]] < w.nodes["threshold"][i]))
        x[s, w.nodes["feature"][i]] = w.nodes["threshold"][i]
    nan_rows = r.choice(x.shape[0], size=5_000, replace=False)
    x[nan_rows, r.integers(0, F, size=nan_rows.size)] = np.nan
    x[::4099, :] = np.nan
    assert (oracle.tree_leaves(w.nodes, x, F) != leaf).any()     # the planting moved rows
    t = dt.Tree(w.nodes, F, w.n_classes, spec_window_depth=sd)
    info = t.info
    print("C4 tree, spec depth", sd, info, flush=True)
    assert info["spec_window_depth"] == sd
    _check_all_outputs(dt, t, w.nodes, x, _gpu(x), F)


@pytest.mark.parametrize("hops", [1, 2, 3, 8])
@pytest.mark.parametrize("sd", [1, 3, 4, 6])
def test_path_reduction_hops(dt, hops, sd):
    """The path kernel with every reach per round (path[i] <- entry `hops` further on)."""
    w = W.config(3, n_samples=9_000)
    x = w.features()
    t = dt.Tree(w.nodes, w.n_features, w.n_classes, spec_window_depth=sd, path_hops=hops)
    want = oracle.tree_leaves(w.nodes, x, w.n_features)
    got = t.classify(_gpu(x), algo="path", out_kind="leaf_i32").cpu().numpy()
    np.testing.assert_array_equal(got, want)


# ------------------------------------------------------------------ edge cases

@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 127, 129, 1000, 4097])
def test_ragged_sizes(dt, n):
    w = W.config(2, n_samples=n)
    x = w.features()
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    _check_all_outputs(dt, t, w.nodes, x, _gpu(x), w.n_features)


@pytest.mark.parametrize("sd", [5, 6])
@pytest.mark.parametrize("n", [1, 15, 16, 17, 31, 33, 47, 63, 65, 1000, 4097])
def test_ragged_sizes_32_record_tiles(dt, sd, n):
    """Speculative windows of depth 5 and 6 (32- and 64-lane record groups, Section 3.4)
    run on tiles of 32 records; at depth 5 records 16-31 of a tile are walked in lanes
    32-47 and moved back to record order at the end.  Inputs whose last tile is partial
    in either half of it, or a single record."""
    w = W.config(2, n_samples=n)
    x = w.features()
    t = dt.Tree(w.nodes, w.n_features, w.n_classes, spec_window_depth=sd)
    xd = _gpu(x)
    assert t.launch_info(xd, algo="speculative")["tile_rows"] == 32
    _check_all_outputs(dt, t, w.nodes, x, xd, w.n_features, algos=("speculative",))


def test_empty_input(dt):
    w = W.config(1, n_samples=0)
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    x = torch.empty((0, w.n_features), dtype=torch.float32, device="cuda")
    for algo in ALGOS:
        assert t.classify(x, algo=algo).numel() == 0


def test_empty_input_does_not_write(dt):
    w = W.config(1, n_samples=10)
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    x = _gpu(w.features())
    out = torch.full((10,), 77, dtype=torch.uint8, device="cuda")
    st = dt._lib.dt_classify(t._h, x.data_ptr(), 0, w.n_features, out.data_ptr(), 0, 0, None)
    assert st == dt.DT_OK
    torch.cuda.synchronize()
    assert (out == 77).all()


@pytest.mark.parametrize("F", [1, 3, 4, 19, 33, 64, 100, 128, 256])
def test_feature_counts_and_strides(dt, F):
    """Dense rows (vectorised path when F % 4 == 0), padded rows (ld > F) and an
    unaligned base pointer (general path)."""
    r = np.random.Generator(np.random.PCG64(F))
    nodes = W.random_full_tree(r, 300, F, 11)
    x = W.uniform_f32(r, (3001, F + 5))
    t = dt.Tree(nodes, F, 11)
    dense = np.ascontiguousarray(x[:, :F])
    _check_all_outputs(dt, t, nodes, dense, _gpu(dense), F)
    xd = _gpu(x)
    _check_all_outputs(dt, t, nodes, x, xd[:, :F], F)          # ld = F + 5
    shifted = xd.reshape(-1)[1:1 + 3000 * F].reshape(3000, F)    # 4-byte aligned only
    _check_all_outputs(dt, t, nodes, x.reshape(-1)[1:1 + 3000 * F].reshape(3000, F), shifted, F)


def test_special_values_and_ties(dt):
    r = np.random.Generator(np.random.PCG64(31))
    F = 8
    pool = TU.special_pool()
    nodes = W.random_full_tree(r, 200, F, 9, threshold_values=np.concatenate([pool, W.uniform_f32(r, 16)]))
    x = W.uniform_f32(r, (20000, F))
    m = r.random(x.shape) < 0.3
    x[m] = pool[r.integers(0, len(pool), size=int(m.sum()))]
    internal = np.nonzero(nodes["cls"] < 0)[0]
    for k in range(0, 20000, 3):             # exact ties on decision nodes
        i = internal[k % len(internal)]
        x[k, nodes["feature"][i]] = nodes["threshold"][i]
    den = np.float32(np.ldexp(1.0, -149))
    x[1::97, :] = den
    x[2::97, :] = -den
    t = dt.Tree(nodes, F, 9)
    _check_all_outputs(dt, t, nodes, x, _gpu(x), F)


@pytest.mark.parametrize("n_int", [1, 15, 63, 64, 255, 1023, 4095])
def test_tree_sizes(dt, n_int):
    r = np.random.Generator(np.random.PCG64(n_int))
    nodes = W.random_full_tree(r, n_int, 16, 32)
    x = W.uniform_f32(r, (5000, 16))
    t = dt.Tree(nodes, 16, 32)
    print(n_int, t.info, flush=True)
    _check_all_outputs(dt, t, nodes, x, _gpu(x), 16)


def test_single_leaf_and_chain(dt):
    leaf = np.zeros(1, dtype=W.NODE_DTYPE)
    leaf[0] = (0, 0.0, -1, 5)
    x = W.uniform_f32(np.random.Generator(np.random.PCG64(1)), (300, 4))
    t = dt.Tree(leaf, 4, 6)
    _check_all_outputs(dt, t, leaf, x, _gpu(x), 4)
    # a chain of depth 40 (the paper's tree is chain-like: 15 decision nodes, depth 11)
    d = 40
    chain = np.zeros(2 * d + 1, dtype=W.NODE_DTYPE)
    for i in range(d):
        chain[2 * i] = (i % 4, np.float32(0.5 + 0.01 * (i % 7) - 0.03), 2 * i + 1, -1)
        chain[2 * i + 1] = (0, 0.0, -1, i % 6)
    chain[2 * d] = (0, 0.0, -1, 5)
    # right child continues the chain: node 2i's children are 2i+1 (leaf) and 2i+2
    x = W.uniform_f32(np.random.Generator(np.random.PCG64(2)), (20000, 4)) * np.float32(0.1) + np.float32(0.5)
    t = dt.Tree(chain, 4, 6)
    _check_all_outputs(dt, t, chain, x, _gpu(x), 4)


def test_paper_shape_tree(dt):
    """The paper's experiment shape (Section 4.1): 19 features, 7 classes, 15 decision
    nodes, depth 11, 65,536 records (a 256x256 image); synthetic stand-in."""
    r = np.random.Generator(np.random.PCG64(1111))
    nodes = W.paper_shape_tree(r)
    assert int(TU.depths(nodes).max()) == 11 and int((nodes["cls"] < 0).sum()) == 15
    x = W.uniform_f32(r, (65536, 19))
    t = dt.Tree(nodes, 19, 7)
    _check_all_outputs(dt, t, nodes, x, _gpu(x), 19)


# ------------------------------------------------------------------ errors and streams

def test_argument_errors(dt):
    w = W.config(1, n_samples=100)
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    x = _gpu(w.features())
    out = torch.empty(100, dtype=torch.uint8, device="cuda")
    L = dt._lib
    assert L.dt_classify(t._h, x.data_ptr(), 100, 7, out.data_ptr(), 0, 0, None) == dt.DT_ERR_INVALID_ARG
    assert L.dt_classify(t._h, x.data_ptr(), -1, 8, out.data_ptr(), 0, 0, None) == dt.DT_ERR_INVALID_ARG
    assert L.dt_classify(t._h, x.data_ptr(), 100, 8, out.data_ptr(), 5, 0, None) == dt.DT_ERR_INVALID_ARG
    assert L.dt_classify(t._h, x.data_ptr(), 100, 8, out.data_ptr(), 0, 9, None) == dt.DT_ERR_INVALID_ARG
    assert L.dt_classify(None, x.data_ptr(), 100, 8, out.data_ptr(), 0, 0, None) == dt.DT_ERR_INVALID_ARG
    assert L.dt_classify(t._h, None, 100, 8, out.data_ptr(), 0, 0, None) == dt.DT_ERR_INVALID_ARG
    big = np.zeros(3, dtype=W.NODE_DTYPE)
    big[0] = (0, 0.5, 1, -1); big[1] = (0, 0, -1, 0); big[2] = (0, 0, -1, 300)
    tb = dt.Tree(big, 8, 301)
    assert L.dt_classify(tb._h, x.data_ptr(), 100, 8, out.data_ptr(), 0, 0, None) == dt.DT_ERR_INVALID_ARG
    i32 = tb.classify(x, out_kind="class_i32").cpu().numpy()
    np.testing.assert_array_equal(i32, oracle.tree_classes(big, w.features(), 8))
    wide = np.zeros(3, dtype=W.NODE_DTYPE)
    wide[0] = (300, 0.5, 1, -1); wide[1] = (0, 0, -1, 0); wide[2] = (0, 0, -1, 1)
    tw = dt.Tree(wide, 301, 2)
    xw = torch.zeros((10, 301), dtype=torch.float32, device="cuda")
    with pytest.raises(dt.DTreeError) as e:
        tw.classify(xw)
    assert e.value.status == dt.DT_ERR_UNSUPPORTED
    assert (out >= 0).all()


def test_non_default_stream(dt):
    w = W.config(3, n_samples=100_000)
    x = w.features()
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    s = torch.cuda.Stream()
    xd = _gpu(x)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        outs = [t.classify(xd, algo=a) for a in ALGOS]
    s.synchronize()
    want = oracle.tree_classes(w.nodes, x, w.n_features)
    for o in outs:
        np.testing.assert_array_equal(o.cpu().numpy().astype(np.int32), want)


def test_repeated_calls_are_deterministic(dt):
    w = W.config(2, n_samples=100_000)
    x = _gpu(w.features())
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    first = t.classify(x, algo="speculative").cpu()
    for _ in range(5):
        assert torch.equal(t.classify(x, algo="speculative").cpu(), first)
        assert torch.equal(t.classify(x, algo="data").cpu(), first)


def test_probe_copy(dt):
    src = torch.arange(1 << 20, dtype=torch.int32, device="cuda")
    dst = torch.zeros_like(src)
    dt.probe_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


def test_probe_read(dt):
    """The streaming-read probe reads any 16-byte multiple and writes nothing."""
    sink = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    for n in (4, 4096, (1 << 20) + 12):                 # partial tile, whole tiles, ragged
        src = torch.arange(n, dtype=torch.int32, device="cuda")
        for wpc in (1, 8, 32):
            dt.probe_read(src, sink, wpc)
    torch.cuda.synchronize()
    assert int(sink.item()) == 7
    src = torch.zeros(8, dtype=torch.int32, device="cuda")
    lib = dt._lib
    assert lib.dt_probe_read(src.data_ptr(), 20, sink.data_ptr(), 8, None) == dt.DT_ERR_INVALID_ARG
    assert lib.dt_probe_read(src.data_ptr() + 4, 16, sink.data_ptr(), 8, None) == dt.DT_ERR_INVALID_ARG
    assert lib.dt_probe_read(src.data_ptr(), 16, sink.data_ptr(), 0, None) == dt.DT_ERR_INVALID_ARG
    assert lib.dt_probe_read(src.data_ptr(), 0, None, 8, None) == dt.DT_OK


def test_more_than_2_31_elements(dt):
    """64-bit indexing: 2.25 x 10^9 feature elements (9 GB) on the device, built by repeating
    the C4 records; the labels must repeat the oracle's C4 labels."""
    w = W.config(4)
    x = w.features()
    want = oracle.tree_classes(w.nodes, x, w.n_features)
    xd = _gpu(x)
    reps, extra = 2, 1_500_001
    big = torch.cat([xd] * reps + [xd[:extra]])
    del xd
    n = big.shape[0]
    assert n * w.n_features > 2 ** 31
    print("rows", n, "elements", n * w.n_features, flush=True)
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    expect = torch.from_numpy(np.concatenate([want] * reps + [want[:extra]]).astype(np.uint8))
    for algo in ALGOS[:2]:
        got = t.classify(big, algo=algo).cpu()
        assert torch.equal(got, expect), algo
    # strided view of the same memory (scalar loads, 64-bit row offsets)
    view = big[:, : w.n_features - 1]
    nodes = w.nodes.copy()
    inner = nodes["cls"] < 0
    nodes["feature"][inner] = np.minimum(nodes["feature"][inner], w.n_features - 2)
    want2 = oracle.tree_classes(nodes, x[-100_000:, : w.n_features - 1], w.n_features - 1)
    t2 = dt.Tree(nodes, w.n_features - 1, w.n_classes)
    got2 = t2.classify(view, algo="data").cpu().numpy()
    np.testing.assert_array_equal(got2[n - extra - 100_000: n - extra].astype(np.int32), want2)

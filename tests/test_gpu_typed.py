"""GPU parity for narrow record types (dt_classify_typed): fp16, bf16 and uint8 records.

The expected labels are the oracle's on the exactly widened fp32 records; integer outputs,
so the comparison is exact.
"""
import numpy as np
import pytest

import oracle
from paper_1111_1373_amd import workloads as W
from tests import treeutil as TU

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

X_TYPES = ["f16", "bf16", "u8"]
ALGOS = ["data", "speculative"]


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


def _check(dt, tree, nodes, xn, x_type, F, xd=None, algos=ALGOS, outs=("leaf_i32", "class_i32", "class_u8")):
    xw = TU.widen(xn, x_type)
    want_cls = oracle.tree_classes(nodes, xw, F)
    want_leaf = oracle.tree_leaves(nodes, xw, F)
    xd = _gpu(xn, x_type) if xd is None else xd
    for algo in algos:
        for o in outs:
            if o == "class_u8" and tree.n_classes > 256:
                continue
            got = tree.classify(xd, algo=algo, out_kind=o).cpu().numpy().astype(np.int32)
            np.testing.assert_array_equal(got, want_leaf if o == "leaf_i32" else want_cls,
                                          err_msg="%s/%s/%s" % (x_type, algo, o))


@pytest.mark.parametrize("x_type", X_TYPES)
@pytest.mark.parametrize("k", [1, 2, 3])
def test_configs(dt, x_type, k):
    w = W.config(k)
    xn = W.narrow_records(w.features(), x_type, w.feature_dist)
    nodes = W.narrow_tree(w.nodes, x_type, w.feature_dist)
    t = dt.Tree(nodes, w.n_features, w.n_classes)
    print("config", w.name, x_type, t.launch_info(_gpu(xn[:64], x_type)), flush=True)
    _check(dt, t, nodes, xn, x_type, w.n_features)


@pytest.mark.parametrize("x_type", X_TYPES)
def test_config4_full_size(dt, x_type):
    w = W.config(4)
    xn = W.narrow_records(w.features(), x_type)
    nodes = W.narrow_tree(w.nodes, x_type)
    print("C4", x_type, "generated", flush=True)
    t = dt.Tree(nodes, w.n_features, w.n_classes)
    _check(dt, t, nodes, xn, x_type, w.n_features, outs=("class_u8",))
    print("C4", x_type, "ok", flush=True)


@pytest.mark.parametrize("x_type", X_TYPES)
@pytest.mark.parametrize("F", [1, 3, 4, 8, 16, 17, 32, 64, 100, 128, 256])
def test_feature_counts_and_layouts(dt, x_type, F):
    """Every LDS row stride, with dense, strided and 16-byte-misaligned rows (the vector,
    exact and scalar staging paths)."""
    r = np.random.Generator(np.random.PCG64(1000 + F))
    n = 3000 + F
    x = W.uniform_f32(r, (n, F + 3))
    xn_wide = W.narrow_records(x, x_type)
    nodes = W.narrow_tree(W.random_full_tree(r, 60, F, 7), x_type)
    t = dt.Tree(nodes, F, 7, spec_window_depth=3)
    dense = np.ascontiguousarray(xn_wide[:, :F])
    _check(dt, t, nodes, dense, x_type, F, outs=("leaf_i32",))
    # strided rows: ld = F + 3
    full = _gpu(xn_wide, x_type)
    _check(dt, t, nodes, dense, x_type, F, xd=full[:, :F], outs=("leaf_i32",))
    # start one element past a 16-byte boundary
    flat = _gpu(np.concatenate([xn_wide.reshape(-1)[:1], dense.reshape(-1)]), x_type)
    _check(dt, t, nodes, dense, x_type, F, xd=flat[1:].view(n, F), outs=("leaf_i32",))


@pytest.mark.parametrize("x_type", X_TYPES)
def test_special_values_and_ties(dt, x_type):
    """Signed zeros, subnormals, infinities, NaN and values equal to a threshold (ties go
    right), against thresholds on, between and outside the type's grid."""
    r = np.random.Generator(np.random.PCG64(5))
    spec = TU.narrow_specials(x_type)
    F = 4
    vals = TU.widen(spec, x_type)
    finite = vals[np.isfinite(vals)]
    with np.errstate(over="ignore"):
        pool = np.concatenate([vals, TU.special_pool(),
                               np.nextafter(finite, np.float32(np.inf)),
                               np.nextafter(finite, np.float32(-np.inf)),
                               (finite.astype(np.float64) + 0.5).astype(np.float32)]).astype(np.float32)
    nodes = W.random_full_tree(r, 200, F, 5, threshold_values=pool)
    xn = spec[r.integers(0, len(spec), size=(20_000, F))]
    t = dt.Tree(nodes, F, 5)
    _check(dt, t, nodes, xn, x_type, F)


@pytest.mark.parametrize("x_type", X_TYPES)
def test_ragged_and_empty(dt, x_type):
    w = W.config(2, n_samples=4097)
    xn = W.narrow_records(w.features(), x_type)
    nodes = W.narrow_tree(w.nodes, x_type)
    t = dt.Tree(nodes, w.n_features, w.n_classes)
    for n in (0, 1, 63, 64, 65, 4097):
        if n == 0:
            assert t.classify(_gpu(xn[:1], x_type)[:0]).numel() == 0
            continue
        _check(dt, t, nodes, xn[:n], x_type, w.n_features, outs=("class_u8",))


@pytest.mark.parametrize("x_type", X_TYPES)
@pytest.mark.parametrize("sd", [5, 6])
def test_ragged_wide_windows(dt, x_type, sd):
    """Speculative windows of depth 5 and 6 on narrow records (32-record tiles where the
    rows take at least 32 bytes), on inputs whose last tile is partial."""
    w = W.config(2, n_samples=4097)
    xn = W.narrow_records(w.features(), x_type)
    nodes = W.narrow_tree(w.nodes, x_type)
    t = dt.Tree(nodes, w.n_features, w.n_classes, spec_window_depth=sd)
    for n in (1, 17, 33, 65, 4097):
        _check(dt, t, nodes, xn[:n], x_type, w.n_features, algos=("speculative",))


def test_errors(dt):
    w = W.config(1, n_samples=64)
    t = dt.Tree(w.nodes, w.n_features, w.n_classes)
    xh = _gpu(W.narrow_records(w.features(), "f16"), "f16")
    out = torch.zeros(64, dtype=torch.int32, device="cuda")
    lib = dt._lib
    # path kernel: fp32 records only
    with pytest.raises(dt.DTreeError) as e:
        t.classify(xh, algo="path")
    assert e.value.status == dt.DT_ERR_UNSUPPORTED
    # unknown type, misaligned element pointer: rejected before any launch
    assert lib.dt_classify_typed(t._h, xh.data_ptr(), 9, 64, 8, out.data_ptr(), 1, 0, None) == dt.DT_ERR_INVALID_ARG
    assert lib.dt_classify_typed(t._h, xh.data_ptr() + 1, 1, 63, 8, out.data_ptr(), 1, 0, None) == dt.DT_ERR_INVALID_ARG
    assert lib.dt_classify_typed(t._h, xh.data_ptr(), 1, 64, 7, out.data_ptr(), 1, 0, None) == dt.DT_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert int(out.abs().sum()) == 0
    with pytest.raises(TypeError):
        t.classify(xh.to(torch.int32))

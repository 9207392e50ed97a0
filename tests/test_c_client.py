"""The C ABI from C: tests/c/dt_client.c includes only dtree.h and links only libdtree.so,
built with gcc as strict C11.  On the CPU it runs the host-only calls (ABI version, tree
validation); on the GPU it classifies host-resident records through the library and its
labels are compared with the oracle's, element by element."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from paper_1111_1373_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_1111_1373_amd")
DT_ERR_INVALID_TREE = 2


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    if not os.path.exists(os.path.join(PKG, "libdtree.so")):
        pytest.skip("library not built")
    exe = str(tmp_path_factory.mktemp("c_client") / "dt_client")
    subprocess.run(["gcc", "-std=c11", "-pedantic", "-Wall", "-Wextra", "-Werror",
                    "-I" + os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "dt_client.c"),
                    "-L" + PKG, "-ldtree", "-Wl,-rpath," + PKG, "-o", exe],
                   check=True, capture_output=True, text=True)
    return exe


def _tree_file(path, nodes, F, C):
    with open(path, "wb") as f:
        np.array([len(nodes), F, C], dtype=np.int32).tofile(f)
        np.ascontiguousarray(nodes).tofile(f)


def _forest_file(path, nodes, offsets, F, C):
    with open(path, "wb") as f:
        np.array([len(offsets) - 1, F, C], dtype=np.int32).tofile(f)
        np.ascontiguousarray(offsets, dtype=np.int32).tofile(f)
        np.ascontiguousarray(nodes).tofile(f)


def _records_file(path, x):
    with open(path, "wb") as f:
        np.array([len(x)], dtype=np.int64).tofile(f)
        np.ascontiguousarray(x, dtype=np.float32).tofile(f)


def _run(args):
    return subprocess.run(args, capture_output=True, text=True, timeout=120)


def test_header_is_c11_and_host_calls_work(client, tmp_path):
    from paper_1111_1373_amd import dtree as dt
    for k in (1, 2, 3):
        w = W.config(k)
        tf = str(tmp_path / "tree.bin")
        _tree_file(tf, w.nodes, w.n_features, w.n_classes)
        r = _run([client, "check", tf])
        assert r.returncode == 0, r.stderr
        info = dt.tree_check(w.nodes, w.n_features, w.n_classes)
        assert r.stdout.split() == [str(info["data_window_depth"]), str(info["data_windows"]),
                                    str(info["data_levels"])]
    bad = W.config(1).nodes.copy()
    bad[2]["left"] = 0                          # an edge back to the root
    _tree_file(str(tmp_path / "bad.bin"), bad, 8, 4)
    r = _run([client, "check", str(tmp_path / "bad.bin")])
    assert r.returncode == DT_ERR_INVALID_TREE, r.stdout + r.stderr
    assert "dt_tree_check" in r.stderr


@pytest.mark.gpu
def test_c_client_classifies(client, tmp_path):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.config(3, n_samples=50_001)
    x = w.features()
    tf, xf, of = (str(tmp_path / n) for n in ("tree.bin", "x.bin", "out.bin"))
    _tree_file(tf, w.nodes, w.n_features, w.n_classes)
    _records_file(xf, x)
    want = oracle.tree_classes(w.nodes, x, w.n_features)
    for algo in (0, 1, 2):
        r = _run([client, "classify", tf, xf, of, str(algo)])
        assert r.returncode == 0, r.stderr
        np.testing.assert_array_equal(np.fromfile(of, dtype=np.int32), want,
                                      err_msg="algo %d" % algo)
    wf = W.config(5, n_samples=20_000)
    xf5 = wf.features()
    ff = str(tmp_path / "forest.bin")
    _forest_file(ff, wf.nodes, wf.tree_offsets, wf.n_features, wf.n_classes)
    _records_file(xf, xf5)
    want = oracle.forest_classes(wf.nodes, wf.tree_offsets, xf5, wf.n_features, wf.n_classes)
    for algo in (0, 1):
        r = _run([client, "forest", ff, xf, of, str(algo)])
        assert r.returncode == 0, r.stderr
        np.testing.assert_array_equal(np.fromfile(of, dtype=np.int32), want,
                                      err_msg="forest algo %d" % algo)

"""Narrow record types on the CPU: the widening that defines the expected labels is pinned
to torch's own dtype conversions, and the generators keep what they promise."""
import numpy as np
import pytest

from paper_1111_1373_amd import workloads as W
from tests import treeutil as TU

torch = pytest.importorskip("torch")


def _same_bits(a, b):
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))


def test_f16_widening_matches_torch():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)   # every binary16 value
    h = bits.view(np.float16)
    want = torch.from_numpy(h.copy()).float().numpy()
    got = TU.widen(h, "f16")
    nan = np.isnan(want)
    assert (np.isnan(got) == nan).all()
    _same_bits(got[~nan], want[~nan])


def test_bf16_widening_matches_torch():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)   # every bfloat16 value
    want = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    got = TU.widen(bits, "bf16")
    nan = np.isnan(want)
    assert (np.isnan(got) == nan).all()
    _same_bits(got[~nan], want[~nan])


def test_u8_widening_is_the_integer():
    v = np.arange(256, dtype=np.uint8)
    np.testing.assert_array_equal(TU.widen(v, "u8"), np.arange(256, dtype=np.float32))


@pytest.mark.parametrize("x_type", ["f16", "bf16"])
def test_narrowing_rounds_to_nearest_even_like_torch(x_type):
    r = np.random.Generator(np.random.PCG64(11))
    x = np.concatenate([W.uniform_f32(r, 100_000), W.normal_f32(r, 100_000) * np.float32(300),
                        np.float32([0.0, -0.0, 1.0, 65504.0, 65520.0, 1e-8])])
    dt = torch.float16 if x_type == "f16" else torch.bfloat16
    want = torch.from_numpy(x).to(dt).float().numpy()
    got = TU.widen(W.narrow_records(x, x_type), x_type)
    _same_bits(got, want)


def test_u8_quantisation_range_and_tree():
    w = W.config(2, n_samples=10_000)
    x = w.features()
    q = W.narrow_records(x, "u8")
    assert q.dtype == np.uint8 and q.min() == 0 and q.max() == 255
    np.testing.assert_array_equal(q, np.floor(x.astype(np.float64) * 256).astype(np.uint8))
    t = W.narrow_tree(w.nodes, "u8")
    inner = w.nodes["cls"] < 0
    np.testing.assert_array_equal(t["threshold"][inner], w.nodes["threshold"][inner] * 256)
    np.testing.assert_array_equal(t[["feature", "left", "cls"]], w.nodes[["feature", "left", "cls"]])
    qn = W.narrow_records(W.config(3, n_samples=10_000).features(), "u8", "normal")
    assert qn.min() == 0 and qn.max() == 255


def test_narrow_specials_widen_as_documented():
    f = TU.widen(TU.narrow_specials("f16"), "f16")
    assert f[2] == 2.0 ** -24 and np.signbit(f[1]) and np.isnan(f[10]) and f[6] == 65504.0
    b = TU.widen(TU.narrow_specials("bf16"), "bf16")
    assert b[2] == np.float32(np.ldexp(1.0, -133)) and np.isinf(b[8]) and np.isnan(b[10])
    assert b[11] == 1.0 and np.signbit(b[1])

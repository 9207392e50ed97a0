"""Python binding of the C ABI in ``include/dtree.h`` (ctypes; argument marshalling only).

Every evaluation step runs in the gfx950 kernels of ``libdtree.so``; this module only
converts arguments.  PyTorch supplies device memory and the current stream.  Importing
this module raises ``ImportError`` if the library has not been built
(``python -m paper_1111_1373_amd.build``): there is no other code path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

# torch ships its own HIP runtime (same SONAME as ROCm's libamdhip64.so.7).  Load it
# first so that libdtree.so binds to the very runtime that owns torch's device pointers
# and streams; two HIP runtimes in one process do not share devices.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdtree.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        "libdtree.so is not built; run `python -m paper_1111_1373_amd.build` "
        "(the GPU library has no fallback)")

_lib = ctypes.CDLL(LIB_PATH)

DT_OK, DT_ERR_INVALID_ARG, DT_ERR_INVALID_TREE, DT_ERR_UNSUPPORTED, DT_ERR_HIP, DT_ERR_NO_MEMORY = range(6)
ALGOS = {"data": 0, "speculative": 1, "path": 2}
OUT_KINDS = {"class_u8": 0, "class_i32": 1, "leaf_i32": 2}
X_TYPES = {"f32": 0, "f16": 1, "bf16": 2, "u8": 3}

NODE_DTYPE = np.dtype(
    [("feature", "<i4"), ("threshold", "<f4"), ("left", "<i4"), ("cls", "<i4")], align=False)


class TreeOptions(ctypes.Structure):
    _fields_ = [("data_window_depth", ctypes.c_int32), ("spec_window_depth", ctypes.c_int32),
                ("waves_per_cu", ctypes.c_int32), ("path_hops", ctypes.c_int32)]


class TreeInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_nodes", "n_internal", "n_leaves", "depth", "n_features", "n_classes",
        "data_window_depth", "data_windows", "data_levels",
        "spec_window_depth", "spec_windows", "spec_levels")] + [
        ("data_table_bytes", ctypes.c_int64), ("spec_table_bytes", ctypes.c_int64)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class PipelineOptions(ctypes.Structure):
    _fields_ = [("chunk_rows", ctypes.c_int64), ("n_slots", ctypes.c_int32),
                ("serial", ctypes.c_int32), ("host_threads", ctypes.c_int32)]


class PipelineStats(ctypes.Structure):
    _fields_ = [("outer_us", ctypes.c_double), ("kernel_us", ctypes.c_double),
                ("h2d_us", ctypes.c_double), ("d2h_us", ctypes.c_double),
                ("chunks", ctypes.c_int64), ("input_pinned", ctypes.c_int32),
                ("output_pinned", ctypes.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class LaunchInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "waves_per_workgroup", "workgroups_per_cu", "lds_bytes", "result_buffer_tiles",
        "tables_in_lds", "load_mode", "tile_rows")]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


_p, _i32, _i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
_PROTOS = {
    "dt_abi_version": (_i32, []),
    "dt_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "dt_last_error": (ctypes.c_char_p, []),
    "dt_tree_check": (ctypes.c_int, [_p, _i32, _i32, _i32, _p, _p]),
    "dt_encode_windows": (ctypes.c_int, [_p, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p]),
    "dt_threshold_keys": (ctypes.c_int, [_p, _i64, ctypes.c_int, _p]),
    "dt_tree_create": (ctypes.c_int, [_p, _i32, _i32, _i32, _p, _p]),
    "dt_tree_get_info": (ctypes.c_int, [_p, _p]),
    "dt_tree_destroy": (None, [_p]),
    "dt_tree_launch_info": (ctypes.c_int, [_p, _p, ctypes.c_int, _i64, ctypes.c_int, ctypes.c_int, _p]),
    "dt_classify": (ctypes.c_int, [_p, _p, _i64, _i64, _p, ctypes.c_int, ctypes.c_int, _p]),
    "dt_classify_typed": (ctypes.c_int, [_p, _p, ctypes.c_int, _i64, _i64, _p, ctypes.c_int,
                                         ctypes.c_int, _p]),
    "dt_forest_create": (ctypes.c_int, [_p, _p, _i32, _i32, _i32, _p, _p]),
    "dt_forest_destroy": (None, [_p]),
    "dt_forest_classify": (ctypes.c_int, [_p, _p, _i64, _i64, _p, ctypes.c_int, ctypes.c_int, _p]),
    "dt_probe_copy": (ctypes.c_int, [_p, _p, _i64, _p]),
    "dt_probe_read": (ctypes.c_int, [_p, _i64, _p, _i32, _p]),
    "dt_pipeline_create": (ctypes.c_int, [_i32, _p, _p]),
    "dt_pipeline_destroy": (None, [_p]),
    "dt_classify_host": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _p, ctypes.c_int, ctypes.c_int, _p]),
    "dt_forest_classify_host": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _p, ctypes.c_int, ctypes.c_int, _p]),
    "dt_classify_host_typed": (ctypes.c_int, [_p, _p, _p, ctypes.c_int, _i64, _i64, _p, ctypes.c_int,
                                              ctypes.c_int, _p]),
    "dt_classify_host_noalloc": (ctypes.c_int, [_p, _p, _i64, _i64, _p, ctypes.c_int, ctypes.c_int,
                                                _p]),
    "dt_noalloc_scratch_bytes": (_i64, []),
}
for _name, (_res, _args) in _PROTOS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

ABI_VERSION = _lib.dt_abi_version()


class DTreeError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib.dt_last_error().decode() or _lib.dt_status_string(status).decode()
        super().__init__("%s: %s (%s)" % (where, _lib.dt_status_string(status).decode(), msg))


def _check(status: int, where: str):
    if status != DT_OK:
        raise DTreeError(status, where)


def _nodes(nodes) -> np.ndarray:
    arr = np.ascontiguousarray(nodes)
    if arr.dtype != NODE_DTYPE:
        arr = np.ascontiguousarray(arr.astype(NODE_DTYPE))
    return arr


def _options(data_window_depth: int, spec_window_depth: int, waves_per_cu: int = 0,
             path_hops: int = 0) -> TreeOptions:
    return TreeOptions(int(data_window_depth), int(spec_window_depth), int(waves_per_cu),
                       int(path_hops))


def tree_check(nodes, n_features: int, n_classes: int, data_window_depth: int = 0,
               spec_window_depth: int = 0, waves_per_cu: int = 0, path_hops: int = 0) -> dict:
    """Validate a tree on the host and describe its encodings (no GPU needed)."""
    nd = _nodes(nodes)
    info = TreeInfo()
    opt = _options(data_window_depth, spec_window_depth, waves_per_cu, path_hops)
    _check(_lib.dt_tree_check(nd.ctypes.data, len(nd), n_features, n_classes,
                              ctypes.byref(opt), ctypes.byref(info)), "dt_tree_check")
    return info.as_dict()


def encode_windows(nodes, n_features: int, n_classes: int, window_depth: int) -> dict:
    """The window tables the kernels use (host only), as numpy arrays of
    shape [n_windows, 2**window_depth]."""
    nd = _nodes(nodes)
    nw, lv = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(_lib.dt_encode_windows(nd.ctypes.data, len(nd), n_features, n_classes, window_depth,
                                  0, None, None, None, None, ctypes.byref(nw), ctypes.byref(lv)),
           "dt_encode_windows")
    s = 1 << window_depth
    feat = np.empty((nw.value, s), dtype=np.int32)
    thr = np.empty((nw.value, s), dtype=np.float32)
    ec = np.empty((nw.value, s), dtype=np.int32)
    el = np.empty((nw.value, s), dtype=np.int32)
    _check(_lib.dt_encode_windows(nd.ctypes.data, len(nd), n_features, n_classes, window_depth,
                                  nw.value, feat.ctypes.data, thr.ctypes.data, ec.ctypes.data,
                                  el.ctypes.data, ctypes.byref(nw), ctypes.byref(lv)),
           "dt_encode_windows")
    return dict(feature=feat, threshold=thr, exit_class=ec, exit_leaf=el, levels=lv.value,
                n_windows=nw.value, depth=window_depth)


def threshold_keys(thresholds, x_type: str) -> np.ndarray:
    """Thresholds moved onto a narrow record type's grid, as the kernels compare them
    (host only): uint16 bits for "f16" / "bf16", integers 0..256 for "u8"."""
    t = np.ascontiguousarray(thresholds, dtype=np.float32).ravel()
    keys = np.empty(t.size, dtype=np.uint16)
    _check(_lib.dt_threshold_keys(t.ctypes.data, t.size, X_TYPES[x_type], keys.ctypes.data),
           "dt_threshold_keys")
    return keys


def _stream_handle(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _x_type(x) -> int:
    """dt_dtype of a record tensor: float32, float16, bfloat16 or uint8."""
    import torch
    types = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2, torch.uint8: 3}
    if x.dtype not in types:
        raise TypeError("records must be float32, float16, bfloat16 or uint8, not %s" % x.dtype)
    return types[x.dtype]


def _features_arg(x, n_features: int, typed: bool = False):
    import torch
    if not isinstance(x, torch.Tensor) or x.device.type != "cuda":
        raise TypeError("features must be a CUDA (HIP) torch tensor")
    if x.dim() != 2 or (not typed and x.dtype != torch.float32):
        raise TypeError("features must be a 2-D float32 tensor")
    if x.shape[1] < n_features:
        raise ValueError("features has %d columns, tree needs %d" % (x.shape[1], n_features))
    if x.stride(1) != 1:
        raise ValueError("feature rows must be contiguous (stride(1) == 1)")
    ld = x.stride(0) if x.shape[0] > 1 else max(x.shape[1], n_features)
    return x.data_ptr(), x.shape[0], ld


def _out_tensor(out, n: int, out_kind: str, device):
    import torch
    dtype = torch.uint8 if out_kind == "class_u8" else torch.int32
    if out is None:
        return torch.empty(n, dtype=dtype, device=device)
    if out.dtype != dtype or out.numel() != n or not out.is_contiguous() or out.device != device:
        raise ValueError("out must be a contiguous %s tensor of %d elements on %s" % (dtype, n, device))
    return out


class Tree:
    """A tree uploaded to the current device (``dt_tree_create``)."""

    def __init__(self, nodes, n_features: int, n_classes: int, data_window_depth: int = 0,
                 spec_window_depth: int = 0, waves_per_cu: int = 0, path_hops: int = 0):
        nd = _nodes(nodes)
        self.n_features = int(n_features)
        self.n_classes = int(n_classes)
        self._h = ctypes.c_void_p()
        opt = _options(data_window_depth, spec_window_depth, waves_per_cu, path_hops)
        _check(_lib.dt_tree_create(nd.ctypes.data, len(nd), n_features, n_classes,
                                   ctypes.byref(opt), ctypes.byref(self._h)), "dt_tree_create")

    @property
    def info(self) -> dict:
        info = TreeInfo()
        _check(_lib.dt_tree_get_info(self._h, ctypes.byref(info)), "dt_tree_get_info")
        return info.as_dict()

    def launch_info(self, x, algo: str = "data", out_kind: str = "class_u8") -> dict:
        """Launch shape classify() uses for ``x`` (diagnostic)."""
        ptr, _, ld = _features_arg(x, self.n_features, typed=True)
        info = LaunchInfo()
        _check(_lib.dt_tree_launch_info(self._h, ptr, _x_type(x), ld, OUT_KINDS[out_kind],
                                        ALGOS[algo], ctypes.byref(info)), "dt_tree_launch_info")
        return info.as_dict()

    def classify(self, x, algo: str = "data", out_kind: str = "class_u8", out=None, stream=None):
        """Labels (or leaf indices) of the rows of ``x`` (float32, float16, bfloat16 or uint8
        records); asynchronous on ``stream`` (default: torch's current stream)."""
        ptr, n, ld = _features_arg(x, self.n_features, typed=True)
        out = _out_tensor(out, n, out_kind, x.device)
        _check(_lib.dt_classify_typed(self._h, ptr, _x_type(x), n, ld,
                                      out.data_ptr() if n else None, OUT_KINDS[out_kind],
                                      ALGOS[algo], _stream_handle(stream)),
               "dt_classify_typed")
        return out

    def close(self):
        if self._h:
            _lib.dt_tree_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Forest:
    """A forest uploaded to the current device (``dt_forest_create``)."""

    def __init__(self, nodes, tree_offsets, n_features: int, n_classes: int,
                 data_window_depth: int = 0, spec_window_depth: int = 0, waves_per_cu: int = 0):
        nd = _nodes(nodes)
        off = np.ascontiguousarray(tree_offsets, dtype=np.int32)
        self.n_features = int(n_features)
        self.n_classes = int(n_classes)
        self._h = ctypes.c_void_p()
        opt = _options(data_window_depth, spec_window_depth, waves_per_cu)
        _check(_lib.dt_forest_create(nd.ctypes.data, off.ctypes.data, len(off) - 1, n_features,
                                     n_classes, ctypes.byref(opt), ctypes.byref(self._h)),
               "dt_forest_create")

    def classify(self, x, algo: str = "data", out_kind: str = "class_u8", out=None, stream=None):
        ptr, n, ld = _features_arg(x, self.n_features)
        out = _out_tensor(out, n, out_kind, x.device)
        _check(_lib.dt_forest_classify(self._h, ptr, n, ld, out.data_ptr() if n else None,
                                       OUT_KINDS[out_kind], ALGOS[algo], _stream_handle(stream)),
               "dt_forest_classify")
        return out

    def close(self):
        if self._h:
            _lib.dt_forest_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def probe_copy(src, dst, stream=None):
    """Streaming copy of ``src`` into ``dst`` (same byte size): counter calibration."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("size mismatch")
    _check(_lib.dt_probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, _stream_handle(stream)),
           "dt_probe_copy")


def _host_features_arg(x, n_features: int, x_type=None):
    """(pointer, rows, row stride in elements, dt_dtype) of a host record matrix (numpy or
    CPU tensor) of float32, float16, bfloat16 (torch, or numpy uint16 with x_type="bf16")
    or uint8."""
    import torch
    if isinstance(x, torch.Tensor):
        if x.device.type != "cpu":
            raise TypeError("host features must be a CPU tensor or a numpy array")
        if x.dim() != 2:
            raise TypeError("features must be a 2-D array")
        xt = _x_type(x)
        rows, cols, st0, st1, ptr = x.shape[0], x.shape[1], x.stride(0), x.stride(1), x.data_ptr()
    else:
        if not isinstance(x, np.ndarray) or x.ndim != 2:
            raise TypeError("features must be a 2-D array")
        kinds = {np.dtype(np.float32): 0, np.dtype(np.float16): 1, np.dtype(np.uint8): 3}
        if x.dtype == np.uint16 and x_type == "bf16":
            xt = 2
        elif x.dtype in kinds:
            xt = kinds[x.dtype]
        else:
            raise TypeError("host records must be float32, float16, uint8 or (with "
                            "x_type='bf16') uint16 bfloat16 bits, not %s" % x.dtype)
        es = x.dtype.itemsize
        rows, cols, ptr = x.shape[0], x.shape[1], x.ctypes.data
        if x.strides[0] % es or x.strides[1] % es:
            raise ValueError("feature strides must be whole elements")
        st0, st1 = x.strides[0] // es, x.strides[1] // es
    if x_type is not None and X_TYPES[x_type] != xt:
        raise TypeError("records are %s, not %s" % ({v: k for k, v in X_TYPES.items()}[xt], x_type))
    if cols < n_features:
        raise ValueError("features has %d columns, tree needs %d" % (cols, n_features))
    if st1 != 1 and cols > 1:
        raise ValueError("feature rows must be contiguous")
    ld = st0 if rows > 1 else max(cols, n_features)
    if ld < n_features:
        raise ValueError("row stride smaller than n_features")
    return ptr, rows, ld, xt


class Pipeline:
    """Classification of host-resident records (``dt_pipeline_create`` and
    ``dt_classify_host``): chunked copies overlapped with the kernels, or with
    ``serial=True`` per-call allocation and serial copies."""

    def __init__(self, n_features: int, chunk_rows: int = 0, n_slots: int = 0,
                 serial: bool = False, host_threads: int = 0):
        self.n_features = int(n_features)
        self._h = ctypes.c_void_p()
        opt = PipelineOptions(int(chunk_rows), int(n_slots), 1 if serial else 0, int(host_threads))
        _check(_lib.dt_pipeline_create(self.n_features, ctypes.byref(opt), ctypes.byref(self._h)),
               "dt_pipeline_create")
        self.last_stats = None

    def classify(self, model, x, algo: str = "data", out_kind: str = "class_u8", out=None,
                 x_type=None):
        """Labels of the rows of the host matrix ``x`` for a :class:`Tree` or :class:`Forest`,
        in ``out`` (host, allocated if None: numpy for numpy input, else a CPU tensor).
        Records may be float32, float16, bfloat16 or uint8 (trees; forests read float32).
        Timing of the call is left in ``self.last_stats``."""
        import torch
        ptr, n, ld, xt = _host_features_arg(x, self.n_features, x_type)
        np_dtype = np.uint8 if out_kind == "class_u8" else np.int32
        if out is None:
            out = (np.empty(n, dtype=np_dtype) if isinstance(x, np.ndarray)
                   else torch.empty(n, dtype=torch.uint8 if out_kind == "class_u8" else torch.int32))
        if isinstance(out, np.ndarray):
            if out.dtype != np_dtype or out.size != n or not out.flags.c_contiguous:
                raise ValueError("out must be a contiguous %s array of %d elements" % (np_dtype, n))
            optr = out.ctypes.data
        else:
            want = torch.uint8 if out_kind == "class_u8" else torch.int32
            if out.dtype != want or out.numel() != n or not out.is_contiguous() or out.device.type != "cpu":
                raise ValueError("out must be a contiguous CPU %s tensor of %d elements" % (want, n))
            optr = out.data_ptr()
        st = PipelineStats()
        if isinstance(model, Forest):
            if xt != 0:
                raise TypeError("forests classify float32 records")
            _check(_lib.dt_forest_classify_host(model._h, self._h, ptr if n else None, n, ld,
                                                optr if n else None, OUT_KINDS[out_kind],
                                                ALGOS[algo], ctypes.byref(st)),
                   "dt_forest_classify_host")
        elif xt == 0:
            _check(_lib.dt_classify_host(model._h, self._h, ptr if n else None, n, ld,
                                         optr if n else None, OUT_KINDS[out_kind], ALGOS[algo],
                                         ctypes.byref(st)), "dt_classify_host")
        else:
            _check(_lib.dt_classify_host_typed(model._h, self._h, ptr if n else None, xt, n, ld,
                                               optr if n else None, OUT_KINDS[out_kind],
                                               ALGOS[algo], ctypes.byref(st)),
                   "dt_classify_host_typed")
        self.last_stats = st.as_dict()
        return out

    def close(self):
        if self._h:
            _lib.dt_pipeline_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def noalloc_scratch_bytes() -> int:
    """Size in bytes of the per-device staging area of ``classify_host_noalloc``."""
    return int(_lib.dt_noalloc_scratch_bytes())


def classify_host_noalloc(tree, x, algo: str = "data", out_kind: str = "class_u8", out=None,
                          stream=None):
    """``dt_classify_host_noalloc``: labels of host-resident fp32 records (numpy or CPU
    tensor) staged through the library's fixed per-device area; returns a numpy array
    (or fills ``out``, a numpy array of n uint8 / int32)."""
    ptr, n, ld, xt = _host_features_arg(x, tree.n_features, "f32")
    dtype = np.uint8 if out_kind == "class_u8" else np.int32
    if out is None:
        out = np.empty(n, dtype=dtype)
    if not isinstance(out, np.ndarray) or out.dtype != dtype or out.shape != (n,) or \
            not out.flags.c_contiguous:
        raise TypeError("out must be a contiguous numpy array of %d %s" % (n, np.dtype(dtype)))
    _check(_lib.dt_classify_host_noalloc(tree._h, ptr if n else None, n, ld,
                                         out.ctypes.data if n else None, OUT_KINDS[out_kind],
                                         ALGOS[algo], _stream_handle(stream)),
           "dt_classify_host_noalloc")
    return out


def probe_read(src, sink, waves_per_cu: int = 8, stream=None):
    """Stream-read every byte of the device tensor ``src`` (one kernel); ``sink`` is a
    device int32 tensor the kernel never writes in practice.  Streaming-read ceiling."""
    nbytes = src.numel() * src.element_size()
    _check(_lib.dt_probe_read(src.data_ptr(), nbytes, sink.data_ptr(), int(waves_per_cu),
                              _stream_handle(stream)), "dt_probe_read")

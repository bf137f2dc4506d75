"""CPU oracle of the HPAC-ML surrogate-inference region (arXiv 2407.18352).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
(``paper_2407_18352_amd`` and its HIP library) never imports it, and it imports
nothing from the product.

The arithmetic lives in ``hpacml_oracle.c`` (plain C, fp64, scalar loops,
OpenMP over points only); this module marshals numpy arrays into it.  Specs are
plain data:

* map spec: ``{"rank": R, "slices": [(lo, count), ...],
  "sweep": (start, stop, step), "bnd": [b0, ...]}`` with ``bnd`` entries
  0 = none, 1 = periodic, 2 = clamp.  ``lo``/``count`` describe one right-hand
  side slice of a tensor functor (Sec. III-B, Fig. 2); the sweep is the concrete
  slice of a tensor map (Sec. III-C).
* targets: a list of float32 numpy arrays of one shape (the index space);
  strides are taken from the arrays.
* model spec: ``{"dims": [...], "W": [...], "b": [...], "act": [...],
  "compute": "f32" | "bf16"}`` with ``W[l]`` of shape ``[dims[l+1], dims[l]]``.
* convolutional model spec: ``{"kind": "cnn", "in_channels": C, "image": (H, W),
  "layers": [...]}``, each layer ``{"kind": "conv" | "pool" | "linear", "out",
  "kernel", "stride", "padding": "same" | "valid", "mode": "zeros" | "circular"
  | "replicate", "act", "W", "b"}`` (conv ``W`` is ``[out, in, kh, kw]``,
  linear ``W`` is ``[out, in]`` over the flattened [row][column][channel]
  input).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hpacml_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

MAX_RANK = 4
BND = {"none": 0, "periodic": 1, "clamp": 2}


def build(force: bool = False) -> str:
    """Compile ``liboracle.so`` with gcc (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-Wall", "-Wextra", "-Wno-unused-parameter",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Map(C.Structure):
    _fields_ = [("rank", C.c_int32), ("n_slices", C.c_int32), ("n_targets", C.c_int32),
                ("pad_", C.c_int32),
                ("lo", C.POINTER(C.c_int32)), ("count", C.POINTER(C.c_int32)),
                ("start", C.c_int64 * MAX_RANK), ("stop", C.c_int64 * MAX_RANK),
                ("step", C.c_int64 * MAX_RANK), ("bnd", C.c_int32 * MAX_RANK),
                ("extent", C.c_int64 * MAX_RANK),
                ("data", C.POINTER(C.c_void_p)), ("stride", C.POINTER(C.c_int64))]


class _Layer(C.Structure):
    _fields_ = [("kind", C.c_int32), ("out_channels", C.c_int32), ("kh", C.c_int32), ("kw", C.c_int32),
                ("sh", C.c_int32), ("sw", C.c_int32), ("padding", C.c_int32), ("pad_mode", C.c_int32),
                ("act", C.c_int32), ("pad_", C.c_int32),
                ("W", C.POINTER(C.c_float)), ("b", C.POINTER(C.c_float))]


LAYER_KIND = {"conv": 0, "pool": 1, "linear": 2}
PADDING = {"valid": 0, "same": 1}
PAD_MODE = {"zeros": 0, "circular": 1, "replicate": 2}


class _Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("bf16", C.c_int32),
                ("dims", C.POINTER(C.c_int32)), ("W", C.POINTER(C.POINTER(C.c_float))),
                ("b", C.POINTER(C.POINTER(C.c_float))), ("act", C.POINTER(C.c_int32))]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build()
            L = C.CDLL(_LIB)
            P = C.POINTER
            L.or_num_threads.restype = C.c_int
            L.or_set_num_threads.argtypes = [C.c_int]
            L.or_set_num_threads.restype = None
            L.or_bf16_bits.argtypes = [P(C.c_float), P(C.c_uint16), C.c_int64]
            L.or_map_points.argtypes = [P(_Map)]
            L.or_map_points.restype = C.c_int64
            L.or_map_features.argtypes = [P(_Map)]
            L.or_map_features.restype = C.c_int32
            L.or_point_coords.argtypes = [P(_Map), C.c_int64, P(C.c_int64)]
            L.or_gather.argtypes = [P(_Map), P(C.c_int64), C.c_int64, P(C.c_double)]
            L.or_collect.argtypes = [P(_Map), P(C.c_int64), C.c_int64, P(C.c_uint32), C.c_int64]
            L.or_mlp.argtypes = [P(_Model), P(C.c_double), C.c_int64, P(C.c_float)]
            L.or_infer_rows.argtypes = [P(_Map), P(_Model), P(C.c_int64), C.c_int64, P(C.c_float)]
            L.or_scatter.argtypes = [P(_Map), P(C.c_int64), C.c_int64, P(C.c_float)]
            L.or_cnn_shapes.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, P(_Layer), P(C.c_int32)]
            L.or_cnn.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, P(_Layer), P(C.c_double),
                                 C.c_int64, P(C.c_float)]
            for fn in (L.or_gather, L.or_collect, L.or_mlp, L.or_infer_rows, L.or_scatter, L.or_cnn_shapes,
                       L.or_cnn):
                fn.restype = C.c_int
            _lib = L
    return _lib


def num_threads() -> int:
    return lib().or_num_threads()


def set_num_threads(n: int) -> None:
    """Threads used by later oracle calls (timing only: every result is
    independent of the thread count)."""
    lib().or_set_num_threads(int(n))


def _ptr(a, ct):
    return a.ctypes.data_as(C.POINTER(ct))


class _Keep:
    """Holds the ctypes structure and every buffer it points into."""

    def __init__(self, struct, *refs):
        self.s = struct
        self.refs = refs


def _bnd_code(b):
    return BND[b] if isinstance(b, str) else int(b)


def _map(spec, targets) -> _Keep:
    R = int(spec["rank"])
    if not 1 <= R <= MAX_RANK:
        raise ValueError("rank must be 1..4")
    slices = spec["slices"]
    lo = np.zeros((max(len(slices), 1), 4), np.int32)
    cnt = np.ones((max(len(slices), 1), 4), np.int32)
    for s, (l, c) in enumerate(slices):
        lo[s, :R] = l
        cnt[s, :R] = c
    shape = targets[0].shape
    stride = np.zeros((len(targets), 4), np.int64)
    for t, a in enumerate(targets):
        if a.dtype != np.float32 or a.shape != shape:
            raise ValueError("targets must be float32 arrays of one shape")
        stride[t, :R] = [s // 4 for s in a.strides]
    data = (C.c_void_p * max(len(targets), 1))(*[a.ctypes.data for a in targets])
    m = _Map()
    m.rank, m.n_slices, m.n_targets = R, len(slices), len(targets)
    m.lo, m.count = _ptr(lo, C.c_int32), _ptr(cnt, C.c_int32)
    start, stop, step = spec["sweep"]
    bnd = spec.get("bnd", [0] * R)
    for d in range(R):
        m.start[d], m.stop[d], m.step[d] = int(start[d]), int(stop[d]), int(step[d])
        m.bnd[d] = _bnd_code(bnd[d])
        m.extent[d] = shape[d]
    m.data = C.cast(data, C.POINTER(C.c_void_p))
    m.stride = _ptr(stride, C.c_int64)
    return _Keep(m, lo, cnt, stride, data, targets)


def _model(spec) -> _Keep:
    L = len(spec["W"])
    dims = np.asarray(spec["dims"], np.int32)
    Ws = [np.ascontiguousarray(w, np.float32) for w in spec["W"]]
    bs = [np.ascontiguousarray(b, np.float32) for b in spec["b"]]
    for l in range(L):
        assert Ws[l].shape == (dims[l + 1], dims[l]) and bs[l].shape == (dims[l + 1],)
    act = np.asarray(spec["act"], np.int32)
    Wp = (C.POINTER(C.c_float) * L)(*[_ptr(w, C.c_float) for w in Ws])
    bp = (C.POINTER(C.c_float) * L)(*[_ptr(b, C.c_float) for b in bs])
    m = _Model()
    m.n_layers = L
    m.bf16 = 1 if spec.get("compute", "f32") == "bf16" else 0
    m.dims, m.act = _ptr(dims, C.c_int32), _ptr(act, C.c_int32)
    m.W = C.cast(Wp, C.POINTER(C.POINTER(C.c_float)))
    m.b = C.cast(bp, C.POINTER(C.POINTER(C.c_float)))
    return _Keep(m, dims, Ws, bs, act, Wp, bp)


def _layers(model) -> _Keep:
    Ls = model["layers"]
    arr = (_Layer * len(Ls))()
    keep = []
    for i, ly in enumerate(Ls):
        a = arr[i]
        a.kind = LAYER_KIND[ly["kind"]]
        a.out_channels = int(ly.get("out", 0))
        a.kh, a.kw = (int(v) for v in ly.get("kernel", (1, 1)))
        # default steps: 1 for a convolution, the window for a pool (PyTorch's defaults)
        a.sh, a.sw = (int(v) for v in ly.get("stride", ly.get("kernel") if ly["kind"] == "pool" else (1, 1)))
        a.padding = PADDING[ly.get("padding", "valid")]
        a.pad_mode = PAD_MODE[ly.get("mode", "zeros")]
        a.act = int(ly.get("act", 0))
        if ly["kind"] != "pool":
            W = np.ascontiguousarray(ly["W"], np.float32)
            b = np.ascontiguousarray(ly["b"], np.float32)
            keep += [W, b]
            a.W, a.b = _ptr(W, C.c_float), _ptr(b, C.c_float)
    return _Keep(arr, keep)


def cnn_shapes(model) -> list:
    """(rows, columns, channels) of every layer's input and of the output."""
    k = _layers(model)
    L = len(model["layers"])
    sh = np.zeros(3 * (L + 1), np.int32)
    H, W = model["image"]
    _check(lib().or_cnn_shapes(model["in_channels"], H, W, L, k.s, _ptr(sh, C.c_int32)), "cnn shapes")
    return [tuple(int(v) for v in sh[3 * l: 3 * l + 3]) for l in range(L + 1)]


def cnn(model, X) -> np.ndarray:
    """Convolutional model on composed tensors X[S*H*W, C] (S images in sweep
    order) -> float32 Y[S*H'*W', C']."""
    k = _layers(model)
    L = len(model["layers"])
    H, W = model["image"]
    C0 = model["in_channels"]
    X = np.ascontiguousarray(X, np.float64)
    assert X.ndim == 2 and X.shape[1] == C0 and X.shape[0] % (H * W) == 0
    S = X.shape[0] // (H * W)
    h2, w2, c2 = cnn_shapes(model)[-1]
    Y = np.zeros((S * h2 * w2, c2), np.float32)
    _check(lib().or_cnn(C0, H, W, L, k.s, _ptr(X, C.c_double), S, _ptr(Y, C.c_float)), "cnn")
    return Y


def _rows(rows):
    if rows is None:
        return None, None
    r = np.ascontiguousarray(rows, np.int64)
    return r, _ptr(r, C.c_int64)


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle %s failed (code %d)" % (what, rc))


def n_points(spec, targets) -> int:
    k = _map(spec, targets)
    return int(lib().or_map_points(C.byref(k.s)))


def n_features(spec, targets) -> int:
    k = _map(spec, targets)
    return int(lib().or_map_features(C.byref(k.s)))


def point_coords(spec, targets, b) -> tuple:
    k = _map(spec, targets)
    p = np.zeros(4, np.int64)
    lib().or_point_coords(C.byref(k.s), int(b), _ptr(p, C.c_int64))
    return tuple(int(v) for v in p[: spec["rank"]])


def gather(spec, targets, rows=None) -> np.ndarray:
    """Composed input tensor X[n, F] in fp64 (Sec. IV-A, Tensor Composition)."""
    k = _map(spec, targets)
    B = int(lib().or_map_points(C.byref(k.s)))
    F = int(lib().or_map_features(C.byref(k.s)))
    r, rp = _rows(rows)
    n = B if r is None else len(r)
    X = np.zeros((n, F), np.float64)
    _check(lib().or_gather(C.byref(k.s), rp, n, _ptr(X, C.c_double)), "gather")
    return X


def collect(spec, targets, ld=None, rows=None) -> np.ndarray:
    """Record rows [n, ld] of 32-bit patterns (uint32); columns >= F stay 0."""
    k = _map(spec, targets)
    B = int(lib().or_map_points(C.byref(k.s)))
    F = int(lib().or_map_features(C.byref(k.s)))
    ld = F if ld is None else int(ld)
    r, rp = _rows(rows)
    n = B if r is None else len(r)
    D = np.zeros((n, max(ld, 1)), np.uint32)
    _check(lib().or_collect(C.byref(k.s), rp, n, _ptr(D, C.c_uint32), ld), "collect")
    return D[:, :ld]


def mlp(model, X) -> np.ndarray:
    """Model forward on a composed tensor X[n, dims[0]] -> float32 Y[n, dims[-1]]."""
    k = _model(model)
    X = np.ascontiguousarray(X, np.float64)
    dims = model["dims"]
    assert X.ndim == 2 and X.shape[1] == dims[0]
    Y = np.zeros((X.shape[0], dims[-1]), np.float32)
    _check(lib().or_mlp(C.byref(k.s), _ptr(X, C.c_double), X.shape[0], _ptr(Y, C.c_float)), "mlp")
    return Y


def infer_rows(in_spec, in_targets, model, rows=None) -> np.ndarray:
    """Model outputs Y[n, dims[-1]] for the listed sweep rows (no scatter)."""
    km = _map(in_spec, in_targets)
    kd = _model(model)
    B = int(lib().or_map_points(C.byref(km.s)))
    r, rp = _rows(rows)
    n = B if r is None else len(r)
    Y = np.zeros((n, model["dims"][-1]), np.float32)
    _check(lib().or_infer_rows(C.byref(km.s), C.byref(kd.s), rp, n, _ptr(Y, C.c_float)), "infer")
    return Y


def scatter(spec, targets, Y, rows=None) -> None:
    """Write Y[n, F] through a `from` map into ``targets`` (modified in place)."""
    k = _map(spec, targets)
    Y = np.ascontiguousarray(Y, np.float32)
    r, rp = _rows(rows)
    n = Y.shape[0]
    _check(lib().or_scatter(C.byref(k.s), rp, n, _ptr(Y, C.c_float)), "scatter")


def infer(in_spec, in_targets, out_spec, out_targets, model) -> np.ndarray:
    """The whole region: every gather, then the model, then every scatter.
    Returns Y and writes the `from` targets in place."""
    if model.get("kind") == "cnn":
        Y = cnn(model, gather(in_spec, in_targets))
    else:
        Y = infer_rows(in_spec, in_targets, model)
    scatter(out_spec, out_targets, Y)
    return Y


def bf16_bits(x) -> np.ndarray:
    """bf16 (round to nearest even) bit patterns of float32 values."""
    x = np.ascontiguousarray(x, np.float32)
    out = np.zeros(x.shape, np.uint16)
    lib().or_bf16_bits(_ptr(x, C.c_float), _ptr(out, C.c_uint16), x.size)
    return out

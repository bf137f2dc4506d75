"""Python binding of the C ABI, with torch tensors as device memory.

Argument marshalling only: descriptors are filled from plain-data specs and
tensor metadata, and the calls go straight to ``libhpacml.so``.  Specs have the
form ``{"rank", "slices": [(lo, count), ...], "sweep": (start, stop, step),
"bnd": [...]}`` (one right-hand-side slice per entry, Sec. III-B; the sweep is
the concrete slice of a tensor map, Sec. III-C).
"""
from __future__ import annotations

import ctypes as C

from . import _abi
from ._abi import check, lib


def _functor(spec, n_targets, n_features=None):
    R = min(max(int(spec["rank"]), 0), _abi.MAX_RANK)
    slices = spec["slices"]
    arr = (_abi.Slice * max(1, len(slices)))()
    per = 0
    for s, (lo, cnt) in enumerate(slices):
        e = 1
        for d in range(_abi.MAX_RANK):
            arr[s].lo[d] = int(lo[d]) if d < R else 0
            arr[s].count[d] = int(cnt[d]) if d < R else 1
            if d < R:
                e *= int(cnt[d])
        per += e
    f = _abi.Functor()
    f.rank, f.n_slices = int(spec["rank"]), len(slices)
    f.slices = C.cast(arr, C.POINTER(_abi.Slice))
    f.n_features = per * n_targets if n_features is None else int(n_features)
    return f, arr


def _sweep(spec):
    R = min(max(int(spec["rank"]), 0), _abi.MAX_RANK)
    sw = _abi.Sweep()
    start, stop, step = spec["sweep"]
    for d in range(_abi.MAX_RANK):
        sw.start[d] = int(start[d]) if d < R else 0
        sw.stop[d] = int(stop[d]) if d < R else 1
        sw.step[d] = int(step[d]) if d < R else 1
    bl = [int(b) for b in spec.get("bnd", [0] * R)][:R]
    bnd = (C.c_int32 * _abi.MAX_RANK)(*(bl + [0] * (_abi.MAX_RANK - len(bl))))
    return sw, bnd


def array_desc(data_ptr: int, shape, strides, dtype: int = _abi.F32):
    """An ``hpacml_array`` from raw metadata (strides in elements)."""
    a = _abi.Array()
    a.data = C.c_void_p(int(data_ptr))
    a.dtype = dtype
    a.reserved = 0
    for d in range(_abi.MAX_RANK):
        a.extent[d] = int(shape[d]) if d < len(shape) else 1
        a.stride[d] = int(strides[d]) if d < len(strides) else 0
    return a


def _tensor_desc(t):
    import torch
    if t.dtype != torch.float32:
        raise TypeError("map targets must be float32 tensors")
    return array_desc(t.data_ptr(), tuple(t.shape), tuple(t.stride()))


def validate_map(spec, arrays, direction: int, n_features=None):
    """``hpacml_map_validate`` on descriptors (no device access).  ``arrays`` are
    ``hpacml_array`` structures (see ``array_desc``).  Returns
    ``(status, n_points, n_features)``."""
    f, keep = _functor(spec, len(arrays), n_features)
    sw, bnd = _sweep(spec)
    tarr = (_abi.Array * max(1, len(arrays)))(*arrays)
    npts, nfeat = C.c_int64(-1), C.c_int32(-1)
    st = lib().hpacml_map_validate(C.byref(f), direction, tarr, len(arrays), C.byref(sw), bnd,
                                   C.byref(npts), C.byref(nfeat))
    return st, npts.value, nfeat.value


def validate_model(dims, act, compute: int):
    L = len(dims) - 1
    d = (C.c_int32 * len(dims))(*dims)
    a = (C.c_int32 * max(1, len(act)))(*act)
    return lib().hpacml_model_validate(L, d, a, compute)


class Map:
    """A tensor map over torch tensors (device memory is borrowed: keep the
    tensors alive while work that uses the map is in flight)."""

    def __init__(self, spec, targets, direction: int, n_features=None):
        self.targets = list(targets)
        f, keep = _functor(spec, len(self.targets), n_features)
        sw, bnd = _sweep(spec)
        tarr = (_abi.Array * max(1, len(self.targets)))(*[_tensor_desc(t) for t in self.targets])
        h = C.c_void_p()
        check(lib().hpacml_map_create(C.byref(f), direction, tarr, len(self.targets), C.byref(sw), bnd,
                                      C.byref(h)), "hpacml_map_create")
        self.handle = h
        npts, nfeat = C.c_int64(), C.c_int32()
        check(lib().hpacml_map_shape(h, C.byref(npts), C.byref(nfeat)), "hpacml_map_shape")
        self.n_points, self.n_features = npts.value, nfeat.value

    def close(self):
        if getattr(self, "handle", None):
            lib().hpacml_map_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Model:
    """A surrogate MLP; weights are host fp32 arrays [out][in] (numpy or torch
    CPU), copied into library-owned device memory."""

    def __init__(self, spec):
        import numpy as np
        dims = [int(x) for x in spec["dims"]]
        L = len(dims) - 1
        self.W = [np.ascontiguousarray(np.asarray(w, dtype=np.float32)) for w in spec["W"]]
        self.b = [np.ascontiguousarray(np.asarray(b, dtype=np.float32)) for b in spec["b"]]
        # the library reads dims[l+1] x dims[l] weights through a plain pointer:
        # arrays of another size are refused here (invalid dims are left to
        # the library's own status)
        if len(self.W) != L or len(self.b) != L:
            raise ValueError("model spec: %d weight and %d bias arrays for %d layers" % (len(self.W), len(self.b), L))
        if min(dims) > 0:
            for l in range(L):
                if self.W[l].size != dims[l + 1] * dims[l] or self.b[l].size != dims[l + 1]:
                    raise ValueError("layer %d: weights of %d and biases of %d values, expected %d x %d and %d"
                                     % (l, self.W[l].size, self.b[l].size, dims[l + 1], dims[l], dims[l + 1]))
        Wp = (C.POINTER(C.c_float) * L)(*[w.ctypes.data_as(C.POINTER(C.c_float)) for w in self.W])
        bp = (C.POINTER(C.c_float) * L)(*[b.ctypes.data_as(C.POINTER(C.c_float)) for b in self.b])
        d = (C.c_int32 * (L + 1))(*dims)
        a = (C.c_int32 * L)(*[int(x) for x in spec["act"]])
        compute = _abi.BF16 if spec.get("compute", "f32") == "bf16" else _abi.F32
        h = C.c_void_p()
        check(lib().hpacml_model_create(L, d, Wp, bp, a, compute, C.byref(h)), "hpacml_model_create")
        self.handle = h
        self.dims = dims

    def close(self):
        if getattr(self, "handle", None):
            lib().hpacml_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


_KIND = {"conv": _abi.LAYER_CONV2D, "pool": _abi.LAYER_MAXPOOL2D, "linear": _abi.LAYER_LINEAR}
_PADDING = {"valid": _abi.PAD_VALID, "same": _abi.PAD_SAME}
_PAD_MODE = {"zeros": _abi.PADMODE_ZEROS, "circular": _abi.PADMODE_CIRCULAR, "replicate": _abi.PADMODE_REPLICATE}


def _layers(spec):
    """``hpacml_layer`` array from a convolutional model spec."""
    Ls = spec["layers"]
    arr = (_abi.Layer * len(Ls))()
    for i, ly in enumerate(Ls):
        a = arr[i]
        a.kind = _KIND[ly["kind"]]
        a.out_channels = int(ly.get("out", 0))
        k = ly.get("kernel", (1, 1))
        st = ly.get("stride", k if ly["kind"] == "pool" else (1, 1))
        a.kernel[0], a.kernel[1] = int(k[0]), int(k[1])
        a.stride[0], a.stride[1] = int(st[0]), int(st[1])
        a.padding = _PADDING[ly.get("padding", "valid")]
        a.pad_mode = _PAD_MODE[ly.get("mode", "zeros")]
        a.act = int(ly.get("act", 0))
    return arr


def validate_cnn(spec):
    """``hpacml_cnn_validate``: (status, output (rows, columns, channels))."""
    H, W = spec["image"]
    arr = _layers(spec)
    shp = (C.c_int32 * 3)()
    st = lib().hpacml_cnn_validate(int(spec["in_channels"]), int(H), int(W), len(spec["layers"]), arr, shp)
    return st, tuple(shp)


class CnnModel:
    """A convolutional surrogate (convolution / max-pool / fully connected
    layers on the composed tensor seen as images); spec as in
    ``workloads.make_cnn``.  Weights are host fp32 arrays, copied into
    library-owned device memory."""

    def __init__(self, spec):
        import numpy as np
        Ls = spec["layers"]
        L = len(Ls)
        arr = _layers(spec)
        self.W = [None if ly["kind"] == "pool" else np.ascontiguousarray(np.asarray(ly["W"], np.float32))
                  for ly in Ls]
        self.b = [None if ly["kind"] == "pool" else np.ascontiguousarray(np.asarray(ly["b"], np.float32))
                  for ly in Ls]
        # weight and bias sizes per layer, as the library reads them (for a
        # description it rejects, its own status reports the error below)
        wc, bc = (C.c_int64 * L)(), (C.c_int64 * L)()
        H, W = spec["image"]
        if lib().hpacml_cnn_param_counts(int(spec["in_channels"]), int(H), int(W), L, arr, wc, bc) == _abi.OK:
            for l in range(L):
                nw = 0 if self.W[l] is None else self.W[l].size
                nb = 0 if self.b[l] is None else self.b[l].size
                if nw != wc[l] or nb != bc[l]:
                    raise ValueError("layer %d: weights of %d and biases of %d values, expected %d and %d"
                                     % (l, nw, nb, wc[l], bc[l]))
        null = C.POINTER(C.c_float)()
        Wp = (C.POINTER(C.c_float) * L)(*[null if w is None else w.ctypes.data_as(C.POINTER(C.c_float))
                                          for w in self.W])
        bp = (C.POINTER(C.c_float) * L)(*[null if b is None else b.ctypes.data_as(C.POINTER(C.c_float))
                                          for b in self.b])
        H, W = spec["image"]
        h = C.c_void_p()
        check(lib().hpacml_cnn_create(int(spec["in_channels"]), int(H), int(W), L, arr, Wp, bp, _abi.F32,
                                      C.byref(h)), "hpacml_cnn_create")
        self.handle = h

    close = Model.close
    __del__ = Model.__del__


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def infer(model: Model, in_map: Map, out_map: Map, stream=None) -> None:
    """``hpacml_infer``: gather -> MLP -> scatter on ``stream`` (default: torch's
    current stream)."""
    check(lib().hpacml_infer(model.handle, in_map.handle, out_map.handle, _stream(stream)), "hpacml_infer")


def collect(m: Map, dst, ld: int, stream=None) -> None:
    """``hpacml_collect`` into ``dst`` (a float32 device tensor; ``dst`` may be a
    view offset into a larger record, e.g. ``rec[:, 9:]``)."""
    import torch
    if dst.dtype != torch.float32 or not dst.is_cuda:
        raise TypeError("collect destination must be a float32 device tensor")
    check(lib().hpacml_collect(m.handle, C.c_void_p(dst.data_ptr()), int(ld), _stream(stream)),
          "hpacml_collect")


def collect_pair(a: Map, dst_a, ld_a: int, b: Map, dst_b, ld_b: int, stream=None) -> None:
    """``hpacml_collect_pair``: both records of a region in one call (float32
    device tensors or views)."""
    import torch
    for d in (dst_a, dst_b):
        if d.dtype != torch.float32 or not d.is_cuda:
            raise TypeError("collect destinations must be float32 device tensors")
    check(lib().hpacml_collect_pair(a.handle, C.c_void_p(dst_a.data_ptr()), int(ld_a), b.handle,
                                    C.c_void_p(dst_b.data_ptr()), int(ld_b), _stream(stream)),
          "hpacml_collect_pair")


def variant(model: Model, in_map: Map, out_map: Map) -> str:
    r = lib().hpacml_infer_variant(model.handle, in_map.handle, out_map.handle)
    return r.decode() if r else None


class Region:
    """Execution control of one annotated region (``ml(infer | collect |
    predicated)`` and ``if``): ``run`` infers, or records the inputs, calls
    ``accurate(stream_handle)`` (the region's original code, which enqueues its
    work on that stream) and records the outputs and the accurate path's time
    into a sink of ``capacity`` samples."""

    def __init__(self, model, in_map: Map, out_map: Map, mode: int, capacity: int = 0):
        h = C.c_void_p()
        check(lib().hpacml_region_create(model.handle, in_map.handle, out_map.handle, int(mode), int(capacity),
                                         C.byref(h)), "hpacml_region_create")
        self.handle = h
        self.keep = (model, in_map, out_map)
        self.points, self.f_in = in_map.n_points, in_map.n_features
        self.points_out, self.f_out = out_map.n_points, out_map.n_features

    def run(self, accurate=None, cond: bool = True, enabled: bool = True, stream=None) -> None:
        """``accurate(stream_handle)`` gets the stream as an int (0: the null
        stream); an exception it raises is re-raised here once the library
        call has returned."""
        errors = []

        def call(user, st):
            try:
                accurate(st or 0)
            except BaseException as e:   # must not unwind through the C frame
                errors.append(e)
        cb = _abi.ACCURATE_FN(call) if accurate is not None else _abi.ACCURATE_FN()
        check(lib().hpacml_region_run(self.handle, 1 if cond else 0, 1 if enabled else 0, cb, None,
                                      _stream(stream)), "hpacml_region_run")
        if errors:
            raise errors[0]

    @property
    def samples(self) -> int:
        n = C.c_int64()
        check(lib().hpacml_region_samples(self.handle, C.byref(n)), "hpacml_region_samples")
        return n.value

    def read(self):
        """(inputs [n, points, F_in], outputs [n, points_out, F_out], times_ms [n]) as numpy."""
        import numpy as np
        n = self.samples
        ins = np.zeros((n, self.points, self.f_in), np.float32)
        outs = np.zeros((n, self.points_out, self.f_out), np.float32)
        t = np.zeros(n, np.float32)
        check(lib().hpacml_region_read(self.handle, n, ins.ctypes.data, outs.ctypes.data, t.ctypes.data),
              "hpacml_region_read")
        return ins, outs, t

    def save(self, directory: str, name: str) -> None:
        check(lib().hpacml_region_save(self.handle, directory.encode(), name.encode()), "hpacml_region_save")

    def reset(self) -> None:
        check(lib().hpacml_region_reset(self.handle), "hpacml_region_reset")

    def close(self):
        if getattr(self, "handle", None):
            lib().hpacml_region_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

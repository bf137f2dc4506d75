"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol the header declares, and every descriptor error is reported
before anything reaches a device."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2407_18352_amd import _abi, api
from paper_2407_18352_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hpacml.h")

FAKE = 0x10000000  # never dereferenced: validation does not touch data


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hpacml_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) == 24
    L = C.CDLL(_abi.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_abi.SIGNATURES)
    out = subprocess.run(["nm", "-D", "--defined-only", _abi.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\b(hpacml_\w+)\b", out))
    assert exported == set(names)


def test_version_and_status_strings():
    L = _abi.lib()
    assert L.hpacml_abi_version() == 2
    for s in range(8):
        assert L.hpacml_status_string(s)
    assert L.hpacml_status_string(0) == b"ok"


def _arr(shape, strides=None, ptr=FAKE, dtype=_abi.F32):
    if strides is None:
        strides, acc = [], 1
        for n in reversed(shape):
            strides.insert(0, acc)
            acc *= n
    return api.array_desc(ptr, shape, strides, dtype)


def test_validate_accepts_the_five_configurations():
    for name, (spec_in, spec_out, shape, n_in, n_out, F) in {
        "options": (wl.pointwise_spec(65536), wl.pointwise_spec(65536), (65536,), 5, 1, 5),
        "bonds": (wl.pointwise_spec(1 << 20), wl.pointwise_spec(1 << 20), (1 << 20,), 9, 1, 9),
        "stencil2d": (wl.window2d_spec(2048, 2048), wl.point2d_spec(2048, 2048), (2048, 2048), 4, 4, 36),
        "poses": (wl.pointwise_spec(1 << 22), wl.pointwise_spec(1 << 22), (1 << 22,), 6, 1, 6),
        "stencil3d": (wl.sevenpoint3d_spec(512, 512, 512), wl.point3d_spec(512, 512, 512),
                      (512, 512, 512), 5, 5, 35),
    }.items():
        st, n, f = api.validate_map(spec_in, [_arr(shape, ptr=FAKE + 0x1000000 * k) for k in range(n_in)],
                                    _abi.TO)
        assert st == _abi.OK and f == F, name
        npts = 1
        for x in shape:
            npts *= x
        assert n == npts
        st, n2, g = api.validate_map(spec_out, [_arr(shape)] * n_out if n_out == 1 else
                                     [_arr(shape, ptr=FAKE + 0x4000000 * k) for k in range(n_out)], _abi.FROM)
        assert st == _abi.OK and n2 == npts and g == n_out, name


def test_paper_example_counts():
    # ifnctr on t[1:N-1, 1:M-1] -> [N-2, M-2, 5]  (Fig. 2)
    N, M = 10, 12
    spec = {"rank": 2, "slices": [((-1, 0), (1, 1)), ((1, 0), (1, 1)), ((0, -1), (1, 3))],
            "sweep": ((1, 1), (N - 1, M - 1), (1, 1)), "bnd": [0, 0]}
    st, n, f = api.validate_map(spec, [_arr((N, M))], _abi.TO)
    assert (st, n, f) == (_abi.OK, (N - 2) * (M - 2), 5)
    # the full range reads outside the array without a boundary mode
    spec["sweep"] = ((0, 0), (N, M), (1, 1))
    assert api.validate_map(spec, [_arr((N, M))], _abi.TO)[0] == _abi.E_RANGE
    spec["bnd"] = [wl.PERIODIC, wl.CLAMP]
    assert api.validate_map(spec, [_arr((N, M))], _abi.TO)[0] == _abi.OK


def test_steps_and_empty_sweeps():
    spec = {"rank": 2, "slices": [((0, 0), (1, 1))], "sweep": ((1, 0), (6, 4), (2, 3)), "bnd": [0, 0]}
    assert api.validate_map(spec, [_arr((6, 4))], _abi.TO)[1] == 6
    spec["sweep"] = ((3, 0), (3, 4), (1, 1))
    assert api.validate_map(spec, [_arr((6, 4))], _abi.TO)[:2] == (_abi.OK, 0)
    # empty sweep: no access happens, so offsets outside are not an error
    spec["slices"] = [((-5, 0), (1, 1))]
    assert api.validate_map(spec, [_arr((6, 4))], _abi.TO)[0] == _abi.OK


@pytest.mark.parametrize("case, status", [
    ("rank0", _abi.E_INVAL), ("rank5", _abi.E_INVAL), ("count0", _abi.E_INVAL),
    ("nfeat", _abi.E_SHAPE), ("extent_mismatch", _abi.E_SHAPE), ("dtype", _abi.E_UNSUPPORTED),
    ("null_data", _abi.E_INVAL), ("neg_stride", _abi.E_INVAL), ("step0", _abi.E_INVAL),
    ("stop_gt_extent", _abi.E_RANGE), ("start_gt_stop", _abi.E_RANGE), ("bnd_bad", _abi.E_INVAL),
    ("range_none", _abi.E_RANGE), ("dir_bad", _abi.E_INVAL), ("from_window", _abi.E_UNSUPPORTED),
    ("from_two_slices", _abi.E_UNSUPPORTED), ("from_clamp_offset", _abi.E_INVAL),
    ("too_many_features", _abi.E_UNSUPPORTED), ("reserved", _abi.E_INVAL),
    ("no_targets", _abi.E_INVAL),
])
def test_map_validation_errors(case, status):
    spec = wl.window2d_spec(8, 8)
    arrays = [_arr((8, 8))]
    direction = _abi.TO
    nf = None
    if case == "rank0":
        spec = dict(spec, rank=0)
    elif case == "rank5":
        spec = dict(spec, rank=5, slices=[((0,) * 5, (1,) * 5)], sweep=((0,) * 5, (1,) * 5, (1,) * 5),
                    bnd=[0] * 5)
        arrays = [_arr((1, 1, 1, 1))]
    elif case == "count0":
        spec = dict(spec, slices=[((0, 0), (1, 0))])
    elif case == "nfeat":
        nf = 10
    elif case == "extent_mismatch":
        arrays = [_arr((8, 8)), _arr((8, 9))]
    elif case == "dtype":
        arrays = [_arr((8, 8), dtype=_abi.BF16)]
    elif case == "null_data":
        arrays = [_arr((8, 8), ptr=0)]
    elif case == "neg_stride":
        arrays = [_arr((8, 8), strides=[8, -1])]
    elif case == "step0":
        spec = dict(spec, sweep=((0, 0), (8, 8), (1, 0)))
    elif case == "stop_gt_extent":
        spec = dict(spec, sweep=((0, 0), (9, 8), (1, 1)))
    elif case == "start_gt_stop":
        spec = dict(spec, sweep=((5, 0), (4, 8), (1, 1)))
    elif case == "bnd_bad":
        spec = dict(spec, bnd=[1, 3])
    elif case == "range_none":
        spec = dict(spec, bnd=[wl.PERIODIC, wl.NONE])
    elif case == "dir_bad":
        direction = 2
    elif case == "from_window":
        direction = _abi.FROM
    elif case == "from_two_slices":
        spec = dict(spec, slices=[((0, 0), (1, 1)), ((0, 1), (1, 1))])
        direction = _abi.FROM
    elif case == "from_clamp_offset":
        spec = dict(spec, slices=[((0, 1), (1, 1))], bnd=[wl.CLAMP, wl.CLAMP])
        direction = _abi.FROM
    elif case == "too_many_features":
        spec = dict(spec, slices=[((-8, -8), (17, 17))])
    elif case == "reserved":
        arrays[0].reserved = 1
    elif case == "no_targets":
        arrays = []
    assert api.validate_map(spec, arrays, direction, nf)[0] == status


def _brute_injective(spec, shape, strides):
    """Do the sweep points of a one-element `from` functor land on distinct
    element indices?  (Enumerates every point; tiny shapes only.)"""
    import itertools
    import numpy as np
    start, stop, step = spec["sweep"]
    lo = spec["slices"][0][0]
    seen = set()
    for pt in itertools.product(*[range(a, b, c) for a, b, c in zip(start, stop, step)]):
        q = []
        for d, x in enumerate(pt):
            y = x + lo[d]
            if spec["bnd"][d] == wl.PERIODIC:
                y %= shape[d]
            q.append(y)
        e = int(np.dot(q, strides))
        if e in seen:
            return False
        seen.add(e)
    return True


@pytest.mark.parametrize("shape, strides, sweep, lo, bnd", [
    ((8,), (0,), ((0,), (8,), (1,)), (0,), [0]),                         # broadcast view
    ((4, 4), (1, 1), ((0, 0), (4, 4), (1, 1)), (0, 0), [0, 0]),          # strides {1, 1} fold the sweep
    ((4, 4), (0, 1), ((0, 0), (4, 4), (1, 1)), (0, 0), [0, 0]),          # a zero stride on a swept dimension
    ((3, 5), (2, 1), ((0, 0), (3, 5), (1, 1)), (0, 0), [0, 0]),          # rows overlap by 3 elements
    ((3, 5), (2, 1), ((0, 0), (3, 5), (1, 2)), (0, 0), [0, 0]),          # even columns: 0,2,4 then 2,4,6
    ((3, 5), (5, 1), ((0, 0), (3, 5), (1, 1)), (0, 0), [0, 0]),          # row-major: fine
    ((3, 5), (1, 3), ((0, 0), (3, 5), (1, 1)), (0, 0), [0, 0]),          # column-major: fine
    ((3, 5), (6, 1), ((0, 0), (3, 5), (1, 1)), (0, 0), [0, 0]),          # padded rows: fine
    ((3, 5), (2, 1), ((0, 0), (3, 2), (1, 1)), (0, 0), [0, 0]),          # two columns of overlapping rows: fine
    ((3, 5), (0, 1), ((1, 0), (2, 5), (1, 1)), (0, 0), [0, 0]),          # zero stride on an unswept dimension: fine
    ((6,), (1,), ((0,), (6,), (1,)), (2,), [wl.PERIODIC]),                # periodic shift: a permutation
    ((3, 4), (3, 1), ((0, 0), (3, 4), (1, 1)), (0, 1), [0, wl.PERIODIC]), # wrap spans the whole row: folds
])
def test_from_map_must_be_one_to_one(shape, strides, sweep, lo, bnd):
    """A `from` map whose strides could send two sweep points to one element
    is refused (E_ALIAS); one that cannot is accepted.  The expectation is
    brute force over every point, for the cases where the library's
    sufficient test is exact."""
    spec = {"rank": len(shape), "slices": [(lo, (1,) * len(shape))], "sweep": sweep, "bnd": bnd}
    st = api.validate_map(spec, [_arr(shape, strides=list(strides))], _abi.FROM)[0]
    want = _abi.OK if _brute_injective(spec, shape, strides) else _abi.E_ALIAS
    assert st == want
    # a `to` map may read one element from several points
    assert api.validate_map(spec, [_arr(shape, strides=list(strides))], _abi.TO)[0] == _abi.OK


def test_offsets_beyond_extent_wrap():
    spec = {"rank": 1, "slices": [((-20,), (3,))], "sweep": ((0,), (5,), (1,)), "bnd": [wl.PERIODIC]}
    assert api.validate_map(spec, [_arr((5,))], _abi.TO)[:3] == (_abi.OK, 5, 3)


@pytest.mark.parametrize("dims, act, compute, status", [
    ([5, 64, 64, 1], [1, 1, 0], _abi.F32, _abi.OK),
    ([35, 512, 512, 5], [1, 1, 0], _abi.BF16, _abi.OK),
    ([5], [], _abi.F32, _abi.E_INVAL),
    ([5, 0, 1], [1, 0], _abi.F32, _abi.E_INVAL),
    ([5, 4096, 1], [1, 0], _abi.F32, _abi.OK),
    ([5, 8192, 1], [1, 0], _abi.F32, _abi.E_UNSUPPORTED),
    ([300, 64, 1], [1, 0], _abi.F32, _abi.E_UNSUPPORTED),
    ([5] * 10, [1] * 9, _abi.F32, _abi.E_UNSUPPORTED),
    ([5, 64, 1], [1, 2], _abi.F32, _abi.E_INVAL),
    ([5, 64, 1], [1, 0], 7, _abi.E_INVAL),
])
def test_model_validation(dims, act, compute, status):
    assert api.validate_model(dims, act, compute) == status


def test_model_create_rejects_before_device_work():
    L = _abi.lib()
    h = C.c_void_p(1)
    d = (C.c_int32 * 3)(5, 0, 1)
    a = (C.c_int32 * 2)(1, 0)
    st = L.hpacml_model_create(2, d, None, None, a, _abi.F32, C.byref(h))
    assert st == _abi.E_INVAL and h.value is None
    st = L.hpacml_map_create(None, 0, None, 0, None, None, C.byref(h))
    assert st == _abi.E_INVAL and h.value is None
    assert L.hpacml_infer(None, None, None, None) == _abi.E_INVAL
    assert L.hpacml_collect(None, None, 1, None) == _abi.E_INVAL
    assert L.hpacml_collect_pair(None, None, 1, None, None, 1, None) == _abi.E_INVAL
    assert L.hpacml_infer_variant(None, None, None) is None
    L.hpacml_map_destroy(None)
    L.hpacml_model_destroy(None)


def test_cnn_validate_shapes_and_errors():
    """Convolutional model descriptions: output shapes of the two workload
    stacks, and each rejected form reported without a device."""
    for name, want in [("weather_cnn", (2048, 2048, 4)), ("particle_cnn", (1, 1, 2))]:
        st, shp = api.validate_cnn(wl.cnn_model(name, "full"))
        assert st == _abi.OK and shp == want, name
    conv = wl.conv_layer(1, 0, 4, 8, (3, 3))
    base = {"kind": "cnn", "in_channels": 4, "image": (16, 16), "layers": [conv]}
    assert api.validate_cnn(base)[0] == _abi.OK
    # SAME with a step
    assert api.validate_cnn(dict(base, layers=[dict(conv, stride=(1, 2))]))[0] == _abi.E_INVAL
    # VALID window larger than the image
    assert api.validate_cnn(dict(base, layers=[dict(conv, padding="valid", kernel=(17, 3))]))[0] == _abi.E_SHAPE
    # a convolution after a fully connected layer
    lin = wl.linear_layer(1, 0, 16 * 16 * 8, 5)
    assert api.validate_cnn(dict(base, layers=[conv, lin, conv]))[0] == _abi.E_INVAL
    # no layers, bad channels, bad image
    assert api.validate_cnn(dict(base, layers=[]))[0] == _abi.E_INVAL
    assert api.validate_cnn(dict(base, in_channels=0))[0] == _abi.E_INVAL
    assert api.validate_cnn(dict(base, image=(0, 4)))[0] == _abi.E_INVAL
    # zero output channels
    assert api.validate_cnn(dict(base, layers=[dict(conv, out=0)]))[0] == _abi.E_INVAL


def test_cnn_param_counts_match_the_workload_weights():
    """hpacml_cnn_param_counts gives the weight and bias sizes of every layer
    of the two workload stacks (the arrays the workloads draw), zero for the
    pool; an invalid description and NULL arrays are errors."""
    import ctypes as C
    L = _abi.lib()
    for name in ("weather_cnn", "particle_cnn"):
        spec = wl.cnn_model(name, "full")
        n = len(spec["layers"])
        wc, bc = (C.c_int64 * n)(), (C.c_int64 * n)()
        H, W = spec["image"]
        arr = api._layers(spec)
        assert L.hpacml_cnn_param_counts(spec["in_channels"], H, W, n, arr, wc, bc) == _abi.OK
        for l, ly in enumerate(spec["layers"]):
            want_w = 0 if ly["kind"] == "pool" else np.asarray(ly["W"]).size
            want_b = 0 if ly["kind"] == "pool" else np.asarray(ly["b"]).size
            assert (wc[l], bc[l]) == (want_w, want_b), (name, l)
        assert L.hpacml_cnn_param_counts(spec["in_channels"], H, W, n, arr, None, bc) == _abi.E_INVAL
        assert L.hpacml_cnn_param_counts(0, H, W, n, arr, wc, bc) == _abi.E_INVAL

"""The oracle's in-place regions (outputs written into the fields the inputs
are read from) pinned to the reading that every point's inputs are gathered
before any output is written: the result equals the same region run on an
untouched copy of the fields with its outputs written into the originals.
A point-by-point update (each point's outputs written before the next
point's gather) differs on windowed maps, which the test also shows, so the
pin has teeth."""
import numpy as np

import oracle
from paper_2407_18352_amd import workloads as wl


def _inplace(w):
    f = [a.copy() for a in w.inputs]
    oracle.infer(w.in_spec, f, w.out_spec, f, w.model)
    return f


def _from_copy(w):
    f = [a.copy() for a in w.inputs]
    src = [a.copy() for a in w.inputs]
    oracle.infer(w.in_spec, src, w.out_spec, f, w.model)
    return f


def _point_by_point(w):
    """A wrong in-place update: rows gathered and written one point at a time."""
    f = [a.copy() for a in w.inputs]
    ny, nx = f[0].shape
    for i in range(ny):
        for j in range(nx):
            one = {"rank": 2, "slices": w.in_spec["slices"], "sweep": ((i, j), (i + 1, j + 1), (1, 1)),
                   "bnd": w.in_spec["bnd"]}
            out1 = dict(w.out_spec, sweep=((i, j), (i + 1, j + 1), (1, 1)))
            oracle.infer(one, f, out1, f, w.model)
    return f


def test_inplace_window_equals_gather_from_copy():
    w = wl.make("stencil2d", (9, 13))
    got = _inplace(w)
    want = _from_copy(w)
    for a, b in zip(got, want):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    wrong = _point_by_point(w)
    assert any(not np.array_equal(a, b) for a, b in zip(wrong, want))


def test_inplace_pointwise_is_element_for_element():
    w = wl.make("options", 257)
    f = [a.copy() for a in w.inputs]
    out = {"rank": 1, "slices": [((0,), (1,))], "sweep": ((0,), (257,), (1,)), "bnd": [0]}
    oracle.infer(w.in_spec, f, out, [f[0]], w.model)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    assert np.array_equal(f[0], Y[:, 0].astype(np.float32))
    for k in range(1, 5):
        assert np.array_equal(f[k], w.inputs[k])


def test_inplace_convolution_equals_gather_from_copy():
    w = wl.make_cnn("weather_cnn", (11, 17))
    got = _inplace(w)
    want = _from_copy(w)
    for a, b in zip(got, want):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))

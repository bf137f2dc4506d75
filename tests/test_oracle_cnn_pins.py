"""Pins of the oracle's convolutional surrogates (the MiniWeather and
ParticleFilter model spaces of Table IV), each against something other than
the oracle's own formula:

* random stacks of convolution (every padding mode, even and odd windows,
  steps), max-pool and fully connected layers equal the same stack run by
  torch in fp64 (``F.pad`` + ``F.conv2d``, ``F.max_pool2d``, ``F.linear`` on the
  [row][column][channel] flattening);
* a one-hot convolution window is a shifted copy of the image, enumerated with
  ``np.pad`` (wrap / edge / constant), bit for bit, also where the padding is
  wider than the image;
* a 3x3 circular convolution followed by 1x1 convolutions on a pointwise map
  equals the MLP oracle on the 3x3 periodic window map (two independently
  pinned paths of the oracle);
* max-pool equals numpy's reshape-and-max, NaN included.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import oracle
from paper_2407_18352_amd import workloads as wl


def _conv(g, cin, cout, k, padding="same", mode="zeros", stride=(1, 1), act=1):
    fan = cin * k[0] * k[1]
    return {"kind": "conv", "out": cout, "kernel": k, "stride": stride, "padding": padding, "mode": mode,
            "act": act, "W": (g.standard_normal((cout, cin) + tuple(k)) / np.sqrt(fan)).astype(np.float32),
            "b": g.uniform(-0.5, 0.5, cout).astype(np.float32)}


def _linear(g, fin, fout, act=1):
    return {"kind": "linear", "out": fout, "act": act,
            "W": (g.standard_normal((fout, fin)) / np.sqrt(fin)).astype(np.float32),
            "b": g.uniform(-0.5, 0.5, fout).astype(np.float32)}


def _torch_cnn(model, X):
    """The stack in torch fp64 on X[S*H*W, C] (NHWC rows) -> [S*H'*W', C']."""
    H, W = model["image"]
    C0 = model["in_channels"]
    t = torch.from_numpy(X).reshape(-1, H, W, C0).permute(0, 3, 1, 2)      # NCHW
    flat = False
    for ly in model["layers"]:
        if ly["kind"] == "conv":
            kh, kw = ly["kernel"]
            if ly["padding"] == "same":
                top, left = (kh - 1) // 2, (kw - 1) // 2
                pads = (left, kw - 1 - left, top, kh - 1 - top)
                mode = {"zeros": "constant", "circular": "circular", "replicate": "replicate"}[ly["mode"]]
                t = Fn.pad(t, pads, mode=mode)
            t = Fn.conv2d(t, torch.from_numpy(ly["W"].astype(np.float64)),
                          torch.from_numpy(ly["b"].astype(np.float64)), stride=tuple(ly["stride"]))
        elif ly["kind"] == "pool":
            t = Fn.max_pool2d(t, tuple(ly["kernel"]), stride=tuple(ly.get("stride", ly["kernel"])))
        else:
            if not flat:
                t = t.permute(0, 2, 3, 1).reshape(t.shape[0], -1)               # [row][col][channel]
                flat = True
            t = Fn.linear(t, torch.from_numpy(ly["W"].astype(np.float64)),
                          torch.from_numpy(ly["b"].astype(np.float64)))
        if ly.get("act", 0) == 1:
            t = torch.relu(t)
    if flat:
        return t.numpy()
    return t.permute(0, 2, 3, 1).reshape(-1, t.shape[1]).numpy()


@pytest.mark.parametrize("mode", ["zeros", "circular", "replicate"])
@pytest.mark.parametrize("k1, k2", [((3, 3), (1, 1)), ((5, 5), (3, 3)), ((4, 4), (2, 6)), ((8, 8), (6, 6)),
                                    ((2, 7), (0, 0))])
def test_conv_stack_matches_torch(mode, k1, k2):
    """MiniWeather-shaped stacks: one or two same-padded convolutions."""
    g = np.random.default_rng(hash((mode, k1, k2)) & 0xFFFF)
    H, W, C0, C1 = 9, 11, 4, 8
    layers = [_conv(g, C0, C1, k1, mode=mode, act=1)]
    if k2 != (0, 0):
        layers.append(_conv(g, C1, C0, k2, mode=mode, act=0))
    model = {"kind": "cnn", "in_channels": C0, "image": (H, W), "layers": layers}
    X = g.standard_normal((2 * H * W, C0))
    got = oracle.cnn(model, X)
    want = _torch_cnn(model, X)
    assert got.shape == want.shape
    np.testing.assert_allclose(got, want.astype(np.float32), rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("k, s, pool, fc", [(4, 4, 2, 16), (2, 2, 3, 0), (7, 7, 1, 8), (3, 2, 2, 5)])
def test_conv_pool_linear_matches_torch(k, s, pool, fc):
    """ParticleFilter-shaped stacks: a strided valid convolution, a max-pool,
    then fully connected layers to a 2-value estimate."""
    g = np.random.default_rng(k * 100 + s * 10 + pool)
    H, W, C0, C1 = 29, 31, 1, 6
    layers = [_conv(g, C0, C1, (k, k), padding="valid", stride=(s, s), act=1),
              {"kind": "pool", "kernel": (pool, pool), "act": 0}]
    model = {"kind": "cnn", "in_channels": C0, "image": (H, W), "layers": layers}
    h, w, c = oracle.cnn_shapes(model)[-1]
    if fc:
        layers += [_linear(g, h * w * c, fc, act=1), _linear(g, fc, 2, act=0)]
    else:
        layers += [_linear(g, h * w * c, 2, act=0)]
    X = g.standard_normal((3 * H * W, C0))
    got = oracle.cnn(model, X)
    want = _torch_cnn(model, X)
    assert got.shape == (3, 2) == want.shape
    np.testing.assert_allclose(got, want.astype(np.float32), rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("mode, np_mode", [("zeros", "constant"), ("circular", "wrap"), ("replicate", "edge")])
@pytest.mark.parametrize("H, W", [(5, 7), (2, 3), (1, 1)])
def test_one_hot_window_is_a_shifted_copy(mode, np_mode, H, W):
    """Weight 1 at one window position: out[y][x] = padded[y + ky][x + kx],
    bit for bit, for every position of windows up to 8 wide (the padding may
    be wider than the image)."""
    g = np.random.default_rng(7)
    img = g.standard_normal((H, W)).astype(np.float32)
    for kh, kw in [(3, 3), (8, 5), (4, 1)]:
        top, left = (kh - 1) // 2, (kw - 1) // 2
        P = np.pad(img, ((top, kh - 1 - top), (left, kw - 1 - left)), mode=np_mode)
        for ky in range(kh):
            for kx in range(kw):
                Wt = np.zeros((1, 1, kh, kw), np.float32)
                Wt[0, 0, ky, kx] = 1.0
                model = {"kind": "cnn", "in_channels": 1, "image": (H, W),
                         "layers": [{"kind": "conv", "out": 1, "kernel": (kh, kw), "padding": "same",
                                     "mode": mode, "act": 0, "W": Wt, "b": np.zeros(1, np.float32)}]}
                got = oracle.cnn(model, img.reshape(-1, 1).astype(np.float64)).reshape(H, W)
                assert np.array_equal(got.view(np.uint32), P[ky:ky + H, kx:kx + W].view(np.uint32)), \
                    (mode, kh, kw, ky, kx)


def test_circular_conv_stack_equals_window_mlp():
    """[3x3 circular conv -> ReLU -> 1x1 conv -> ReLU -> 1x1 conv] on a
    pointwise map is the 36 -> 16 -> 16 -> 4 MLP on the 3x3 periodic window
    map: the window map's features are target-major, then row-major over the
    window, i.e. the conv weight [out][channel][ky][kx] flattened."""
    g = np.random.default_rng(11)
    ny, nx, C = 7, 10, 4
    fields = [g.standard_normal((ny, nx)).astype(np.float32) for _ in range(C)]
    c1, c2, c3 = _conv(g, C, 16, (3, 3), mode="circular"), _conv(g, 16, 16, (1, 1)), _conv(g, 16, C, (1, 1), act=0)
    cnn = {"kind": "cnn", "in_channels": C, "image": (ny, nx), "layers": [c1, c2, c3]}
    mlp = {"dims": [36, 16, 16, 4], "W": [c1["W"].reshape(16, 36), c2["W"].reshape(16, 16), c3["W"].reshape(4, 16)],
           "b": [c1["b"], c2["b"], c3["b"]], "act": [1, 1, 0], "compute": "f32"}
    got = oracle.cnn(cnn, oracle.gather(wl.point2d_spec(ny, nx), fields))
    want = oracle.infer_rows(wl.window2d_spec(ny, nx), fields, mlp)
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=1e-6)


def test_maxpool_equals_reshape_max_with_nan():
    g = np.random.default_rng(5)
    S, H, W, Cc, k = 2, 6, 8, 3, 2
    X = g.standard_normal((S, H, W, Cc))
    X[0, 1, 2, 1] = np.nan
    X[1, 5, 7, 0] = np.nan
    model = {"kind": "cnn", "in_channels": Cc, "image": (H, W), "layers": [{"kind": "pool", "kernel": (k, k)}]}
    got = oracle.cnn(model, X.reshape(-1, Cc)).reshape(S, H // k, W // k, Cc)
    want = X.reshape(S, H // k, k, W // k, k, Cc).max(axis=(2, 4)).astype(np.float32)
    assert np.array_equal(np.isnan(got), np.isnan(want)) and np.isnan(got).sum() == 2
    assert np.array_equal(got[~np.isnan(got)], want[~np.isnan(want)])


def test_shapes_and_rejections():
    g = np.random.default_rng(3)
    model = {"kind": "cnn", "in_channels": 1, "image": (16, 20),
             "layers": [_conv(g, 1, 4, (4, 4), padding="valid", stride=(2, 2)), {"kind": "pool", "kernel": (3, 3)},
                        _linear(g, 2 * 2 * 4, 2)]}
    assert oracle.cnn_shapes(model) == [(16, 20, 1), (7, 9, 4), (2, 3, 4), (1, 1, 2)]
    # same padding with a step, and a window larger than a valid input, are errors
    bad = dict(model, layers=[_conv(g, 1, 4, (3, 3), stride=(2, 1))])
    with pytest.raises(ValueError):
        oracle.cnn_shapes(bad)
    bad = dict(model, layers=[_conv(g, 1, 4, (17, 3), padding="valid")])
    with pytest.raises(ValueError):
        oracle.cnn_shapes(bad)

"""GPU parity of the convolutional surrogates (called through the C ABI)
against the oracle: fp32 outputs within |g - o| <= 1e-5 * max(|o|, s)
(s = RMS of the oracle's output column), no NaN where the oracle has none,
untouched elements keep their sentinel bits."""
import numpy as np
import pytest

import oracle
from paper_2407_18352_amd import _abi, api
from paper_2407_18352_amd import workloads as wl
from gpu_util import RTOL, assert_close, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def _run(w, fields_out=None):
    """The region on the GPU; returns (outputs as numpy, variant)."""
    import torch
    ins = to_dev(w.inputs)
    outs = ins if fields_out == "inplace" else to_dev(w.outputs)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.FROM)
    m = api.CnnModel(w.model)
    var = api.variant(m, mi, mo)
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in outs], var


def _expected(w, inplace=False):
    src = [a.copy() for a in w.inputs]
    dst = src if inplace else [a.copy() for a in w.outputs]
    oracle.infer(w.in_spec, src, w.out_spec, dst, w.model)
    return dst


def _compare(got, want, what, rtol=RTOL["f32"]):
    g = np.stack([a.reshape(-1) for a in got], 1)
    e = np.stack([a.reshape(-1) for a in want], 1)
    return assert_close(g, e, rtol, what)


def _rtol_for(model):
    """The fp32 bar holds for the searched stacks (at most two convolutions,
    sums of at most 256 terms: 8x8 windows over 4 channels, 6x6 over 8).
    Beyond that space it widens by sqrt(n / 256) for n-term sums and by L / 2
    for L layers: rounding errors of an n-term fp32 sum grow like sqrt(n),
    and each layer passes the earlier layers' errors on."""
    n, L = 1, 0
    c = model["in_channels"]
    for ly in model["layers"]:
        if ly["kind"] == "conv":
            n = max(n, c * ly["kernel"][0] * ly["kernel"][1])
            c = ly["out"]
            L += 1
    return RTOL["f32"] * max(1.0, (n / 256) ** 0.5) * max(1.0, L / 2)


@pytest.mark.parametrize("name, want", [("weather_cnn", "cnn_fused_f32"), ("particle_cnn", "cnn_layers_f32")])
def test_cnn_small(name, want):
    w = wl.make_cnn(name, "small")
    got, var = _run(w)
    assert var == want
    worst, norm = _compare(got, _expected(w), "%s via %s" % (name, var))
    print("%s [%s]: worst scaled %.3e, normwise %.3e" % (name, var, worst, norm))


def _random_stack(g, cin, n_layers, modes, max_c=16, max_k=8):
    layers, c = [], cin
    for l in range(n_layers):
        cout = int(g.integers(1, max_c + 1))
        k = (int(g.integers(1, max_k + 1)), int(g.integers(1, max_k + 1)))
        layers.append(wl.conv_layer(int(g.integers(1 << 20)), 0, c, cout, k, mode=modes[l],
                                    act=int(g.integers(0, 2))))
        c = cout
    return layers, c


@pytest.mark.parametrize("case", range(12))
def test_fused_random_stacks(case):
    """Random SAME stacks (1-4 layers, windows 1-8 incl. even, 1-16 channels,
    every padding-mode family) on ragged images, one or several images."""
    g = np.random.default_rng(1000 + case)
    family = ["circular", "zeros", "replicate", "mixed"][case % 4]
    n_layers = 1 + case % 4
    if family == "mixed":
        modes = [["zeros", "replicate"][int(g.integers(0, 2))] for _ in range(n_layers)]
    else:
        modes = [family] * n_layers
    cin = int(g.integers(1, 17))
    S = 1 + case % 3
    H, W = [(1, 1), (2, 3), (5, 70), (33, 65), (40, 130), (3, 200)][case % 6]
    layers, cout = _random_stack(g, cin, n_layers, modes)
    model = {"kind": "cnn", "in_channels": cin, "image": (H, W), "layers": layers}
    inputs = [g.standard_normal((S, H, W)).astype(np.float32) for _ in range(cin)]
    spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
            "bnd": [0, 0, 0]}
    outputs = [wl.sentinel_like((S, H, W)) for _ in range(cout)]
    w = wl.Workload("random", 0, "f32", [cin, cout], spec, spec, inputs, outputs, model)
    got, var = _run(w)
    assert var == "cnn_fused_f32", var
    _compare(got, _expected(w), "case %d (%s, %d layers, %dx%dx%d)" % (case, family, n_layers, S, H, W),
             _rtol_for(model))


@pytest.mark.parametrize("case", range(4))
def test_layered_path_stacks(case):
    """Stacks only the layer-by-layer path takes: circular mixed with other
    modes, valid / strided convolutions, pools and fully connected layers,
    more than 16 channels."""
    g = np.random.default_rng(2000 + case)
    S, H, W, cin = 2, 19, 23, 3
    if case == 0:
        layers = [wl.conv_layer(1, 0, cin, 5, (3, 3), mode="circular"), wl.conv_layer(2, 0, 5, 4, (4, 2), mode="zeros")]
    elif case == 1:
        layers = [wl.conv_layer(3, 0, cin, 20, (3, 3), mode="replicate"),
                  wl.conv_layer(4, 0, 20, 2, (1, 1), act=0)]
    elif case == 2:
        layers = [wl.conv_layer(5, 0, cin, 6, (5, 3), padding="valid", stride=(2, 3)),
                  {"kind": "pool", "kernel": (2, 2), "stride": (1, 2)}]
    else:
        layers = [wl.conv_layer(6, 0, cin, 4, (3, 3), padding="valid", mode="zeros", stride=(2, 2)),
                  {"kind": "pool", "kernel": (3, 3)}]
        h, w_, c = oracle.cnn_shapes({"kind": "cnn", "in_channels": cin, "image": (H, W), "layers": layers})[-1]
        layers += [wl.linear_layer(7, 0, h * w_ * c, 9), wl.linear_layer(8, 0, 9, 3, act=0)]
    model = {"kind": "cnn", "in_channels": cin, "image": (H, W), "layers": layers}
    h2, w2, c2 = oracle.cnn_shapes(model)[-1]
    inputs = [g.standard_normal((S, H, W)).astype(np.float32) for _ in range(cin)]
    ins = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
           "bnd": [0, 0, 0]}
    outs = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, h2, w2), (1, 1, 1)),
            "bnd": [0, 0, 0]}
    outputs = [wl.sentinel_like((S, h2, w2)) for _ in range(c2)]
    w = wl.Workload("layered", 0, "f32", [cin, c2], ins, outs, inputs, outputs, model)
    got, var = _run(w)
    assert var == "cnn_layers_f32", var
    _compare(got, _expected(w), "layered case %d" % case)


@pytest.mark.parametrize("view", ["interleaved", "sweep_offset", "padded_rows"])
def test_layered_input_read_in_place_or_gathered(view):
    """Channels interleaved in one array [S][H][W*C] (a sweep of step C over
    the last dimension, a slice of C elements): the map's tensor is then the
    array itself, row for row, and the first layer reads it there; a sweep
    that starts past the first frame, or rows padded past W*C, leave a
    tensor that must be gathered first.  All three match the oracle.  The
    1980-term fully connected sums are split over blocks with a ragged last
    chunk."""
    import torch
    g = np.random.default_rng(4100 + ["interleaved", "sweep_offset", "padded_rows"].index(view))
    S, H, W, C = 3, 24, 20, 2
    layers = [wl.conv_layer(11, 0, C, 5, (3, 3), padding="valid"),
              wl.linear_layer(12, 0, 22 * 18 * 5, 7), wl.linear_layer(13, 0, 7, 2, act=0)]
    model = {"kind": "cnn", "in_channels": C, "image": (H, W), "layers": layers}
    first = 1 if view == "sweep_offset" else 0
    pad = 6 if view == "padded_rows" else 0
    host = g.standard_normal((S + first, H, W * C + pad)).astype(np.float32)
    host_view = host[:, :, :W * C]
    spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, C))],
            "sweep": ((first, 0, 0), (S + first, H, W * C), (1, 1, C)), "bnd": [0, 0, 0]}
    dev = torch.from_numpy(host).cuda()
    mi = api.Map(spec, [dev[:, :, :W * C]], _abi.TO)
    outs = to_dev([wl.sentinel_like((S,)) for _ in range(2)])
    mo = api.Map(wl.pointwise_spec(S), outs, _abi.FROM)
    m = api.CnnModel(model)
    assert api.variant(m, mi, mo) == "cnn_layers_f32"
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    exp = [wl.sentinel_like((S,)) for _ in range(2)]
    oracle.infer(spec, [host_view], wl.pointwise_spec(S), exp, model)
    _compare([o.cpu().numpy() for o in outs], exp, "first-layer input, %s" % view)
    assert np.array_equal(dev.cpu().numpy().view(np.uint32), host.view(np.uint32))   # inputs untouched


@pytest.mark.parametrize("pool_k", [(2, 2), (3, 3), (1, 3), (4, 4)])
def test_conv_then_pool_in_one_kernel(pool_k):
    """Convolutions followed by max-pools whose windows do not overlap run as
    one kernel each (a lane group per pooled pixel): NaN inputs pass identity
    convolutions and pools to the outputs (a ReLU on the last pool, for two
    of the window shapes, clears them), conv outputs past the last whole
    window are dropped as the pool drops them, and the second convolution
    has 9 channels (a partial channel group)."""
    g = np.random.default_rng(300 + 10 * pool_k[0] + pool_k[1])
    S, H, W, C = 3, 23, 29, 2
    imgs = [g.standard_normal((S, H, W)).astype(np.float32) for _ in range(C)]
    imgs[0][1, 5, 7] = np.nan
    imgs[1][2, 20, 3] = np.nan
    layers = [wl.conv_layer(21, 0, C, 4, (3, 3), mode="zeros", act=0), {"kind": "pool", "kernel": pool_k},
              wl.conv_layer(22, 0, 4, 9, (2, 2), padding="valid", act=0),
              {"kind": "pool", "kernel": (2, 2), "act": int(pool_k in ((3, 3), (1, 3)))}]
    model = {"kind": "cnn", "in_channels": C, "image": (H, W), "layers": layers}
    h2, w2, c2 = oracle.cnn_shapes(model)[-1]
    spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
            "bnd": [0, 0, 0]}
    out_spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, h2, w2), (1, 1, 1)),
                "bnd": [0, 0, 0]}
    w = wl.Workload("convpool", 0, "f32", [C, c2], spec, out_spec, imgs,
                    [wl.sentinel_like((S, h2, w2)) for _ in range(c2)], model)
    got, var = _run(w)
    assert var == "cnn_layers_f32", var
    exp = _expected(w)
    g2 = np.stack([a.reshape(-1) for a in got], 1)
    e2 = np.stack([a.reshape(-1) for a in exp], 1)
    assert np.array_equal(np.isnan(g2), np.isnan(e2))
    ok = ~np.isnan(e2)
    assert_close(np.where(ok, g2, 0), np.where(ok, e2, 0), RTOL["f32"], "conv + pool %s" % (pool_k,))


TAIL_CASES = ["fc_only", "long_tail", "reduce_only", "two_closing"]


@pytest.mark.parametrize("case", TAIL_CASES)
def test_fully_connected_tails(case):
    """The fully connected layers closing a stack run with the scatter in one
    kernel: a stack of fully connected layers only (256 wide, one image per
    block), more small layers than that kernel takes (the layer-by-layer
    kernels instead), a single wide-K layer (split K, then only the partial
    sums, bias and scatter), and a split-K layer followed by two small
    layers of different widths.  37 images: a ragged last block."""
    g = np.random.default_rng(TAIL_CASES.index(case) + 500)
    S, H, W, C = 37, 12, 14, 2
    if case == "fc_only":
        layers = [wl.linear_layer(31, 0, H * W * C, 200), wl.linear_layer(32, 0, 200, 256),
                  wl.linear_layer(33, 0, 256, 3, act=0)]
    elif case == "long_tail":
        layers = [wl.conv_layer(34, 0, C, 3, (3, 3), padding="valid"), wl.linear_layer(35, 0, 10 * 12 * 3, 32)]
        layers += [wl.linear_layer(36 + k, 0, 32, 32) for k in range(5)] + [wl.linear_layer(41, 0, 32, 2, act=0)]
    elif case == "reduce_only":
        layers = [wl.conv_layer(42, 0, C, 4, (3, 3), mode="circular"), {"kind": "pool", "kernel": (2, 2)},
                  wl.linear_layer(43, 0, 6 * 7 * 4, 17, act=0)]
    else:
        layers = [wl.conv_layer(44, 0, C, 8, (3, 3), mode="zeros"), wl.linear_layer(45, 0, H * W * 8, 48),
                  wl.linear_layer(46, 0, 48, 40), wl.linear_layer(47, 0, 40, 5, act=0)]
    model = {"kind": "cnn", "in_channels": C, "image": (H, W), "layers": layers}
    c2 = oracle.cnn_shapes(model)[-1][2]
    imgs = [g.standard_normal((S, H, W)).astype(np.float32) for _ in range(C)]
    spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
            "bnd": [0, 0, 0]}
    w = wl.Workload("tail", 0, "f32", [C, c2], spec, wl.pointwise_spec(S), imgs,
                    [wl.sentinel_like((S,)) for _ in range(c2)], model)
    got, var = _run(w)
    assert var == "cnn_layers_f32", var
    _compare(got, _expected(w), "fully connected tail, %s" % case, _rtol_for(model))


def test_many_small_images_take_the_unsplit_kernels():
    """140,000 images of 3x3: the tiles alone cover the chip, so the fully
    connected layer of 32 outputs runs unsplit on the 64 x 64 VALU tiles and
    the closing layer in the tail kernel; every image against the oracle."""
    g = np.random.default_rng(800)
    S, H, W = 140000, 3, 3
    layers = [wl.conv_layer(71, 0, 1, 4, (2, 2), padding="valid"), wl.linear_layer(72, 0, 2 * 2 * 4, 32),
              wl.linear_layer(73, 0, 32, 3, act=0)]
    model = {"kind": "cnn", "in_channels": 1, "image": (H, W), "layers": layers}
    frames = g.standard_normal((S, H, W)).astype(np.float32)
    spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
            "bnd": [0, 0, 0]}
    w = wl.Workload("many", 0, "f32", [1, 3], spec, wl.pointwise_spec(S), [frames],
                    [wl.sentinel_like((S,)) for _ in range(3)], model)
    got, var = _run(w)
    assert var == "cnn_layers_f32", var
    _compare(got, _expected(w), "many small images")


def test_zero_images_launch_nothing():
    """Sweeps with no images: inference returns OK, writes nothing, and the
    record of the (empty) input map is empty."""
    import torch
    H, W = 16, 16
    model = {"kind": "cnn", "in_channels": 1, "image": (H, W),
             "layers": [wl.conv_layer(51, 0, 1, 4, (4, 4), padding="valid", stride=(4, 4)),
                        {"kind": "pool", "kernel": (2, 2)}, wl.linear_layer(52, 0, 2 * 2 * 4, 3, act=0)]}
    frames = to_dev([np.ones((2, H, W), np.float32)])
    spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((1, 0, 0), (1, H, W), (1, 1, 1)),
            "bnd": [0, 0, 0]}
    outs = to_dev([wl.sentinel_like((2,)) for _ in range(3)])
    mi = api.Map(spec, frames, _abi.TO)
    mo = api.Map({"rank": 1, "slices": [((0,), (1,))], "sweep": ((2,), (2,), (1,)), "bnd": [0]}, outs, _abi.FROM)
    assert mi.n_points == 0 and mo.n_points == 0
    m = api.CnnModel(model)
    api.infer(m, mi, mo)
    conv = api.CnnModel({"kind": "cnn", "in_channels": 1, "image": (H, W),
                         "layers": [wl.conv_layer(53, 0, 1, 2, (3, 3), mode="circular")]})
    mo2 = api.Map(spec, to_dev([wl.sentinel_like((2, H, W)) for _ in range(2)]), _abi.FROM)
    api.infer(conv, mi, mo2)
    torch.cuda.synchronize()
    for o in outs:
        assert np.array_equal(o.cpu().numpy().view(np.uint32), wl.sentinel_like((2,)).view(np.uint32))


def test_window_map_channels_and_strided_views():
    """Channels from a 3x3 periodic window map (36 channels: layer by layer)
    and from column views of one array of structures (fused)."""
    import torch
    g = np.random.default_rng(77)
    ny, nx = 21, 67
    fields = [wl.sinusoid_field(3, k, ny, nx) for k in range(4)]
    model = {"kind": "cnn", "in_channels": 36, "image": (ny, nx),
             "layers": [wl.conv_layer(1, 0, 36, 4, (3, 3), mode="replicate", act=0)]}
    outputs = [wl.sentinel_like((ny, nx)) for _ in range(4)]
    w = wl.Workload("window", 0, "f32", [36, 4], wl.window2d_spec(ny, nx), wl.point2d_spec(ny, nx), fields,
                    outputs, model)
    got, var = _run(w)
    assert var == "cnn_layers_f32"
    _compare(got, _expected(w), "window channels")
    # array of structures [ny][nx][4]: four strided column views
    aos = np.stack(fields, -1).copy()
    dev = torch.from_numpy(aos).cuda()
    views = [dev[:, :, k] for k in range(4)]
    m4 = {"kind": "cnn", "in_channels": 4, "image": (ny, nx),
          "layers": [wl.conv_layer(2, 0, 4, 7, (4, 4), mode="circular"), wl.conv_layer(3, 0, 7, 2, (3, 5),
                                                                                       mode="circular", act=0)]}
    outs = to_dev([wl.sentinel_like((ny, nx)) for _ in range(2)])
    mi = api.Map(wl.point2d_spec(ny, nx), views, _abi.TO)
    mo = api.Map(wl.point2d_spec(ny, nx), outs, _abi.FROM)
    m = api.CnnModel(m4)
    assert api.variant(m, mi, mo) == "cnn_fused_f32"
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    exp = [wl.sentinel_like((ny, nx)) for _ in range(2)]
    oracle.infer(wl.point2d_spec(ny, nx), fields, wl.point2d_spec(ny, nx), exp, m4)
    _compare([o.cpu().numpy() for o in outs], exp, "array of structures")


@pytest.mark.parametrize("stack", ["fused", "layers", "single_field"])
def test_inplace_update_reads_every_input_first(stack):
    """A MiniWeather-like step written back into its own fields.  The fused
    tiles would read pixels other tiles have overwritten, so the inputs go to
    the map's snapshot record first and the fused kernel reads them there; a
    stack the fused kernel does not take (circular and zero padding mixed)
    runs layer by layer (every input gathered first).  Both match the
    oracle's region on the same arrays, and a second step reuses the
    snapshot record."""
    import torch
    w = wl.make_cnn("weather_cnn", (29, 70))
    want = "snapshot+cnn_fused_f32"
    if stack == "layers":
        model = {"kind": "cnn", "in_channels": 4, "image": (29, 70),
                 "layers": [wl.conv_layer(61, 0, 4, 6, (3, 3), mode="circular"),
                            wl.conv_layer(62, 0, 6, 4, (3, 3), mode="zeros", act=0)]}
        w = wl.Workload("inplace_layers", 0, "f32", [4, 4], w.in_spec, w.out_spec, w.inputs, w.outputs, model)
        want = "cnn_layers_f32"
    elif stack == "single_field":
        # one field: the snapshot record is row-major [points][1]
        model = {"kind": "cnn", "in_channels": 1, "image": (29, 70),
                 "layers": [wl.conv_layer(63, 0, 1, 4, (3, 3), mode="circular"),
                            wl.conv_layer(64, 0, 4, 1, (3, 3), mode="circular", act=0)]}
        w = wl.Workload("inplace_single", 0, "f32", [1, 1], w.in_spec, w.out_spec, w.inputs[:1], w.outputs[:1],
                        model)
    fields = to_dev(w.inputs)
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.CnnModel(w.model)
    assert api.variant(m, mi, mo) == want
    exp = [a.copy() for a in w.inputs]
    for step in range(2):
        api.infer(m, mi, mo)
        oracle.infer(w.in_spec, exp, w.out_spec, exp, w.model)
        torch.cuda.synchronize()
        _compare([f.cpu().numpy() for f in fields], exp, "in place (%s), step %d" % (stack, step))


def test_pool_nan_propagates_and_relu_clears_nan():
    g = np.random.default_rng(9)
    S, H, W = 2, 8, 10
    img = g.standard_normal((S, H, W)).astype(np.float32)
    img[0, 3, 4] = np.nan
    img[1, 0, 9] = np.nan
    spec3 = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
             "bnd": [0, 0, 0]}
    pool = {"kind": "cnn", "in_channels": 1, "image": (H, W), "layers": [{"kind": "pool", "kernel": (2, 2)}]}
    out_spec = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, 4, 5), (1, 1, 1)),
                "bnd": [0, 0, 0]}
    w = wl.Workload("pool", 0, "f32", [1, 1], spec3, out_spec, [img], [wl.sentinel_like((S, 4, 5))], pool)
    got, _ = _run(w)
    exp = _expected(w)
    assert np.array_equal(np.isnan(got[0]), np.isnan(exp[0])) and np.isnan(got[0]).sum() == 2
    assert np.array_equal(got[0][~np.isnan(got[0])], exp[0][~np.isnan(exp[0])])
    # a NaN pixel through a ReLU convolution: 0 where the oracle has 0
    conv = {"kind": "cnn", "in_channels": 1, "image": (H, W),
            "layers": [wl.conv_layer(4, 0, 1, 3, (3, 3), mode="zeros", act=1)]}
    outs3 = [wl.sentinel_like((S, H, W)) for _ in range(3)]
    w2 = wl.Workload("nan", 0, "f32", [1, 3], spec3, spec3, [img], outs3, conv)
    got2, var2 = _run(w2)
    assert var2 == "cnn_fused_f32"
    _compare(got2, _expected(w2), "NaN through ReLU conv")


def test_cnn_errors():
    import torch
    w = wl.make_cnn("weather_cnn", (16, 64))
    ins, outs = to_dev(w.inputs), to_dev(w.outputs)
    m = api.CnnModel(w.model)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    # image size differs from the model's
    small = api.Map(wl.point2d_spec(16, 63), [x[:, :63] for x in outs], _abi.FROM)
    mi63 = api.Map(wl.point2d_spec(16, 63), [x[:, :63] for x in ins], _abi.TO)
    with pytest.raises(_abi.HpacmlError) as e:
        api.infer(m, mi63, small)
    assert e.value.status == _abi.E_SHAPE
    # output feature count differs from the last layer's channels
    mo3 = api.Map(w.out_spec, outs[:3], _abi.FROM)
    with pytest.raises(_abi.HpacmlError) as e:
        api.infer(m, mi, mo3)
    assert e.value.status == _abi.E_SHAPE
    # two outputs that can write one element
    race = api.Map(w.out_spec, [outs[0], outs[0], outs[1], outs[2]], _abi.FROM)
    with pytest.raises(_abi.HpacmlError) as e:
        api.infer(m, mi, race)
    assert e.value.status == _abi.E_ALIAS
    # descriptions
    bad = dict(w.model, layers=[dict(w.model["layers"][0], stride=(2, 1))])
    assert api.validate_cnn(bad)[0] == _abi.E_INVAL
    st, shp = api.validate_cnn(w.model)
    assert st == _abi.OK and shp == (16, 64, 4)
    torch.cuda.synchronize()

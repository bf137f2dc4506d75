"""GPU parity at the five configurations' full sizes, in the launch
configuration the benchmark times: inference checked against the oracle on
every point of the four smaller workloads and, on the 512^3 grid, on a fixed
seeded sample of 2^20 cells plus every cell on the grid's 12 edges; collect
indexing checked bit-exactly on whole grids (3-D: all sixteen 32-plane
z-slabs, the first and last of which include the periodic wrap)."""
import numpy as np
import pytest

import oracle
from paper_2407_18352_amd import _abi, api
from paper_2407_18352_amd import workloads as wl
from gpu_util import RTOL, assert_close, require_gpu, run_collect, run_infer

pytestmark = pytest.mark.gpu

_cache = {}


def full(name):
    if name not in _cache:
        _cache.clear()
        _cache[name] = wl.make(name)
    return _cache[name]


def edges(w):
    shape = w.inputs[0].shape
    if len(shape) == 3:
        return wl.edge_rows_3d(*shape)
    if len(shape) == 2:
        return wl.edge_rows_2d(*shape)
    return np.array([0, shape[0] - 1], np.int64)


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


@pytest.mark.parametrize("name", wl.NAMES)
def test_infer_fullsize(name):
    """Every point of options, bonds, the 2-D stencil and poses (4,194,304
    poses: ~10 s of the oracle on 16 threads); 2^20 seeded cells plus the
    6,128 edge cells of the 512^3 grid.  Prints the worst scaled error."""
    w = full(name)
    got, var = run_infer(w)
    if name == "stencil3d":
        rows = wl.sample_rows(w.n_points, 1 << 20, must=edges(w))
        Y = oracle.infer_rows(w.in_spec, w.inputs, w.model, rows)
        gotY = np.stack([a.reshape(-1)[rows] for a in got], 1)
        n = len(rows)
    else:
        Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
        gotY = np.stack([a.reshape(-1) for a in got], 1)
        n = w.n_points
    worst, norm = assert_close(gotY, Y, RTOL[w.compute], "%s via %s" % (name, var))
    print("%s [%s] full size, %d of %d points against the oracle: worst scaled error %.3e (bar %.0e), "
          "normwise %.3e" % (name, var, n, w.n_points, worst, RTOL[w.compute], norm))
    for a in got:
        assert not np.any(a.view(np.uint32) == wl.SENTINEL_BITS), "unwritten output element"


@pytest.mark.parametrize("name", ["options", "bonds", "stencil2d", "poses"])
def test_collect_fullsize_bitexact(name):
    w = full(name)
    got = run_collect(w.in_spec, w.inputs)
    assert np.array_equal(got, oracle.collect(w.in_spec, w.inputs))


@pytest.mark.parametrize("z0, z1", [(z, z + 32) for z in range(0, 512, 32)])
def test_collect_stencil3d_slabs_bitexact(z0, z1):
    w = full("stencil3d")
    spec = dict(w.in_spec, sweep=((z0, 0, 0), (z1, 512, 512), (1, 1, 1)))
    got = run_collect(spec, w.inputs)
    assert np.array_equal(got, oracle.collect(spec, w.inputs))


@pytest.mark.parametrize("name", wl.CNN_NAMES)
def test_cnn_fullsize(name):
    """The convolutional workloads at full size in the benchmark's launch
    configuration, against the oracle over whole images: every pixel of the
    2048 x 2048 step (4.2 G multiply-adds in fp64), every frame estimate."""
    w = wl.make_cnn(name)
    import torch
    ins = [torch.from_numpy(a).cuda() for a in w.inputs]
    outs = [torch.from_numpy(a).cuda() for a in w.outputs]
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.FROM)
    m = api.CnnModel(w.model)
    var = api.variant(m, mi, mo)
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    got = np.stack([o.cpu().numpy().reshape(-1) for o in outs], 1)
    Y = oracle.cnn(w.model, oracle.gather(w.in_spec, w.inputs))
    worst, norm = assert_close(got, Y, RTOL["f32"], "%s full via %s" % (name, var))
    print("%s full [%s]: worst scaled %.3e, normwise %.3e" % (name, var, worst, norm))


def test_cnn_inplace_fullsize():
    """The 2048 x 2048 convolutional step written back into its own four
    fields: the inputs go to the snapshot record and the fused kernel reads
    them there; every pixel against the oracle's region (all gathers, then
    the model, then all writes) on the original fields."""
    import torch
    w = wl.make_cnn("weather_cnn")
    fields = [torch.from_numpy(a).cuda() for a in w.inputs]
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.CnnModel(w.model)
    var = api.variant(m, mi, mo)
    assert var == "snapshot+cnn_fused_f32", var
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    got = np.stack([f.cpu().numpy().reshape(-1) for f in fields], 1)
    Y = oracle.cnn(w.model, oracle.gather(w.in_spec, w.inputs))
    worst, norm = assert_close(got, Y, RTOL["f32"], "weather_cnn full, in place via %s" % var)
    print("weather_cnn full in place [%s]: worst scaled %.3e, normwise %.3e" % (var, worst, norm))


@pytest.mark.parametrize("name", ["stencil2d", "stencil3d"])
def test_inplace_step_fullsize_sampled(name):
    """One step written back into the fields it reads, at full size: the
    snapshot record (feature-major, 18.8 GB for the 512^3 grid) keeps the
    32-bit fused kernels; sampled outputs against the oracle's region on the
    original fields."""
    import torch
    w = full(name)
    fields = [torch.from_numpy(a).cuda() for a in w.inputs]
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.Model(w.model)
    var = api.variant(m, mi, mo)
    assert var.startswith("snapshot+mlp_" + w.compute), var
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    rows = wl.sample_rows(w.n_points, 2048, must=edges(w))
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model, rows)
    gotY = np.stack([f.reshape(-1)[torch.from_numpy(rows).cuda()].cpu().numpy() for f in fields], 1)
    worst, norm = assert_close(gotY, Y, RTOL[w.compute], "%s in place via %s" % (name, var))
    print("%s in place [%s] full size: worst %.3e normwise %.3e" % (name, var, worst, norm))
    del mi, mo, m


def test_layers_path_fullsize_sampled():
    """The 4,194,304 poses through a 6-1024-512-256-1 bf16 model, wider than
    the fused kernels take: layer by layer at the default chunk size (32
    chunks of 131,072 points), in the configuration the benchmark's --dims
    run times; 2^14 seeded poses plus the first and last against the oracle."""
    w = wl.make("poses")
    w.dims = [6, 1024, 512, 256, 1]
    w.model = wl.make_model(w.cfg, w.dims, w.compute)
    got, var = run_infer(w)
    assert var == "mlp_layers_bf16", var
    rows = wl.sample_rows(w.n_points, 1 << 14, must=np.array([0, w.n_points - 1], np.int64))
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model, rows)
    gotY = np.stack([a.reshape(-1)[rows] for a in got], 1)
    worst, norm = assert_close(gotY, Y, RTOL["bf16"], "poses wide via " + var)
    print("poses 6-1024-512-256-1 [%s]: %d sampled points, worst scaled %.3e normwise %.3e"
          % (var, len(rows), worst, norm))
    for a in got:
        assert not np.any(a.view(np.uint32) == wl.SENTINEL_BITS), "unwritten output element"

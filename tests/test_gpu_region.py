"""GPU tests of region execution control (``ml(infer | collect | predicated)``
and ``if``) and of the collection sink, through the C ABI.  The accurate path
is a stand-in that writes a known pattern, so recorded outputs have exact
expected values; recorded inputs are compared bit for bit with the oracle's
collect of the same arrays."""
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


class Setup:
    """A bond-pricing region of n points: 9 input arrays, 1 output array."""

    def __init__(self, n=5003):
        self.w = wl.make("bonds", n)
        self.ins = to_dev(self.w.inputs)
        self.outs = to_dev(self.w.outputs)
        self.mi = api.Map(self.w.in_spec, self.ins, _abi.TO)
        self.mo = api.Map(self.w.out_spec, self.outs, _abi.FROM)
        self.model = api.Model(self.w.model)
        self.calls = 0

    def pattern(self, k):
        return (np.arange(self.w.n_points, dtype=np.float32) * np.float32(0.5) + np.float32(k)).astype(np.float32)

    def accurate(self, k):
        """The region's original code: out[i] = 0.5 i + k, on the given stream."""
        import torch

        def run(stream_handle):
            self.calls += 1
            st = torch.cuda.ExternalStream(stream_handle) if stream_handle else torch.cuda.default_stream()
            with torch.cuda.stream(st):
                self.outs[0].copy_(torch.from_numpy(self.pattern(k)).cuda(non_blocking=False))
        return run

    def host_inputs(self):
        return [t.cpu().numpy() for t in self.ins]


def test_infer_mode_is_hpacml_infer():
    import torch
    s = Setup()
    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_INFER)
    r.run()
    torch.cuda.synchronize()
    got = s.outs[0].cpu().numpy().copy()
    s.outs[0].fill_(0)
    api.infer(s.model, s.mi, s.mo)
    torch.cuda.synchronize()
    assert np.array_equal(got.view(np.uint32), s.outs[0].cpu().numpy().view(np.uint32))
    assert r.samples == 0


def test_predicated_region_with_a_layer_by_layer_model():
    """A bond model wider than the fused kernels (9-600-300-1 fp32: the
    layer-by-layer path) under predicated control: the inferring run equals
    hpacml_infer bit for bit and the oracle within the fp32 bar; the
    collecting run records the inputs bit for bit."""
    import torch
    s = Setup()
    s.w.model = wl.make_model(s.w.cfg, [9, 600, 300, 1], "f32")
    s.model = api.Model(s.w.model)
    assert api.variant(s.model, s.mi, s.mo) == "mlp_layers_f32"
    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_PREDICATED, capacity=1)
    r.run(s.accurate(0), cond=True)
    torch.cuda.synchronize()
    got = s.outs[0].cpu().numpy().copy()
    s.outs[0].fill_(0)
    api.infer(s.model, s.mi, s.mo)
    torch.cuda.synchronize()
    assert np.array_equal(got.view(np.uint32), s.outs[0].cpu().numpy().view(np.uint32))
    Y = oracle.infer_rows(s.w.in_spec, s.w.inputs, s.w.model)
    assert_close(got.reshape(-1, 1), Y, RTOL["f32"], "region over mlp_layers_f32")
    r.run(s.accurate(3), cond=False)
    inp, out, _ = r.read()
    assert np.array_equal(inp[0].view(np.uint32), oracle.collect(s.w.in_spec, s.host_inputs()))
    assert np.array_equal(out[0].reshape(-1), s.pattern(3))


def test_collect_mode_records_inputs_outputs_and_time():
    import torch
    s = Setup()
    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_COLLECT, capacity=3)
    expect_in = []
    for k in range(3):
        # new inputs per invocation (the application's state changes)
        for t in s.ins:
            t.mul_(1.25).add_(0.5)
        torch.cuda.synchronize()
        expect_in.append(oracle.collect(s.w.in_spec, s.host_inputs()))
        r.run(s.accurate(k))
    assert s.calls == 3 and r.samples == 3
    ins, outs, t = r.read()
    for k in range(3):
        assert np.array_equal(ins[k].view(np.uint32), expect_in[k]), k
        assert np.array_equal(outs[k, :, 0], s.pattern(k)), k
    assert np.all(t > 0) and np.all(np.isfinite(t))


def test_predicated_toggles_inference_and_collection():
    import torch
    s = Setup()
    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_PREDICATED, capacity=4)
    Y = oracle.infer_rows(s.w.in_spec, s.w.inputs, s.w.model)
    for k, cond in enumerate([True, False, True, False]):
        r.run(s.accurate(k), cond=cond)
        torch.cuda.synchronize()
        got = s.outs[0].cpu().numpy()
        if cond:
            assert_close(got[:, None], Y, RTOL["f32"], "inference invocation %d" % k)
        else:
            assert np.array_equal(got, s.pattern(k))
    assert s.calls == 2 and r.samples == 2
    _, outs, _ = r.read()
    assert np.array_equal(outs[0, :, 0], s.pattern(1)) and np.array_equal(outs[1, :, 0], s.pattern(3))


def test_if_false_runs_the_accurate_path_only():
    import torch
    s = Setup()
    for mode in (_abi.MODE_INFER, _abi.MODE_COLLECT, _abi.MODE_PREDICATED):
        r = api.Region(s.model, s.mi, s.mo, mode, capacity=2)
        r.run(s.accurate(7), cond=True, enabled=False)
        torch.cuda.synchronize()
        assert np.array_equal(s.outs[0].cpu().numpy(), s.pattern(7))
        assert r.samples == 0
        r.close()


def test_full_sink_is_an_error_before_anything_runs_and_reset_reuses_it():
    import torch
    s = Setup(300)
    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_COLLECT, capacity=2)
    r.run(s.accurate(0))
    r.run(s.accurate(1))
    with pytest.raises(_abi.HpacmlError) as e:
        r.run(s.accurate(2))
    assert e.value.status == _abi.E_RANGE and s.calls == 2
    r.reset()
    assert r.samples == 0
    r.run(s.accurate(5))
    torch.cuda.synchronize()
    _, outs, _ = r.read()
    assert outs.shape == (1, 300, 1) and np.array_equal(outs[0, :, 0], s.pattern(5))
    # collecting needs the accurate path
    with pytest.raises(_abi.HpacmlError) as e:
        r.run(None)
    assert e.value.status == _abi.E_INVAL


def test_save_writes_the_region_group_as_npy(tmp_path):
    s = Setup(1000)
    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_COLLECT, capacity=2)
    r.run(s.accurate(0))
    r.run(s.accurate(1))
    ins, outs, t = r.read()
    r.save(str(tmp_path / "db"), "bonds_region")
    g = tmp_path / "db" / "bonds_region"
    a = np.load(g / "inputs.npy")
    b = np.load(g / "outputs.npy")
    c = np.load(g / "time.npy")
    assert a.dtype == np.float32 and a.shape == (2, 1000, 9) and np.array_equal(a, ins)
    assert b.shape == (2, 1000, 1) and np.array_equal(b, outs)
    assert c.shape == (2,) and np.array_equal(c, t)
    with pytest.raises(_abi.HpacmlError) as e:
        r.save(str(tmp_path / "db"), "a/b")
    assert e.value.status == _abi.E_INVAL


def test_region_create_errors():
    s = Setup(500)
    with pytest.raises(_abi.HpacmlError) as e:
        api.Region(s.model, s.mi, s.mo, 7)
    assert e.value.status == _abi.E_INVAL
    with pytest.raises(_abi.HpacmlError) as e:
        api.Region(s.model, s.mo, s.mi, _abi.MODE_INFER)      # directions swapped
    assert e.value.status == _abi.E_INVAL
    other = api.Model(wl.make_model(2, [9, 32, 2], "f32"))
    with pytest.raises(_abi.HpacmlError) as e:
        api.Region(other, s.mi, s.mo, _abi.MODE_COLLECT, capacity=1)
    assert e.value.status == _abi.E_SHAPE


def test_collect_around_a_convolutional_region():
    """A ParticleFilter-like region: frames in, one 2-value estimate per frame
    out; the two datasets have different point counts."""
    import torch
    w = wl.make_cnn("particle_cnn", (3, 64, 64))
    ins, outs = to_dev(w.inputs), to_dev(w.outputs)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.FROM)
    m = api.CnnModel(w.model)
    r = api.Region(m, mi, mo, _abi.MODE_PREDICATED, capacity=1)

    def accurate(handle):
        for k, o in enumerate(outs):
            o.fill_(float(k + 1))
    r.run(accurate, cond=False)
    r.run(None, cond=True)
    torch.cuda.synchronize()
    ins_rec, outs_rec, _ = r.read()
    assert ins_rec.shape == (1, 3 * 64 * 64, 1) and outs_rec.shape == (1, 3, 2)
    assert np.array_equal(ins_rec[0, :, 0], w.inputs[0].reshape(-1))
    assert np.array_equal(outs_rec[0], np.array([[1, 2]] * 3, np.float32))
    exp = [o.copy() for o in w.outputs]
    oracle.infer(w.in_spec, w.inputs, w.out_spec, exp, w.model)
    got = np.stack([o.cpu().numpy() for o in outs], 1)
    assert_close(got, np.stack(exp, 1), RTOL["f32"], "convolutional inference through a region")


def test_predicated_region_over_an_in_place_convolutional_step():
    """A MiniWeather-like step that writes its own fields, as a predicated
    region: inference invocations run the fused convolution on the snapshot
    of the fields; collecting invocations record the fields before and after
    the accurate path (here: every field scaled by 1/2)."""
    import torch
    w = wl.make_cnn("weather_cnn", (24, 70))
    fields = to_dev(w.inputs)
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.CnnModel(w.model)
    assert api.variant(m, mi, mo) == "snapshot+cnn_fused_f32"
    r = api.Region(m, mi, mo, _abi.MODE_PREDICATED, capacity=2)

    def accurate(handle):
        st = torch.cuda.ExternalStream(handle) if handle else torch.cuda.default_stream()
        with torch.cuda.stream(st):
            for f in fields:
                f.mul_(0.5)

    exp = [a.copy() for a in w.inputs]
    recs = []
    for k, cond in enumerate([True, False, True, False]):
        r.run(accurate, cond=cond)
        if cond:
            oracle.infer(w.in_spec, exp, w.out_spec, exp, w.model)
        else:
            recs.append(oracle.collect(w.in_spec, exp))
            exp = [(a * np.float32(0.5)).astype(np.float32) for a in exp]
            recs.append(oracle.collect(w.out_spec, exp))
        torch.cuda.synchronize()
        got = np.stack([f.cpu().numpy().reshape(-1) for f in fields], 1)
        assert_close(got, np.stack([a.reshape(-1) for a in exp], 1), RTOL["f32"], "invocation %d" % k)
        # carry the GPU's state forward so later comparisons see the same inputs
        exp = [f.cpu().numpy().copy() for f in fields]
    assert r.samples == 2
    ins, outs, t = r.read()
    for j in range(2):
        assert np.array_equal(ins[j].view(np.uint32), recs[2 * j]), j
        assert np.array_equal(outs[j].view(np.uint32), recs[2 * j + 1]), j
    assert np.all(t > 0)


def test_read_waits_for_a_region_run_on_a_side_stream():
    """A collecting region run on a non-blocking stream, read back with no
    synchronisation by the caller: the read must wait for each sample's
    records (the accurate path here queues ~10 ms of matrix products before it
    writes the outputs, so a read that did not wait would see stale data)."""
    import torch
    s = Setup(n=1 << 18)
    side = torch.cuda.Stream()
    a = torch.randn(4096, 4096, device="cuda")
    pat = [torch.from_numpy(s.pattern(k)).cuda() for k in range(2)]
    expect_in = oracle.collect(s.w.in_spec, s.host_inputs())
    torch.cuda.synchronize()

    def slow(k):
        def run(stream_handle):
            st = torch.cuda.ExternalStream(stream_handle)
            with torch.cuda.stream(st):
                x = a
                for _ in range(10):
                    x = (x @ a) * (1.0 / 64)
                s.outs[0].copy_(pat[k] + 0 * x[0, 0])
        return run

    r = api.Region(s.model, s.mi, s.mo, _abi.MODE_COLLECT, capacity=2)
    with torch.cuda.stream(side):
        for k in range(2):
            r.run(slow(k), stream=side)
    ins, outs, t = r.read()          # no synchronize before this
    for k in range(2):
        assert np.array_equal(ins[k].view(np.uint32), expect_in), k
        assert np.array_equal(outs[k, :, 0], s.pattern(k)), k
    assert np.all(t > 0)
    torch.cuda.synchronize()

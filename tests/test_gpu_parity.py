"""GPU parity: the HIP library (called through the C ABI) against the oracle.

Bars: gather/scatter/collect indexing bit-exact; fp32 inference within
|g - o| <= 1e-5 * max(|o|, s) and bf16 within 2e-2 (s = RMS of the oracle's
output column); no NaN; untouched elements keep their sentinel bits.
"""
import ctypes as C

import numpy as np
import pytest

import oracle
from paper_2407_18352_amd import _abi, api
from paper_2407_18352_amd import workloads as wl
from gpu_util import RTOL, assert_close, parity_stats, pure_relative, require_gpu, run_collect, run_infer, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def _flat_rows(arrs, rows):
    return np.stack([a.reshape(-1)[rows] for a in arrs], axis=1)


# ------------------------------------------------------------------ collect
@pytest.mark.parametrize("name", wl.NAMES)
def test_collect_small_bitexact(name):
    w = wl.make(name, "small")
    got = run_collect(w.in_spec, w.inputs)
    want = oracle.collect(w.in_spec, w.inputs)
    assert got.shape == want.shape
    assert np.array_equal(got, want)


def test_collect_input_output_pairs_ld():
    """bonds: record 9 inputs + 1 output per point in one [B x 10] buffer."""
    import torch
    w = wl.make("bonds", "small")
    outv = wl.rng(2, 100).uniform(0, 1, w.n_points).astype(np.float32)
    ins, outs = to_dev(w.inputs), to_dev([outv])
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.TO)
    rec = torch.empty((w.n_points, 10), device="cuda")
    rec.view(torch.int32).fill_(-1)
    api.collect(mi, rec, 10)
    api.collect(mo, rec[:, 9:], 10)
    torch.cuda.synchronize()
    got = rec.cpu().numpy().view(np.uint32)
    assert np.array_equal(got[:, :9], oracle.collect(w.in_spec, w.inputs))
    assert np.array_equal(got[:, 9:], oracle.collect(w.out_spec, [outv]))


def test_collect_preserves_bit_patterns_and_gaps():
    g = np.random.default_rng(3)
    a = g.standard_normal((33, 70)).astype(np.float32)
    bits = a.view(np.uint32)
    bits[0, 0], bits[1, 1], bits[2, 2] = 0x7FC0DEAD, 0x80000000, 0xFF800001
    spec = wl.window2d_spec(33, 70)
    got = run_collect(spec, [a], ld=13)
    assert np.array_equal(got[:, :9], oracle.collect(spec, [a]))
    assert np.all(got[:, 9:] == 0xFFFFFFFF)          # columns >= F untouched


@pytest.mark.parametrize("shape", [(33, 70), (5, 7), (61, 133)])
def test_collect_dense_and_offset_records(shape):
    """ld == F with a 16-byte aligned record (one contiguous run per tile,
    vector stores) and the same record shifted by one word (row-wise path);
    point counts that leave a ragged last tile and a word count that is not a
    multiple of 4."""
    import torch
    g = np.random.default_rng(sum(shape))
    a = g.standard_normal(shape).astype(np.float32)
    spec = wl.window2d_spec(*shape)
    want = oracle.collect(spec, [a])
    dev = to_dev([a])
    m = api.Map(spec, dev, _abi.TO)
    F, n = m.n_features, m.n_points
    rec = torch.empty(n * F + 8, device="cuda", dtype=torch.int32)
    for off in (0, 1):
        rec.fill_(-1)
        api.collect(m, rec[off:].view(torch.float32), F)
        torch.cuda.synchronize()
        got = rec.cpu().numpy().view(np.uint32)
        assert np.array_equal(got[off:off + n * F].reshape(n, F), want), off
        assert np.all(got[:off] == 0xFFFFFFFF) and np.all(got[off + n * F:] == 0xFFFFFFFF), off
    m.close()


@pytest.mark.parametrize("F", [1, 2, 3, 4])
def test_collect_few_features_several_points_per_lane(F):
    """Maps of 1-4 features take several points per lane: a periodic column
    window of F elements (edges on both sides), a point count that leaves a
    ragged last tile, dense, shifted and row-wise records, and one call that
    pairs it with a map of another width."""
    import torch
    g = np.random.default_rng(60 + F)
    ny, nx = 37, 71
    a = g.standard_normal((ny, nx)).astype(np.float32)
    spec = {"rank": 2, "slices": [((-1, 0), (F, 1))], "sweep": ((0, 0), (ny, nx), (1, 1)),
            "bnd": [wl.PERIODIC, wl.CLAMP]}
    want = oracle.collect(spec, [a])
    dev = to_dev([a])
    m = api.Map(spec, dev, _abi.TO)
    n = m.n_points
    assert m.n_features == F and n == ny * nx
    rec = torch.empty(n * (F + 1) + 8, device="cuda", dtype=torch.int32)
    for off, ld in ((0, F), (1, F), (0, F + 1)):
        rec.fill_(-1)
        api.collect(m, rec[off:off + n * ld].view(torch.float32), ld)
        torch.cuda.synchronize()
        got = rec.cpu().numpy().view(np.uint32)
        body = got[off:off + n * ld].reshape(n, ld)
        assert np.array_equal(body[:, :F], want), (off, ld)
        assert np.all(body[:, F:] == 0xFFFFFFFF) and np.all(got[:off] == 0xFFFFFFFF), (off, ld)
        assert np.all(got[off + n * ld:] == 0xFFFFFFFF), (off, ld)
    # paired with a 3-feature pointwise map of another point count
    b = [g.standard_normal(1234).astype(np.float32) for _ in range(3)]
    mb = api.Map(wl.pointwise_spec(1234), to_dev(b), _abi.TO)
    ra = torch.full((n, F), -1, device="cuda", dtype=torch.int32)
    rb = torch.full((1234, 3), -1, device="cuda", dtype=torch.int32)
    api.collect_pair(m, ra.view(torch.float32), F, mb, rb.view(torch.float32), 3)
    torch.cuda.synchronize()
    assert np.array_equal(ra.cpu().numpy().view(np.uint32), want)
    assert np.array_equal(rb.cpu().numpy().view(np.uint32), oracle.collect(wl.pointwise_spec(1234), b))


@pytest.mark.parametrize("name", wl.NAMES)
def test_collect_pair_matches_two_collects(name):
    """Both records of a region in one call == the oracle's two records."""
    import torch
    w = wl.make(name, "small")
    outv = [wl.rng(7, 100 + k).uniform(-1, 1, o.shape).astype(np.float32) for k, o in enumerate(w.outputs)]
    ins, outs = to_dev(w.inputs), to_dev(outv)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.TO)
    ri = torch.full((mi.n_points, mi.n_features), -1, device="cuda", dtype=torch.int32)
    ro = torch.full((mo.n_points, mo.n_features), -1, device="cuda", dtype=torch.int32)
    api.collect_pair(mi, ri.view(torch.float32), mi.n_features, mo, ro.view(torch.float32), mo.n_features)
    torch.cuda.synchronize()
    assert np.array_equal(ri.cpu().numpy().view(np.uint32), oracle.collect(w.in_spec, w.inputs))
    assert np.array_equal(ro.cpu().numpy().view(np.uint32), oracle.collect(w.out_spec, outv))


def test_collect_pair_interleaved_record_and_alias():
    """Inputs in columns 0..8 and the output in column 9 of one [B x 12]
    record; columns 10, 11 untouched.  Overlapping column ranges are
    HPACML_E_ALIAS with nothing written."""
    import torch
    w = wl.make("bonds", "small")
    outv = wl.rng(2, 101).uniform(0, 1, w.n_points).astype(np.float32)
    ins, outs = to_dev(w.inputs), to_dev([outv])
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.TO)
    rec = torch.full((w.n_points, 12), -1, device="cuda", dtype=torch.int32)
    rf = rec.view(torch.float32)
    api.collect_pair(mi, rf, 12, mo, rf[:, 9:], 12)
    torch.cuda.synchronize()
    got = rec.cpu().numpy().view(np.uint32)
    assert np.array_equal(got[:, :9], oracle.collect(w.in_spec, w.inputs))
    assert np.array_equal(got[:, 9:10], oracle.collect(w.out_spec, [outv]))
    assert np.all(got[:, 10:] == 0xFFFFFFFF)
    rec.fill_(-1)
    with pytest.raises(_abi.HpacmlError) as e:
        api.collect_pair(mi, rf, 12, mo, rf[:, 8:], 12)
    assert e.value.status == _abi.E_ALIAS
    torch.cuda.synchronize()
    assert np.all(rec.cpu().numpy().view(np.uint32) == 0xFFFFFFFF)


@pytest.mark.parametrize("shape", [(6, 8, 24), (3, 4, 32), (9, 8, 8)])
def test_collect_rank3_pair_with_general_map(shape):
    """Rank-3 windows (one call and the pair call), and a map with an offset
    beyond a signed byte, which takes the general kernel inside the pair
    call; all bit-exact."""
    import torch
    g = np.random.default_rng(sum(shape))
    fields = [g.standard_normal(shape).astype(np.float32) for _ in range(2)]
    spec = wl.sevenpoint3d_spec(*shape)
    far = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1)), ((0, 0, 130), (1, 1, 1))],
           "sweep": ((0, 0, 0), shape, (1, 1, 1)), "bnd": [wl.PERIODIC] * 3}
    dev = to_dev(fields)
    ma = api.Map(spec, dev, _abi.TO)
    mb = api.Map(far, dev, _abi.TO)
    want_a = oracle.collect(spec, fields)
    want_b = oracle.collect(far, fields)
    ra = torch.empty((ma.n_points, ma.n_features), device="cuda")
    rb = torch.empty((mb.n_points, mb.n_features), device="cuda")
    api.collect(ma, ra, ma.n_features)
    torch.cuda.synchronize()
    assert np.array_equal(ra.cpu().numpy().view(np.uint32), want_a)
    ra.fill_(0)
    api.collect_pair(ma, ra, ma.n_features, mb, rb, mb.n_features)
    torch.cuda.synchronize()
    assert np.array_equal(ra.cpu().numpy().view(np.uint32), want_a)
    assert np.array_equal(rb.cpu().numpy().view(np.uint32), want_b)


@pytest.mark.parametrize("R", [1, 2, 3])
def test_collect_random_maps_bitexact(R):
    """Random functors, boundary modes, steps, sub-ranges and strided views."""
    import torch
    g = np.random.default_rng(50 + R)
    done = 0
    for trial in range(40):
        ext = [int(g.integers(1, 40 if R < 3 else 12)) for _ in range(R)]
        bnd = [int(g.choice([wl.PERIODIC, wl.CLAMP])) for _ in range(R)]
        slices = [(tuple(int(g.integers(-3, 4)) for _ in range(R)),
                   tuple(int(g.integers(1, 3)) for _ in range(R))) for _ in range(int(g.integers(1, 4)))]
        start = [int(g.integers(0, e + 1)) for e in ext]
        stop = [int(g.integers(s, e + 1)) for s, e in zip(start, ext)]
        step = [int(g.integers(1, 4)) for _ in range(R)]
        spec = {"rank": R, "slices": slices, "sweep": (start, stop, step), "bnd": bnd}
        n_t = int(g.integers(1, 4))
        bigs = [g.standard_normal([2 * e for e in ext]).astype(np.float32) for _ in range(n_t)]
        views = [b[tuple(slice(1, 2 * e, 2) for e in ext)] for b in bigs]
        F = oracle.n_features(spec, views)
        if F > 256:
            continue
        want = oracle.collect(spec, views)
        dev_big = to_dev(bigs)
        dev = [d[tuple(slice(1, 2 * e, 2) for e in ext)] for d in dev_big]
        m = api.Map(spec, dev, _abi.TO)
        assert (m.n_points, m.n_features) == want.shape
        rec = torch.empty((max(1, m.n_points), F), device="cuda")
        api.collect(m, rec, F)
        torch.cuda.synchronize()
        got = rec.cpu().numpy().view(np.uint32)[: m.n_points]
        assert np.array_equal(got, want), (trial, spec)
        m.close()
        done += 1
    assert done > 20


# ------------------------------------------------------------------ infer
@pytest.mark.parametrize("name", wl.NAMES)
def test_infer_small(name):
    w = wl.make(name, "small")
    got, var = run_infer(w)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    exp = [o.copy() for o in w.outputs]
    oracle.scatter(w.out_spec, exp, Y)
    gotY = np.stack([a.reshape(-1) for a in got], 1)
    expY = np.stack([a.reshape(-1) for a in exp], 1)
    worst, norm = assert_close(gotY, expY, RTOL[w.compute], "%s via %s" % (name, var))
    line = "%s [%s]: worst scaled %.3e, normwise %.3e, max relative over |o| >= s %.3e" % (
        name, var, worst, norm, pure_relative(gotY, expY))
    if w.compute == "bf16":
        # context, not graded: against the unquantised fp64 model
        Yf = oracle.infer_rows(w.in_spec, w.inputs, dict(w.model, compute="f32"))
        expF = [o.copy() for o in w.outputs]
        oracle.scatter(w.out_spec, expF, Yf)
        _, normf, _ = parity_stats(gotY, np.stack([a.reshape(-1) for a in expF], 1))
        line += "; normwise vs the unquantised model %.3e" % normf
    print(line)


@pytest.mark.parametrize("name", wl.NAMES)
def test_infer_nan_inputs_follow_relu(name):
    """NaN inputs of either sign make the first layer NaN at the points that
    read them; ReLU takes NaN to 0 (max(x, 0) = 0 unless x > 0), so every
    output stays finite and matches the oracle under the usual bar."""
    w = wl.make(name, "small")
    g = np.random.default_rng(404)
    for k, a in enumerate(w.inputs):
        bits = a.reshape(-1).view(np.uint32)
        at = g.choice(bits.size, size=6, replace=False)
        bits[at[:3]] = 0x7FC00000
        bits[at[3:5]] = 0xFFC00001
        bits[at[5]] = 0x80000000                      # -0 stays a plain zero
    got, var = run_infer(w)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    assert not np.isnan(Y).any()
    exp = [o.copy() for o in w.outputs]
    oracle.scatter(w.out_spec, exp, Y)
    gotY = np.stack([a.reshape(-1) for a in got], 1)
    expY = np.stack([a.reshape(-1) for a in exp], 1)
    assert_close(gotY, expY, RTOL[w.compute], "%s via %s" % (name, var))


@pytest.mark.parametrize("shape", [(9, 5, 256), (3, 2, 128)])
def test_stencil3d_plane_order_visit(shape):
    """Rows made of whole tiles (128 points of the LDS-resident bf16 kernel,
    256 of the register-resident one); every cell must be written exactly as
    the oracle's region writes it."""
    w = wl.make("stencil3d", shape)
    got, var = run_infer(w)
    assert var.startswith("mlp_bf16r_h512"), var
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    exp = [o.copy() for o in w.outputs]
    oracle.scatter(w.out_spec, exp, Y)
    assert_close(np.stack([a.reshape(-1) for a in got], 1), np.stack([a.reshape(-1) for a in exp], 1),
                 RTOL["bf16"], "stencil3d %s via %s" % (shape, var))
    for a in got:
        assert not np.any(a.view(np.uint32) == wl.SENTINEL_BITS)


def test_infer_fast_paths_are_used():
    for name, want in [("options", "mlp_f32_h64"), ("bonds", "mlp_f32_h128"), ("stencil2d", "mlp_f32_h128"),
                       ("poses", "mlp_bf16r_h256"), ("stencil3d", "mlp_bf16r_h512")]:
        w = wl.make(name, {"stencil2d": (20, 40), "stencil3d": (6, 7, 9)}.get(name, 1000))
        _, var = run_infer(w)
        assert var.startswith(want), (name, var)


@pytest.mark.parametrize("compute, H, F_in, F_out, want", [
    ("f32", 64, 5, 1, "mlp_f32_h64_k16"), ("f32", 64, 33, 3, "mlp_f32_h64_k40"),
    ("f32", 64, 57, 8, "mlp_f32_h64_k64"), ("f32", 128, 16, 2, "mlp_f32_h128_k16"),
    ("f32", 128, 40, 4, "mlp_f32_h128_k40"), ("f32", 128, 64, 1, "mlp_f32_h128_k64"),
    ("bf16", 256, 13, 16, "mlp_bf16_h256"), ("bf16", 512, 7, 12, "mlp_bf16_h512"),
    ("bf16", 512, 7, 2, "mlp_bf16r_h512"), ("bf16", 512, 20, 3, "mlp_bf16r_h512"),
    ("bf16", 512, 45, 5, "mlp_bf16_h512"), ("bf16", 512, 61, 9, "mlp_bf16_h512"),
    ("bf16", 512, 35, 5, "mlp_bf16r_h512"), ("bf16", 512, 30, 8, "mlp_bf16r_h512"),
    ("bf16", 512, 42, 1, "mlp_bf16r_h512"),
    # 256 wide, one hidden-to-hidden layer: one and two first-layer K-steps
    ("bf16", 256, 6, 1, "mlp_bf16r_h256"), ("bf16", 256, 13, 4, "mlp_bf16r_h256"),
    ("bf16", 256, 17, 2, "mlp_bf16r_h256")])
def test_fast_kernels_input_widths(compute, H, F_in, F_out, want):
    """Every template variant of the MFMA kernels (input width classes,
    widths of hidden layers, output counts), pointwise maps with a ragged
    last tile, against the oracle.  The point counts give every wave (fp32)
    or block (bf16) more than one tile, so the next tile's gather overlaps
    the current one's layers."""
    n = {"f32": 140001, 256: 70001, 512: 40001}[compute if compute == "f32" else H]
    g = np.random.default_rng(F_in * 1000 + H)
    spec = wl.pointwise_spec(n)
    w = wl.Workload("widths", 0, compute, [F_in, H, H, F_out], spec, spec,
                    [g.uniform(-1, 1, n).astype(np.float32) for _ in range(F_in)],
                    [wl.sentinel_like((n,)) for _ in range(F_out)])
    w.model = wl.make_model(F_in + H, w.dims, compute)
    got, var = run_infer(w)
    assert var == want, var
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    assert_close(np.stack(got, 1), Y, RTOL[compute], var)


@pytest.mark.parametrize("case", ["h512_rank3_clamp_periodic_strided", "h256_rank2_shifted_periodic_output"])
def test_bf16r_window_boundaries(case):
    """The register-resident bf16 kernel on windowed maps whose windows
    leave the arrays along every dimension: clamp and periodic boundaries,
    a sub-sweep that starts inside the array, strided target views, and (for
    the 256-wide model) outputs written one row down with periodic wrap, so
    the branch-free boundary arithmetic of both the gathers and the scatter
    runs at every edge.  Several tiles per block and a ragged last tile."""
    import torch
    g = np.random.default_rng(2407)
    if case.startswith("h512"):
        bigs = [g.standard_normal((40, 64, 200)).astype(np.float32) for _ in range(2)]
        views_np = [b[:, :, ::2] for b in bigs]
        spec = {"rank": 3, "slices": [((-1, 0, -1), (3, 2, 3))], "sweep": ((1, 0, 3), (40, 64, 100), (1, 1, 1)),
                "bnd": [wl.CLAMP, wl.PERIODIC, wl.CLAMP]}
        F = oracle.n_features(spec, views_np)
        assert F == 36
        npts = oracle.n_points(spec, views_np)
        dims, H, want = [F, 512, 512, 3], 512, "mlp_bf16r_h512"
        out_spec = wl.pointwise_spec(npts)
        outs_np = [wl.sentinel_like((npts,)) for _ in range(3)]
        dev = [d[:, :, ::2] for d in to_dev(bigs)]
    else:
        ny, nx = 300, 500
        views_np = [g.standard_normal((ny, nx)).astype(np.float32) for _ in range(2)]
        spec = {"rank": 2, "slices": [((-1, -1), (2, 3))], "sweep": ((0, 0), (ny, nx), (1, 1)),
                "bnd": [wl.PERIODIC, wl.CLAMP]}
        F = oracle.n_features(spec, views_np)
        assert F == 12
        npts = ny * nx
        dims, H, want = [F, 256, 256, 256, 2], 256, "mlp_bf16r_h256"
        out_spec = {"rank": 2, "slices": [((1, 0), (1, 1))], "sweep": ((0, 0), (ny, nx), (1, 1)),
                    "bnd": [wl.PERIODIC, wl.NONE]}
        outs_np = [wl.sentinel_like((ny, nx)) for _ in range(2)]
        dev = to_dev(views_np)
    model = wl.make_model(90 + H // 256, dims, "bf16")
    Y = oracle.infer_rows(spec, views_np, model)
    exp = [o.copy() for o in outs_np]
    oracle.scatter(out_spec, exp, Y)
    outs = to_dev(outs_np)
    mi = api.Map(spec, dev, _abi.TO)
    mo = api.Map(out_spec, outs, _abi.FROM)
    m = api.Model(model)
    var = api.variant(m, mi, mo)
    assert var == want, var
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    got = np.stack([o.cpu().numpy().reshape(-1) for o in outs], 1)
    expY = np.stack([a.reshape(-1) for a in exp], 1)
    assert not np.any(got.view(np.uint32) == wl.SENTINEL_BITS), "unwritten output element"
    worst, norm = assert_close(got, expY, RTOL["bf16"], "%s via %s" % (case, var))
    print("%s [%s]: %d points, worst scaled %.3e, normwise %.3e" % (case, var, npts, worst, norm))
    mi.close(), mo.close(), m.close()


@pytest.mark.parametrize("compute, dims, want", [
    ("f32", [9, 96, 40, 1], "mlp_f32_h128_k16_padded"),          # bonds space: hidden 2 != hidden 1
    ("f32", [5, 50, 20, 1], "mlp_f32_h64_k16_padded"),           # options space
    ("f32", [36, 128, 100, 4], "mlp_f32_h128_k40_padded"),
    ("f32", [9, 128, 128, 1], "mlp_f32_h128_k16"),               # uniform: not padded
    ("bf16", [6, 256, 128, 64, 1], "mlp_bf16r_h256_padded"),     # MiniBUDE space: tapered, multiplier 0.5
    ("bf16", [10, 256, 192, 128, 64, 1], "mlp_bf16r_h256_padded"),
    ("bf16", [35, 400, 300, 5], "mlp_bf16r_h512_padded"),
    ("bf16", [17, 160, 100, 3], "mlp_bf16r_h256_padded"),         # one hidden-to-hidden layer
    ("bf16", [6, 200, 1], "mlp_bf16_h256_padded"),
    ("bf16", [6, 1024, 512, 256, 1], "mlp_layers_bf16"),         # wider than 512: layer by layer
])
def test_padded_hidden_layers(compute, dims, want):
    """Models whose hidden layers are uneven or narrower than a fast kernel's
    width run on that kernel with the hidden layers zero-padded (the added
    neurons have zero weights and bias): outputs against the oracle of the
    unpadded model.  Several tiles per block and a ragged last tile."""
    n = 70001 if compute == "bf16" else 140001
    g = np.random.default_rng(sum(dims) * 7 + len(dims))
    spec = wl.pointwise_spec(n)
    w = wl.Workload("padded", 0, compute, dims, spec, spec,
                    [g.uniform(-1, 1, n).astype(np.float32) for _ in range(dims[0])],
                    [wl.sentinel_like((n,)) for _ in range(dims[-1])])
    w.model = wl.make_model(50 + len(dims), dims, compute)
    got, var = run_infer(w)
    assert var == want, var
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    worst, norm = assert_close(np.stack(got, 1), Y, RTOL[compute], var)
    print("%s %s [%s]: worst scaled %.3e normwise %.3e" % (compute, dims, var, worst, norm))


@pytest.mark.parametrize("seed", range(12))
def test_random_model_shapes_dispatch(seed):
    """Seeded random multilayer perceptrons (1-5 layers, widths 1-1100,
    identity output layer as in the paper's models, random hidden activations
    in fp32 and ReLU in bf16, 1-40 inputs, 1-20 outputs) on 2,777 points of a rank-2
    clamped window map or a pointwise map: whichever kernel the library picks
    (fused, zero-padded, layer by layer) matches the oracle within the bar of
    the precision."""
    g = np.random.default_rng(9100 + seed)
    compute = "bf16" if g.random() < 0.5 else "f32"
    L = int(g.integers(1, 6))
    widths = [int(g.choice([g.integers(1, 65), g.integers(64, 300), g.integers(300, 1101)])) for _ in range(L - 1)]
    F_out = int(g.integers(1, 21))
    if g.random() < 0.5:
        # rank-2 clamped window: 1-4 fields x a (1-3) x (1-3) window
        ny, nx = 41, 67
        nf, wy, wx = int(g.integers(1, 5)), int(g.integers(1, 4)), int(g.integers(1, 4))
        spec = {"rank": 2, "slices": [((-(wy // 2), -(wx // 2)), (wy, wx))], "sweep": ((0, 0), (ny, nx), (1, 1)),
                "bnd": [wl.CLAMP, wl.CLAMP]}
        ins = [g.standard_normal((ny, nx)).astype(np.float32) for _ in range(nf)]
        F_in, n = nf * wy * wx, ny * nx
    else:
        n = 2777
        F_in = int(g.integers(1, 41))
        spec = wl.pointwise_spec(n)
        ins = [g.uniform(-1, 1, n).astype(np.float32) for _ in range(F_in)]
    dims = [F_in] + widths + [F_out]
    model = wl.make_model(60 + seed, dims, compute)
    if compute == "f32":
        # bf16 models keep ReLU hidden layers: in identity stacks a hidden
        # value at a bf16 rounding tie, which an fp32 sum in any order may
        # round the other way from the fp64 oracle, can move an output past
        # the bf16 bar (an fp32-accumulating CPU mirror moves it alike).
        model["act"] = [int(a) for a in g.integers(0, 2, L - 1)] + [wl.IDENTITY]
    w = wl.Workload("random", 0, compute, dims, spec, wl.pointwise_spec(n), ins,
                    [wl.sentinel_like((n,)) for _ in range(F_out)])
    w.model = model
    got, var = run_infer(w)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    worst, norm = assert_close(np.stack([a.reshape(-1) for a in got], 1), Y, RTOL[compute],
                               "%s %s acts %s via %s" % (compute, dims, model["act"], var))
    print("%s %s acts %s [%s]: worst scaled %.3e" % (compute, dims, model["act"], var, worst))


@pytest.mark.parametrize("compute", ["f32", "bf16"])
def test_limits_max_features_targets_width(compute):
    """The ABI's maxima in one region: 64 input targets x a 2x2 clamped
    window = 256 features, a 4096-wide hidden layer, 16 output targets
    (layer by layer); the same map's 256-feature record (64-bit collect)."""
    import torch
    g = np.random.default_rng(1024)
    shape = (23, 31)
    fields = [g.standard_normal(shape).astype(np.float32) for _ in range(64)]
    spec = {"rank": 2, "slices": [((0, 0), (2, 2))], "sweep": ((0, 0), shape, (1, 1)),
            "bnd": [wl.CLAMP, wl.CLAMP]}
    out_spec = {"rank": 2, "slices": [((0, 0), (1, 1))], "sweep": ((0, 0), shape, (1, 1)),
                "bnd": [wl.NONE, wl.NONE]}
    w = wl.Workload("limits", 0, compute, [256, 4096, 16], spec, out_spec, fields,
                    [wl.sentinel_like(shape) for _ in range(16)])
    w.model = wl.make_model(5, w.dims, compute)
    got, var = run_infer(w)
    assert var.startswith("mlp_layers"), var
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    assert_close(np.stack([a.reshape(-1) for a in got], 1), Y, RTOL[compute], var)
    m = api.Map(spec, to_dev(fields), _abi.TO)
    assert m.n_features == 256
    rec = torch.empty((m.n_points, 256), device="cuda")
    api.collect(m, rec, 256)
    torch.cuda.synchronize()
    assert np.array_equal(rec.cpu().numpy().view(np.uint32), oracle.collect(spec, fields))
    m.close()


def _one_hot_chain(F_in, H, n_hidden, pick, compute):
    """Layer 1 copies input i to hidden unit i; hidden layers copy unit o to
    unit o; the output layer picks input `pick`.  Exact on non-negative inputs."""
    dims = [F_in] + [H] * (n_hidden + 1) + [1]
    W, b = [], []
    W1 = np.zeros((H, F_in), np.float32)
    W1[np.arange(F_in), np.arange(F_in)] = 1
    W.append(W1)
    for _ in range(n_hidden):
        W.append(np.eye(H, dtype=np.float32))
    Wo = np.zeros((1, H), np.float32)
    Wo[0, pick] = 1
    W.append(Wo)
    b = [np.zeros(d, np.float32) for d in dims[1:]]
    return {"dims": dims, "W": W, "b": b, "act": [1] * (n_hidden + 1) + [0], "compute": compute}


@pytest.mark.parametrize("H, n_hidden, compute", [(64, 1, "f32"), (128, 2, "f32"), (128, 1, "f32"),
                                                  (256, 2, "bf16"), (512, 1, "bf16"), (96, 1, "f32")])
def test_one_hot_chain_bitexact(H, n_hidden, compute):
    w = wl.make("bonds", 4099)
    for pick in (0, 4, 8):
        w.model = _one_hot_chain(9, H, n_hidden, pick, compute)
        w.outputs = [wl.sentinel_like((4099,))]
        got, var = run_infer(w)
        x = w.inputs[pick]
        if compute == "bf16":
            x = oracle.bf16_bits(x).astype(np.uint32) << 16
            x = x.view(np.float32)
        assert np.array_equal(got[0].view(np.uint32), x.view(np.uint32)), (pick, var)


@pytest.mark.parametrize("shape", [(257, 300), (40, 1636)])
def test_windowed_f32_tile_ranges_per_xcd(shape):
    """Windowed fp32 launches of a full grid (256 blocks) split the tiles into
    one contiguous range per XCD: 2,410 tiles (ranges of 302, several tiles
    per wave, the last range short) and 2,045 tiles (ranges of 256, one tile
    per wave, the last range 253) match the oracle at every point."""
    w = wl.make("stencil2d", shape)
    got, var = run_infer(w)
    assert var == "mlp_f32_h128_k40"
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    exp = [o.copy() for o in w.outputs]
    oracle.scatter(w.out_spec, exp, Y)
    worst, norm = assert_close(np.stack([a.reshape(-1) for a in got], 1),
                               np.stack([a.reshape(-1) for a in exp], 1), RTOL["f32"], "%s via %s" % (shape, var))
    print("stencil2d %s [%s]: worst scaled %.3e" % (shape, var, worst))


def test_guard_band_and_subsweep():
    """A strided sub-sweep writes exactly its points; everything else keeps the
    sentinel bits."""
    ny, nx = 61, 133
    w = wl.make("stencil2d", (ny, nx))
    sweep = ((3, 5), (58, 120), (2, 3))
    w.in_spec = dict(w.in_spec, sweep=sweep)
    w.out_spec = dict(w.out_spec, sweep=sweep)
    got, var = run_infer(w)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    exp = [o.copy() for o in w.outputs]
    oracle.scatter(w.out_spec, exp, Y)
    mask = np.zeros((ny, nx), bool)
    mask[3:58:2, 5:120:3] = True
    for g in range(4):
        assert np.array_equal(got[g][~mask].view(np.uint32), exp[g][~mask].view(np.uint32))
        assert not np.any(got[g][mask].view(np.uint32) == wl.SENTINEL_BITS)
    assert_close(np.stack([a[mask] for a in got], 1), Y, RTOL["f32"], var)


def test_determinism_and_batch_order():
    """Same inputs twice -> identical bits; a shifted sub-sweep (other tile
    alignment) gives the same bits for the shared points."""
    w = wl.make("bonds", 9001)
    a, _ = run_infer(w)
    b, _ = run_infer(w)
    assert np.array_equal(a[0].view(np.uint32), b[0].view(np.uint32))
    w2 = wl.make("bonds", 9001)
    w2.in_spec = dict(w2.in_spec, sweep=((13,), (9001,), (1,)))
    w2.out_spec = dict(w2.out_spec, sweep=((13,), (9001,), (1,)))
    c, _ = run_infer(w2)
    assert np.array_equal(c[0][13:].view(np.uint32), a[0][13:].view(np.uint32))


@pytest.mark.parametrize("compute", ["f32", "bf16"])
def test_generic_shapes_rank3_clamp_strided(compute):
    """A rank-3 clamp/periodic map with steps over strided target views, with
    a hidden layer wider than the MFMA kernels take (layer by layer) and
    with uneven narrow hidden layers (an MFMA kernel, zero-padded)."""
    import torch
    g = np.random.default_rng(77)
    spec = {"rank": 3, "slices": [((-1, 0, 0), (3, 1, 1)), ((0, -2, 1), (1, 2, 2))],
            "sweep": ((1, 0, 2), (9, 11, 13), (2, 1, 3)), "bnd": [wl.CLAMP, wl.PERIODIC, wl.CLAMP]}
    bigs = [g.standard_normal((9, 11, 28)).astype(np.float32) for _ in range(2)]
    views = [b[:, :, ::2] for b in bigs]
    F = oracle.n_features(spec, views)
    npts = oracle.n_points(spec, views)
    wide = 200 if compute == "f32" else 600
    for dims, want in (([F, wide, 24, 3], "mlp_layers"), ([F, 40, 24, 3], "mlp_" + compute)):
        model = wl.make_model(9, dims, compute)
        outs_np = [wl.sentinel_like((npts,)) for _ in range(3)]
        Y = oracle.infer_rows(spec, views, model)
        dev = [d[:, :, ::2] for d in to_dev(bigs)]
        outs = to_dev(outs_np)
        mi = api.Map(spec, dev, _abi.TO)
        mo = api.Map(wl.pointwise_spec(npts), outs, _abi.FROM)
        m = api.Model(model)
        var = api.variant(m, mi, mo)
        assert var.startswith(want), var
        api.infer(m, mi, mo)
        torch.cuda.synchronize()
        got = np.stack([o.cpu().numpy() for o in outs], 1)
        assert_close(got, Y, RTOL[compute], "%s %s" % (var, dims))


@pytest.fixture
def small_chunks(monkeypatch):
    """Layer-by-layer plans created under this fixture take chunks of 1 MB of
    activations (at least 4096 points): at widths of 160 and more, a test of
    ~10^4 points crosses chunk borders and ends on a ragged chunk."""
    monkeypatch.setenv("HPACML_LAYERS_CHUNK_MB", "1")


@pytest.mark.parametrize("compute, dims, acts", [
    ("bf16", [6, 1024, 512, 256, 1], None),          # gather + first layer, 2 matmuls, last layer + scatter
    ("bf16", [35, 600, 5], None),                    # gather, matmul, last layer + scatter
    ("f32", [9, 300, 200, 1], None),
    ("f32", [36, 256, 256, 256, 256, 4], None),
    ("f32", [12, 160, 7], [1, 1]),                   # no matmul; ReLU on the output layer too
    ("bf16", [10, 700, 300, 3], [0, 1, 0]),          # an identity first layer
    ("bf16", [6, 600, 2], None),                     # no matmul
    ("f32", [10, 300, 12], None),                    # 12 outputs: matmul + scatter
    ("bf16", [40, 700, 16], [1, 1]),                 # gather, 2 matmuls, scatter; ReLU output
    ("f32", [9, 3], None),                           # one layer: gather, matmul, scatter
    ("bf16", [20, 5], None),
    ("f32", [11, 1000, 1], None),                    # odd input width; 1000 neurons = 250 groups of 4
    ("bf16", [3, 1000, 9], None),                    # 125 groups of 8; 9 outputs
    ("bf16", [6, 4096, 1], None),                    # 4096 neurons: gather, 2 matmuls, scatter
    ("bf16", [6, 2048, 2], None),                    # 256 groups of 8: the widest fused first layer
    ("f32", [4, 1024, 1500, 1], None),               # 256 groups of 4; 1500 inputs to the last layer
    ("f32", [9, 2048, 512, 3], None),
])
def test_layers_path_chunks_and_tail(compute, dims, acts, small_chunks):
    """Shapes outside the fused kernels run layer by layer (first layer fused
    with the gather for narrow inputs, a matmul per middle layer with bias
    and activation in its epilogue, last layer fused with the scatter for at
    most 8 outputs): 10,001 points, for the wide models in chunks of 4096
    and a ragged last chunk, against the oracle on every point."""
    n = 10001
    g = np.random.default_rng(sum(dims) + 3 * len(dims))
    spec = wl.pointwise_spec(n)
    w = wl.Workload("layers", 0, compute, dims, spec, spec,
                    [g.uniform(-1, 1, n).astype(np.float32) for _ in range(dims[0])],
                    [wl.sentinel_like((n,)) for _ in range(dims[-1])])
    w.model = wl.make_model(70 + len(dims), dims, compute)
    if acts is not None:
        w.model["act"] = list(acts)
    got, var = run_infer(w)
    assert var == "mlp_layers_" + compute, var
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    worst, norm = assert_close(np.stack(got, 1), Y, RTOL[compute], var)
    print("%s %s [%s]: worst scaled %.3e normwise %.3e" % (compute, dims, var, worst, norm))


def test_layers_path_in_place_across_chunks(small_chunks):
    """A 3x3-window step written back into its own fields, one field stored
    transposed (maps outside the 32-bit form), 6,300 cells in two chunks:
    the snapshot record keeps the second chunk's inputs from the first
    chunk's outputs."""
    import torch
    w = wl.make("stencil2d", (70, 90))
    fields = to_dev(w.inputs)
    fields[1] = torch.from_numpy(np.ascontiguousarray(w.inputs[1].T)).cuda().t()
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.Model(w.model)
    var = api.variant(m, mi, mo)
    assert var == "snapshot+mlp_layers_f32", var
    exp = [a.copy() for a in w.inputs]
    api.infer(m, mi, mo)
    oracle.infer(w.in_spec, exp, w.out_spec, exp, w.model)
    torch.cuda.synchronize()
    got = np.stack([f.cpu().numpy().reshape(-1) for f in fields], 1)
    want = np.stack([a.reshape(-1) for a in exp], 1)
    assert_close(got, want, RTOL["f32"], "in place across chunks via " + var)


@pytest.mark.parametrize("compute, dims", [("f32", [9, 300, 40, 2]), ("bf16", [9, 640, 40, 2]),
                                           ("f32", [9, 2500, 40, 2])])
def test_general_kernel_through_noalloc(compute, dims):
    """hpacml_infer_noalloc keeps the general fused kernel for shapes that
    hpacml_infer runs layer by layer (no workspace): both against the
    oracle, up to a 2500-wide layer (3 points per tile in LDS)."""
    import torch
    n = 3001
    g = np.random.default_rng(5)
    spec = wl.pointwise_spec(n)
    ins = [g.uniform(-1, 1, n).astype(np.float32) for _ in range(9)]
    model = wl.make_model(31, dims, compute)
    Y = oracle.infer_rows(spec, ins, model)
    m = api.Model(model)
    for noalloc in (False, True):
        outs = to_dev([wl.sentinel_like((n,)) for _ in range(2)])
        mi = api.Map(spec, to_dev(ins), _abi.TO)
        mo = api.Map(spec, outs, _abi.FROM)
        if noalloc:
            st = torch.cuda.current_stream().cuda_stream
            assert _abi.lib().hpacml_infer_noalloc(m.handle, mi.handle, mo.handle, st) == _abi.OK
        else:
            assert api.variant(m, mi, mo) == "mlp_layers_" + compute
            api.infer(m, mi, mo)
        torch.cuda.synchronize()
        got = np.stack([o.cpu().numpy() for o in outs], 1)
        assert_close(got, Y, RTOL[compute], "noalloc" if noalloc else "infer")
        mi.close(), mo.close()
    m.close()


# ------------------------------------------------------------------ errors
def test_errors_are_reported_before_launch():
    import torch
    w = wl.make("bonds", 1000)
    ins, outs = to_dev(w.inputs), to_dev(w.outputs)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.FROM)
    model = api.Model(w.model)
    # host memory is not a device pointer
    host = [torch.from_numpy(a) for a in w.inputs]
    with pytest.raises(_abi.HpacmlError) as e:
        api.Map(w.in_spec, host, _abi.TO)
    assert e.value.status == _abi.E_INVAL
    # point-count mismatch
    short = api.Map(wl.pointwise_spec(999), [o[:999] for o in outs], _abi.FROM)
    with pytest.raises(_abi.HpacmlError) as e:
        api.infer(model, mi, short)
    assert e.value.status == _abi.E_SHAPE
    # wrong direction
    with pytest.raises(_abi.HpacmlError) as e:
        api.infer(model, mo, mi)
    assert e.value.status == _abi.E_INVAL
    # two outputs that can write one element
    mi999 = api.Map(wl.pointwise_spec(999), [x[:999] for x in ins], _abi.TO)
    two = api.Model(wl.make_model(2, [9, 64, 2], "f32"))
    racing = api.Map(wl.pointwise_spec(999), [outs[0][:999], outs[0][1:]], _abi.FROM)
    with pytest.raises(_abi.HpacmlError) as e:
        api.infer(two, mi999, racing)
    assert e.value.status == _abi.E_ALIAS
    assert api.variant(two, mi999, racing) is None
    # element-for-element in place is allowed
    inplace = api.Map(w.out_spec, [ins[3]], _abi.FROM)
    api.infer(model, mi, inplace)
    torch.cuda.synchronize()
    # a record leading dimension that runs past the end of the allocation
    rec = torch.empty((999, 9), device="cuda")
    with pytest.raises(_abi.HpacmlError) as e:
        api.collect(mi, rec, 1 << 22)
    assert e.value.status == _abi.E_RANGE
    # ld smaller than the feature count
    with pytest.raises(_abi.HpacmlError) as e:
        api.collect(mi, rec, 8)
    assert e.value.status == _abi.E_SHAPE
    # a record overlapping a mapped input
    with pytest.raises(_abi.HpacmlError) as e:
        api.collect(mi, ins[0][:90].view(10, 9), 9)
    assert e.value.status in (_abi.E_ALIAS, _abi.E_RANGE)
    # extents beyond the allocation (1 GiB view of a 400-byte tensor)
    t = torch.zeros(100, device="cuda")
    L = _abi.lib()
    n_big = 1 << 28
    f, keep = api._functor(wl.pointwise_spec(n_big), 1)
    sw, bnd = api._sweep(wl.pointwise_spec(n_big))
    arr = (_abi.Array * 1)(api.array_desc(t.data_ptr(), (n_big,), (1,)))
    h = C.c_void_p()
    assert L.hpacml_map_create(C.byref(f), _abi.TO, arr, 1, C.byref(sw), bnd, C.byref(h)) == _abi.E_RANGE
    assert h.value is None
    # zero points: OK, nothing launched
    e0 = api.Map({"rank": 1, "slices": [((0,), (1,))], "sweep": ((5,), (5,), (1,)), "bnd": [0]},
                 [ins[0]], _abi.TO)
    assert e0.n_points == 0
    api.collect(e0, rec, 9)


def test_inplace_pointwise_matches_oracle():
    """Element-for-element in-place update: the output overwrites input 0 in
    one pass (each point reads its own element before writing it)."""
    import torch
    w = wl.make("options", 5000)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    ins = to_dev(w.inputs)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, [ins[0]], _abi.FROM)
    m = api.Model(w.model)
    assert not api.variant(m, mi, mo).startswith("snapshot+")
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    assert_close(ins[0].cpu().numpy()[:, None], Y, RTOL["f32"], "in place")


def test_inplace_shifted_output_reads_snapshot():
    """Outputs written one element past the inputs they overwrite: point b's
    output lands on point b+1's input, which must still be read as it was."""
    import torch
    w = wl.make("bonds", 999)
    big = [np.concatenate([a, np.float32([0.5])]) for a in w.inputs]
    ins = to_dev(big)
    mi = api.Map(wl.pointwise_spec(999), [x[:999] for x in ins], _abi.TO)
    mo = api.Map(wl.pointwise_spec(999), [ins[0][1:]], _abi.FROM)
    m = api.Model(w.model)
    var = api.variant(m, mi, mo)
    assert var.startswith("snapshot+mlp_f32"), var
    exp = [a.copy() for a in big]
    Y = oracle.infer_rows(wl.pointwise_spec(999), [a[:999] for a in exp], w.model)
    exp[0][1:] = Y[:, 0]
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    got = ins[0].cpu().numpy()
    assert got[0] == big[0][0]
    assert_close(got[1:, None], exp[0][1:, None], RTOL["f32"], "shifted in place via " + var)


def test_inplace_three_fields_shifted_output_reads_snapshot():
    """Three input fields (a feature-major snapshot record of three rows);
    the output lands one element past the points of field 1."""
    import torch
    n = 1999
    g = np.random.default_rng(71)
    big = [g.uniform(-1, 1, n + 1).astype(np.float32) for _ in range(3)]
    model = wl.make_model(5, [3, 64, 64, 1], "f32")
    ins = to_dev(big)
    spec = wl.pointwise_spec(n)
    mi = api.Map(spec, [x[:n] for x in ins], _abi.TO)
    mo = api.Map(spec, [ins[1][1:]], _abi.FROM)
    m = api.Model(model)
    var = api.variant(m, mi, mo)
    assert var.startswith("snapshot+"), var
    Y = oracle.infer_rows(spec, [x[:n] for x in big], model)
    api.infer(m, mi, mo)
    torch.cuda.synchronize()
    got = [x.cpu().numpy() for x in ins]
    assert np.array_equal(got[0], big[0]) and np.array_equal(got[2], big[2]) and got[1][0] == big[1][0]
    assert_close(got[1][1:, None], Y, RTOL["f32"], "three fields shifted in place via " + var)


@pytest.mark.parametrize("name, size, steps", [("stencil2d", (20, 40), 2), ("stencil2d", (3, 130), 1),
                                               ("stencil3d", (6, 7, 9), 1)])
def test_inplace_window_update_reads_snapshot(name, size, steps):
    """A stencil region that writes its results back into the fields its
    windows read (a time step advanced in place).  Every point's window is
    read before any output is written, so each step equals the oracle's
    region (all gathers, then the model, then all scatters) on the same
    arrays; later steps reuse the map's snapshot record."""
    import torch
    w = wl.make(name, size)
    fields = to_dev(w.inputs)
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.Model(w.model)
    var = api.variant(m, mi, mo)
    assert var.startswith("snapshot+mlp_" + w.compute), var
    exp = [a.copy() for a in w.inputs]
    for _ in range(steps):
        api.infer(m, mi, mo)
        oracle.infer(w.in_spec, exp, w.out_spec, exp, w.model)
    torch.cuda.synchronize()
    got = np.stack([f.cpu().numpy().reshape(-1) for f in fields], 1)
    want = np.stack([a.reshape(-1) for a in exp], 1)
    worst, norm = assert_close(got, want, RTOL[w.compute], "%s in place via %s" % (name, var))
    print("%s %s in place, %d steps [%s]: worst scaled %.3e, normwise %.3e" % (name, size, steps, var, worst,
                                                                                norm))


def test_inplace_window_update_general_maps():
    """The same in-place stencil step with one field stored transposed: the
    targets' strides differ, so both maps take the general (64-bit) form."""
    import torch
    w = wl.make("stencil2d", (12, 20))
    fields = to_dev(w.inputs)
    fields[1] = torch.from_numpy(np.ascontiguousarray(w.inputs[1].T)).cuda().t()
    mi = api.Map(w.in_spec, fields, _abi.TO)
    mo = api.Map(w.out_spec, fields, _abi.FROM)
    m = api.Model(w.model)
    var = api.variant(m, mi, mo)
    assert var == "snapshot+mlp_layers_f32", var
    exp = [a.copy() for a in w.inputs]
    api.infer(m, mi, mo)
    oracle.infer(w.in_spec, exp, w.out_spec, exp, w.model)
    torch.cuda.synchronize()
    got = np.stack([f.cpu().numpy().reshape(-1) for f in fields], 1)
    want = np.stack([a.reshape(-1) for a in exp], 1)
    assert_close(got, want, RTOL["f32"], "general in place via " + var)


@pytest.mark.parametrize("case", ["options", "stencil3d", "inplace_stencil2d", "weather_cnn", "particle_cnn"])
def test_graph_captured_inference_replays(case):
    """hpacml_infer captured in a HIP graph and
    replayed several times, with eager work and synchronisations between the
    replays: every replay's outputs equal the eager call's bit for bit (the
    frame stack: conv + pool, split-K products, the closing kernel)."""
    import torch
    if case == "weather_cnn":
        w = wl.make_cnn("weather_cnn", (40, 130))
        model = api.CnnModel(w.model)
    elif case == "particle_cnn":
        w = wl.make_cnn("particle_cnn", "small")
        model = api.CnnModel(w.model)
    else:
        w = wl.make({"inplace_stencil2d": "stencil2d"}.get(case, case),
                    {"options": 5000, "stencil3d": (6, 7, 9), "inplace_stencil2d": (20, 40)}[case])
        model = api.Model(w.model)
    ins = to_dev(w.inputs)
    inplace = case.startswith("inplace")
    outs = ins if inplace else to_dev(w.outputs)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.FROM)
    side = torch.cuda.Stream()

    def reset():
        for t, a in zip(ins, w.inputs):
            t.copy_(torch.from_numpy(a))
        if not inplace:
            for t, a in zip(outs, w.outputs):
                t.copy_(torch.from_numpy(a))
        torch.cuda.synchronize()

    # eager reference: one call (in place: one step from the original fields)
    reset()
    with torch.cuda.stream(side):
        api.infer(model, mi, mo, side)
    torch.cuda.synchronize()
    want = [t.cpu().numpy().copy() for t in outs]
    # capture: lazy set-up (the snapshot record) already happened in the eager call
    g = torch.cuda.CUDAGraph()
    reset()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            api.infer(model, mi, mo, side)
    for k in range(4):
        reset()
        scratch = torch.randn(1 << 16, device="cuda")
        (scratch * 2).sum().item()                      # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for a, t in zip(want, outs):
            assert np.array_equal(a.view(np.uint32), t.cpu().numpy().view(np.uint32)), (case, k)

"""Pins of the CPU oracle against things other than itself.

Each check is chosen so that a plausible slip in the oracle (a dropped term, a
wrong sign or index, a transposed operand, a wrong wrap) fails at least one:

* brute-force enumeration of every window and boundary case with numpy's own
  padding (``np.pad`` wrap/edge) and strided slicing;
* the paper's worked 5-point example (Fig. 2; Sec. IV-A extraction example),
  both from a hand-written fixture and from torch slicing + ``cat``;
* one-hot weights that reproduce the gathered inputs bit for bit;
* a single linear layer equal to a float64 matmul (exact on small integers);
* multi-layer nets equal to torch fp64 ``Linear``/``ReLU`` stacks;
* the 2-D window map + MLP equal to torch ``Conv2d`` with circular padding and
  1x1 convolutions; the 3-D 7-point map equal to a masked ``Conv3d``;
* batch-order invariance (permutation, sub-sweeps);
* bf16 rounding equal to torch's conversion on every fp32 bit pattern.
"""
import itertools
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2407_18352_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- brute force
def _brute_gather(spec, targets):
    """Independent formulation: pad every target per dimension with numpy
    (wrap = periodic, edge = clamp, zero-width for none), then take each slice
    element as one strided slice of the padded array."""
    R = spec["rank"]
    start, stop, step = spec["sweep"]
    bnd = spec["bnd"]
    shape = targets[0].shape
    n = [max(0, -(-(stop[d] - start[d]) // step[d])) for d in range(R)]
    lo_all = [min([0] + [s[0][d] for s in spec["slices"]]) for d in range(R)]
    hi_all = [max([0] + [s[0][d] + s[1][d] - 1 for s in spec["slices"]]) for d in range(R)]
    feats = []
    for a in targets:
        pad = a
        pw = []
        for d in range(R):
            before, after = -lo_all[d], hi_all[d]
            if bnd[d] == wl.NONE:
                # out-of-range must be an error: check explicitly
                if min(n) > 0:
                    first = start[d] + lo_all[d]
                    last = start[d] + (n[d] - 1) * step[d] + hi_all[d]
                    if first < 0 or last >= shape[d]:
                        raise IndexError("out of range")
                before = after = 0
            mode = "wrap" if bnd[d] == wl.PERIODIC else "edge"
            width = [(0, 0)] * R
            width[d] = (before, after)
            if before or after:
                pad = np.pad(pad, width, mode=mode)
            pw.append(before)
        for lo, cnt in spec["slices"]:
            for e in itertools.product(*[range(c) for c in cnt]):
                idx = tuple(slice(start[d] + lo[d] + e[d] + pw[d],
                                  start[d] + lo[d] + e[d] + pw[d] + n[d] * step[d],
                                  step[d]) if n[d] > 0 else slice(0, 0)
                            for d in range(R))
                feats.append(pad[idx].reshape(-1))
    if not feats:
        return np.zeros((int(np.prod(n)), 0))
    return np.stack(feats, axis=1).astype(np.float64)


def _rand_map(g, R):
    ext = [int(g.choice([1, 2, 3, 5, 7])) for _ in range(R)]
    bnd = [int(g.choice([wl.PERIODIC, wl.CLAMP, wl.NONE])) for _ in range(R)]
    slices = []
    for _ in range(int(g.integers(1, 4))):
        lo = [int(g.integers(-3, 4)) for _ in range(R)]
        cnt = [int(g.integers(1, 4)) for _ in range(R)]
        slices.append((tuple(lo), tuple(cnt)))
    start, stop, step = [], [], []
    for d in range(R):
        a = int(g.integers(0, ext[d] + 1))
        b = int(g.integers(a, ext[d] + 1))
        start.append(a), stop.append(b), step.append(int(g.choice([1, 2, 3])))
    return ext, {"rank": R, "slices": slices, "sweep": (tuple(start), tuple(stop), tuple(step)),
                 "bnd": bnd}


def _targets(g, ext, n_t, strided):
    out = []
    for _ in range(n_t):
        if strided:
            big = g.standard_normal([2 * e + 1 for e in ext]).astype(np.float32)
            a = big[tuple(slice(1, 1 + 2 * e, 2) for e in ext)]
        else:
            a = g.standard_normal(ext).astype(np.float32)
        out.append(a)
    return out


@pytest.mark.parametrize("R", [1, 2, 3])
def test_gather_brute_force_random_maps(R):
    g = np.random.default_rng(1000 + R)
    checked = errors = 0
    for trial in range(150):
        ext, spec = _rand_map(g, R)
        targets = _targets(g, ext, int(g.integers(1, 4)), strided=bool(trial % 2))
        try:
            want = _brute_gather(spec, targets)
        except IndexError:
            with pytest.raises(ValueError):
                oracle.gather(spec, targets)
            errors += 1
            continue
        got = oracle.gather(spec, targets)
        assert got.shape == want.shape
        assert np.array_equal(got.view(np.uint64), want.view(np.uint64))
        checked += 1
    assert checked > 50 and errors > 5


def test_every_offset_and_extent_rank1():
    """Every offset -3..3 (incl. |o| >= extent) on every extent 1..7, both
    wrapping modes, every step: the element index is fixed by hand formulas
    of modular arithmetic / clamping in numpy."""
    for ext in range(1, 8):
        a = np.arange(ext, dtype=np.float32) + 100
        for o in range(-3, 4):
            for c in (1, 2, 3):
                for step in (1, 2, 3):
                    for bnd in (wl.PERIODIC, wl.CLAMP):
                        spec = {"rank": 1, "slices": [((o,), (c,))],
                                "sweep": ((0,), (ext,), (step,)), "bnd": [bnd]}
                        X = oracle.gather(spec, [a])
                        p = np.arange(0, ext, step)[:, None] + o + np.arange(c)[None, :]
                        q = np.mod(p, ext) if bnd == wl.PERIODIC else np.clip(p, 0, ext - 1)
                        assert np.array_equal(X, a[q].astype(np.float64))


def test_out_of_range_without_boundary_is_an_error():
    a = np.zeros((5, 5), np.float32)
    spec = wl.window2d_spec(5, 5)
    spec["bnd"] = [wl.NONE, wl.PERIODIC]
    with pytest.raises(ValueError):
        oracle.gather(spec, [a])
    spec["sweep"] = ((1, 0), (4, 5), (1, 1))      # interior in the unbounded dim
    assert oracle.gather(spec, [a]).shape == (15, 9)


def test_empty_sweeps_and_counts():
    a = np.zeros((6, 4), np.float32)
    spec = {"rank": 2, "slices": [((0, 0), (1, 1))], "sweep": ((2, 0), (2, 4), (1, 1)),
            "bnd": [0, 0]}
    assert oracle.n_points(spec, [a]) == 0
    assert oracle.gather(spec, [a]).shape == (0, 1)
    spec["sweep"] = ((1, 0), (6, 4), (2, 3))
    assert oracle.n_points(spec, [a]) == 3 * 2              # ceil(5/2) * ceil(4/3)
    assert [oracle.point_coords(spec, [a], b) for b in range(6)] == \
        [(1, 0), (1, 3), (3, 0), (3, 3), (5, 0), (5, 3)]


# ------------------------------------------------------------ paper example
def _read_golden(name):
    rows, meta = [], {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if line.startswith("# ") and ":" in line and line[2:].split(":")[0].strip() in (
                    "shape", "first_access_of_slice0", "offset_of_slice0"):
                k, v = line[2:].split(":")
                meta[k.strip()] = [int(x) for x in v.split()]
            elif line and not line.startswith("#"):
                ij, f = line.split(":")
                rows.append(([int(x) for x in ij.split()], [float(x) for x in f.split()]))
    return rows, meta


def test_paper_fig2_example_golden():
    rows, meta = _read_golden("paper_fig2_stencil.txt")
    N, M = 4, 5
    t = (10 * np.arange(N)[:, None] + np.arange(M)[None, :]).astype(np.float32)
    ifnctr = [((-1, 0), (1, 1)), ((1, 0), (1, 1)), ((0, -1), (1, 3))]
    spec = {"rank": 2, "slices": ifnctr, "sweep": ((1, 1), (N - 1, M - 1), (1, 1)), "bnd": [0, 0]}
    X = oracle.gather(spec, [t])
    assert list(X.shape) == [meta["shape"][0] * meta["shape"][1], meta["shape"][2]]
    for b, (ij, feats) in enumerate(rows):
        assert oracle.point_coords(spec, [t], b) == tuple(ij)
        assert X[b].tolist() == feats
    # the offset (-1, 0) of slice [i-1, j] lands on t[0][1] at the first sweep point
    first = [1 + o for o in meta["offset_of_slice0"]]
    assert first == meta["first_access_of_slice0"]
    assert X[0, 0] == t[tuple(first)]


def test_paper_fig2_equals_wrap_and_cat():
    """Tensor Wrapping (strided views) + Tensor Composition (flatten + cat),
    done with torch on the paper's example functor (Sec. IV-A)."""
    g = np.random.default_rng(7)
    N, M = 9, 13
    t = g.standard_normal((N, M)).astype(np.float32)
    T = torch.from_numpy(t)
    views = [T[0:N - 2, 1:M - 1].unsqueeze(-1),                   # [i-1, j]
             T[2:N, 1:M - 1].unsqueeze(-1),                       # [i+1, j]
             torch.stack([T[1:N - 1, 0:M - 2], T[1:N - 1, 1:M - 1], T[1:N - 1, 2:M]], -1)]
    want = torch.cat(views, dim=-1).reshape(-1, 5).double().numpy()
    spec = {"rank": 2, "slices": [((-1, 0), (1, 1)), ((1, 0), (1, 1)), ((0, -1), (1, 3))],
            "sweep": ((1, 1), (N - 1, M - 1), (1, 1)), "bnd": [0, 0]}
    assert np.array_equal(oracle.gather(spec, [t]), want)
    # the `from` side: ofnctr [i, j, 0:1] = ([i, j]) on tnew[1:N-1, 1:M-1]
    tnew = np.full((N, M), -7.0, np.float32)
    Y = g.standard_normal(((N - 2) * (M - 2), 1)).astype(np.float32)
    ospec = {"rank": 2, "slices": [((0, 0), (1, 1))], "sweep": ((1, 1), (N - 1, M - 1), (1, 1)),
             "bnd": [0, 0]}
    oracle.scatter(ospec, [tnew], Y)
    ref = np.full((N, M), -7.0, np.float32)
    ref[1:N - 1, 1:M - 1] = Y.reshape(N - 2, M - 2)
    assert np.array_equal(tnew, ref)


# ---------------------------------------------------------------- collect
def test_collect_is_bitwise_copy_of_gather():
    g = np.random.default_rng(3)
    a = g.standard_normal((6, 7)).astype(np.float32)
    bits = a.view(np.uint32)
    bits[0, 0] = 0x7FC0DEAD   # NaN payload must survive
    bits[1, 1] = 0x80000000   # -0
    bits[2, 2] = 0xFF800001   # signalling-NaN pattern
    spec = wl.window2d_spec(6, 7)
    D = oracle.collect(spec, [a], ld=11)
    # compare as patterns: build the expected patterns with integer indexing
    pad = np.pad(bits, 1, mode="wrap")
    exp = np.stack([pad[1 + di:7 + di, 1 + dj:8 + dj].reshape(-1)
                    for di in (-1, 0, 1) for dj in (-1, 0, 1)], 1)
    assert np.array_equal(D[:, :9], exp)
    assert np.all(D[:, 9:] == 0)


# ---------------------------------------------------------------- model pins
def _one_hot_model(F, perm, compute="f32", act=0):
    W = np.zeros((F, F), np.float32)
    W[np.arange(F), perm] = 1.0
    return {"dims": [F, F], "W": [W], "b": [np.zeros(F, np.float32)], "act": [act],
            "compute": compute}


def test_one_hot_reproduces_gather():
    g = np.random.default_rng(11)
    a = [g.standard_normal((5, 6)).astype(np.float32) for _ in range(2)]
    spec = wl.window2d_spec(5, 6)
    X = oracle.gather(spec, a)
    F = X.shape[1]
    perm = g.permutation(F)
    Y = oracle.infer_rows(spec, a, _one_hot_model(F, perm))
    assert np.array_equal(Y, X[:, perm].astype(np.float32))
    # ReLU on non-negative inputs is the identity too
    ap = [np.abs(x) for x in a]
    Y = oracle.infer_rows(spec, ap, _one_hot_model(F, np.arange(F), act=1))
    assert np.array_equal(Y, oracle.gather(spec, ap).astype(np.float32))
    # bf16: output is the bf16 rounding of the input (torch's conversion)
    Y = oracle.infer_rows(spec, a, _one_hot_model(F, np.arange(F), compute="bf16"))
    assert np.array_equal(Y, torch.from_numpy(X.astype(np.float32)).bfloat16().float().numpy())


def test_one_hot_scatter_is_a_permuted_copy():
    g = np.random.default_rng(12)
    n = 37
    ins = [g.standard_normal(n).astype(np.float32) for _ in range(3)]
    outs = [np.zeros(n, np.float32) for _ in range(3)]
    perm = np.array([2, 0, 1])
    model = _one_hot_model(3, perm)
    oracle.infer(wl.pointwise_spec(n), ins, wl.pointwise_spec(n), outs, model)
    for g_ in range(3):
        assert np.array_equal(outs[g_], ins[perm[g_]])


def test_single_linear_layer_integer_exact():
    g = np.random.default_rng(13)
    X = g.integers(-8, 9, (200, 17)).astype(np.float64)
    W = g.integers(-5, 6, (9, 17)).astype(np.float32)
    b = g.integers(-20, 21, 9).astype(np.float32)
    Y = oracle.mlp({"dims": [17, 9], "W": [W], "b": [b], "act": [0]}, X)
    want = X @ W.astype(np.float64).T + b
    assert np.array_equal(Y.astype(np.float64), want)


def test_single_linear_layer_random_matches_matmul():
    g = np.random.default_rng(14)
    X = g.standard_normal((300, 40)).astype(np.float32).astype(np.float64)
    W = g.standard_normal((30, 40)).astype(np.float32)
    b = g.standard_normal(30).astype(np.float32)
    Y = oracle.mlp({"dims": [40, 30], "W": [W], "b": [b], "act": [0]}, X)
    want = (X @ W.astype(np.float64).T + b.astype(np.float64)).astype(np.float32)
    # identical up to the final fp32 rounding of two fp64 sums in different order
    assert np.max(np.abs(Y - want) / np.maximum(np.abs(want), 1e-30)) <= 2 ** -23


def _torch_stack(model, X):
    layers = []
    for l, (W, b) in enumerate(zip(model["W"], model["b"])):
        lin = torch.nn.Linear(W.shape[1], W.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(W.astype(np.float64)))
            lin.bias.copy_(torch.from_numpy(b.astype(np.float64)))
        layers.append(lin)
        if model["act"][l] == 1:
            layers.append(torch.nn.ReLU())
    with torch.no_grad():
        return torch.nn.Sequential(*layers)(torch.from_numpy(X)).numpy()


@pytest.mark.parametrize("dims", [[5, 64, 64, 1], [9, 128, 128, 128, 1], [36, 128, 128, 4], [3, 7, 2]])
def test_mlp_matches_torch_fp64(dims):
    model = wl.make_model(7, dims, "f32")
    g = np.random.default_rng(15)
    X = g.standard_normal((500, dims[0])).astype(np.float32).astype(np.float64)
    Y = oracle.mlp(model, X)
    want = _torch_stack(model, X)
    err = np.abs(Y.astype(np.float64) - want)
    assert np.all(err <= 2 ** -24 * np.abs(want) + 1e-30 + 1e-13 * np.abs(want).max())


def test_bf16_mlp_matches_torch_bf16_roundings():
    """bf16 model: torch rounds weights, inputs and hidden activations with
    its own bf16 conversion; matmuls in fp64."""
    dims = [6, 32, 32, 1]
    model = wl.make_model(4, dims, "bf16")
    g = np.random.default_rng(16)
    X = (g.standard_normal((400, 6)) * 3).astype(np.float32)
    Y = oracle.mlp(model, X.astype(np.float64))

    def q(t):
        return t.float().bfloat16().double()
    h = q(torch.from_numpy(X))
    for l in range(3):
        W = q(torch.from_numpy(model["W"][l]))
        h = h @ W.T + torch.from_numpy(model["b"][l]).double()
        if l < 2:
            h = q(torch.relu(h))
    want = h.float().numpy()
    # identical except where an fp64 summation-order difference flips a bf16
    # rounding; demand near-total agreement
    close = np.abs(Y - want) <= 1e-6 * np.maximum(np.abs(want), 1e-3)
    assert close.mean() > 0.99


# ---------------------------------------------------------------- conv pins
def test_window2d_mlp_equals_circular_conv2d():
    ny, nx = 12, 17
    w = wl.make("stencil2d", (ny, nx))
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    m = w.model
    x = torch.from_numpy(np.stack(w.inputs)).double()[None]          # [1, 4, ny, nx]
    k1 = torch.from_numpy(m["W"][0].astype(np.float64)).reshape(128, 4, 3, 3)
    h = torch.nn.functional.pad(x, (1, 1, 1, 1), mode="circular")
    h = torch.relu(torch.nn.functional.conv2d(h, k1, torch.from_numpy(m["b"][0]).double()))
    h = torch.relu(torch.nn.functional.conv2d(
        h, torch.from_numpy(m["W"][1].astype(np.float64))[:, :, None, None],
        torch.from_numpy(m["b"][1]).double()))
    h = torch.nn.functional.conv2d(h, torch.from_numpy(m["W"][2].astype(np.float64))[:, :, None, None],
                                   torch.from_numpy(m["b"][2]).double())
    want = h[0].permute(1, 2, 0).reshape(-1, 4).numpy()
    err = np.abs(Y.astype(np.float64) - want)
    assert np.all(err <= 2 ** -24 * np.abs(want) + 1e-12 * np.abs(want).max())


def test_sevenpoint3d_equals_masked_circular_conv3d():
    nz, ny, nx = 6, 7, 9
    spec = wl.sevenpoint3d_spec(nz, ny, nx)
    g = np.random.default_rng(17)
    fields = [g.standard_normal((nz, ny, nx)).astype(np.float32) for _ in range(5)]
    model = wl.make_model(5, [35, 16, 5], "f32")
    Y = oracle.infer_rows(spec, fields, model)
    W1 = torch.from_numpy(model["W"][0].astype(np.float64))
    K = torch.zeros(16, 5, 3, 3, 3, dtype=torch.float64)
    taps = [(0, 1, 1), (2, 1, 1), (1, 0, 1), (1, 2, 1), (1, 1, 0), (1, 1, 1), (1, 1, 2)]
    for c in range(5):
        for t, (a, b_, d) in enumerate(taps):
            K[:, c, a, b_, d] = W1[:, 7 * c + t]
    x = torch.from_numpy(np.stack(fields)).double()[None]
    h = torch.nn.functional.pad(x, (1,) * 6, mode="circular")
    h = torch.relu(torch.nn.functional.conv3d(h, K, torch.from_numpy(model["b"][0]).double()))
    h = torch.nn.functional.conv3d(h, torch.from_numpy(model["W"][1].astype(np.float64))[:, :, None, None, None],
                                   torch.from_numpy(model["b"][1]).double())
    want = h[0].permute(1, 2, 3, 0).reshape(-1, 5).numpy()
    err = np.abs(Y.astype(np.float64) - want)
    assert np.all(err <= 2 ** -24 * np.abs(want) + 1e-12 * np.abs(want).max())


# ---------------------------------------------------------- batch order
def test_batch_order_invariance_pointwise():
    w = wl.make("bonds", 3001)
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model)
    perm = np.random.default_rng(5).permutation(3001)
    Yp = oracle.infer_rows(w.in_spec, [a[perm] for a in w.inputs], w.model)
    assert np.array_equal(Yp, Y[perm])
    # rows given explicitly, in any order
    rows = perm[:500]
    assert np.array_equal(oracle.infer_rows(w.in_spec, w.inputs, w.model, rows), Y[rows])


def test_batch_order_invariance_subsweeps():
    ny, nx = 9, 14
    w = wl.make("stencil2d", (ny, nx))
    Y = oracle.infer_rows(w.in_spec, w.inputs, w.model).reshape(ny, nx, 4)
    for (a, b), (c, d) in [((0, 4), (0, 14)), ((4, 9), (3, 11)), ((8, 9), (13, 14))]:
        spec = dict(w.in_spec, sweep=((a, c), (b, d), (1, 1)))
        Ys = oracle.infer_rows(spec, w.inputs, w.model).reshape(b - a, d - c, 4)
        assert np.array_equal(Ys, Y[a:b, c:d])


# ---------------------------------------------------------------- bf16
def test_bf16_rounding_special_values():
    vals = np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.0e38, 1e-40, -1e-45], np.float32)
    assert np.array_equal(oracle.bf16_bits(vals), torch.from_numpy(vals).bfloat16().view(torch.int16).numpy().view(np.uint16))
    # ties: 1 + 2^-8 is halfway between two bf16 values and rounds to even (1.0)
    t = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8], np.float32)
    assert list(oracle.bf16_bits(t)) == [0x3F80, 0x3F82]


@pytest.mark.slow
def test_bf16_rounding_every_fp32_pattern():
    step = 1 << 24
    for base in range(0, 1 << 32, step):
        u = np.arange(base, base + step, dtype=np.uint64).astype(np.uint32)
        f = u.view(np.float32)
        mine = oracle.bf16_bits(f)
        ref = torch.from_numpy(f).bfloat16().view(torch.int16).numpy().view(np.uint16)
        nan = np.isnan(f)
        assert np.array_equal(mine[~nan], ref[~nan]), hex(base)
        # NaN as a class: the result must be a NaN
        assert np.all((mine[nan] & 0x7F80) == 0x7F80) and np.all((mine[nan] & 0x7F) != 0)

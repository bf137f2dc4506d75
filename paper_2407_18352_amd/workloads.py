"""Seeded synthetic workloads for the surrogate-inference region.

This module only draws numbers and describes shapes: it holds none of the
region's arithmetic (no gather, no model, no scatter).  Tests feed the same
arrays and specs to the HIP library and to the CPU oracle; the benchmark uses
them as its inputs.

Five workloads stand in for the paper's benchmarks (Table I); the paper's own
datasets and trained models are not available, so inputs are synthetic with
the value ranges of those applications and the weights are random:

* ``options``   pointwise option pricing, 65,536 points, 5 -> 64 -> 64 -> 1, fp32
* ``bonds``     pointwise bond pricing, 1,048,576 points, 9 -> 128 x3 -> 1, fp32
* ``stencil2d`` 2048 x 2048 grid, 4 fields, periodic 3x3 window (36 features),
                36 -> 128 -> 128 -> 4, fp32
* ``poses``     pose scoring, 4,194,304 poses, 6 -> 256 x3 -> 1, bf16
* ``stencil3d`` 512^3 grid, 5 fields, periodic 7-point window (35 features),
                35 -> 512 -> 512 -> 5, bf16

Random streams: ``numpy.random.PCG64(SeedSequence(240718352, spawn_key=(cfg, k)))``
with one child stream ``k`` per array or layer.  Map specs are plain data in
the form both sides accept: ``{"rank", "slices": [(lo, count), ...],
"sweep": (start, stop, step), "bnd"}``.
"""
from __future__ import annotations

import math
import os
from dataclasses import dataclass, field

import numpy as np

ROOT_SEED = 240718352
NONE, PERIODIC, CLAMP = 0, 1, 2
RELU, IDENTITY = 1, 0

# quiet-NaN bit pattern pre-filled into output arrays; elements that a
# `from` map does not cover must keep it
SENTINEL_BITS = 0x7FC0DEAD

NAMES = ("options", "bonds", "stencil2d", "poses", "stencil3d")


def rng(cfg: int, k: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=(cfg, k))))


def pointwise_spec(n: int) -> dict:
    return {"rank": 1, "slices": [((0,), (1,))], "sweep": ((0,), (n,), (1,)), "bnd": [NONE]}


def window2d_spec(ny: int, nx: int) -> dict:
    # [i, j, 0:9] = ([i-1:i+2, j-1:j+2])
    return {"rank": 2, "slices": [((-1, -1), (3, 3))],
            "sweep": ((0, 0), (ny, nx), (1, 1)), "bnd": [PERIODIC, PERIODIC]}


def point2d_spec(ny: int, nx: int) -> dict:
    return {"rank": 2, "slices": [((0, 0), (1, 1))],
            "sweep": ((0, 0), (ny, nx), (1, 1)), "bnd": [PERIODIC, PERIODIC]}


def sevenpoint3d_spec(nz: int, ny: int, nx: int) -> dict:
    # 3-D extension of the paper's 2-D 5-point functor (Fig. 2):
    # [i,j,k,0:7] = ([i-1,j,k], [i+1,j,k], [i,j-1,k], [i,j+1,k], [i,j,k-1:k+2])
    return {"rank": 3,
            "slices": [((-1, 0, 0), (1, 1, 1)), ((1, 0, 0), (1, 1, 1)),
                       ((0, -1, 0), (1, 1, 1)), ((0, 1, 0), (1, 1, 1)),
                       ((0, 0, -1), (1, 1, 3))],
            "sweep": ((0, 0, 0), (nz, ny, nx), (1, 1, 1)), "bnd": [PERIODIC] * 3}


def point3d_spec(nz: int, ny: int, nx: int) -> dict:
    return {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))],
            "sweep": ((0, 0, 0), (nz, ny, nx), (1, 1, 1)), "bnd": [PERIODIC] * 3}


@dataclass
class Workload:
    name: str
    cfg: int
    compute: str                 # "f32" | "bf16"
    dims: list
    in_spec: dict
    out_spec: dict
    inputs: list                 # float32 arrays (the application's input fields)
    outputs: list                # float32 arrays, pre-filled with the sentinel
    model: dict = field(default_factory=dict)

    @property
    def n_points(self) -> int:
        n = 1
        for a, b, s in zip(*self.in_spec["sweep"]):
            n *= max(0, -(-(b - a) // s))
        return n

    @property
    def flops_per_point(self) -> int:
        return 2 * sum(self.dims[i] * self.dims[i + 1] for i in range(len(self.dims) - 1))

    @property
    def hbm_bytes_per_point(self) -> int:
        return 4 * (len(self.inputs) + len(self.outputs))


def sentinel_like(shape) -> np.ndarray:
    a = np.empty(shape, np.uint32)
    a.fill(SENTINEL_BITS)
    return a.view(np.float32)


def make_model(cfg: int, dims, compute: str) -> dict:
    """He-normal weights N(0, 2/fan_in); biases U(-1/sqrt(fan_in), 1/sqrt(fan_in));
    ReLU on hidden layers, identity on the output layer."""
    W, b = [], []
    L = len(dims) - 1
    for l in range(L):
        fin, fout = dims[l], dims[l + 1]
        W.append((rng(cfg, 200 + l).standard_normal((fout, fin)) * math.sqrt(2.0 / fin)).astype(np.float32))
        bound = 1.0 / math.sqrt(fin)
        b.append(rng(cfg, 300 + l).uniform(-bound, bound, fout).astype(np.float32))
    act = [RELU] * (L - 1) + [IDENTITY]
    return {"dims": list(dims), "W": W, "b": b, "act": act, "compute": compute}


def _uniform(cfg, k, lo, hi, n):
    return rng(cfg, k).uniform(lo, hi, n).astype(np.float32)


def sinusoid_field(cfg: int, k: int, ny: int, nx: int) -> np.ndarray:
    """Sum of 8 periodic sinusoids (integer wave numbers in -8..8, not both 0,
    so the field is seamless under periodic wrap) plus N(0, 0.01) noise."""
    g = rng(cfg, k)
    i = np.arange(ny, dtype=np.float64)[:, None]
    j = np.arange(nx, dtype=np.float64)[None, :]
    f = np.zeros((ny, nx), np.float64)
    for _ in range(8):
        a = g.uniform(0.5, 1.0)
        while True:
            km, lm = g.integers(-8, 9, size=2)
            if km or lm:
                break
        ph = g.uniform(0.0, 2 * math.pi)
        f += a * np.sin(2 * math.pi * (km * i / ny + lm * j / nx) + ph)
    f += g.normal(0.0, 0.01, (ny, nx))
    return f.astype(np.float32)


def _normal_chunked(cfg: int, k: int, shape, workers: int) -> np.ndarray:
    """N(0,1) float32 array drawn in slabs along axis 0, slab c from child
    stream (cfg, k, c) (threads fill slabs in parallel)."""
    from concurrent.futures import ThreadPoolExecutor
    out = np.empty(shape, np.float32)
    n0 = shape[0]
    slabs = [(c, c * n0 // 16, (c + 1) * n0 // 16) for c in range(16)]

    def fill(job):
        c, a, b = job
        if b > a:
            g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=(cfg, k, c))))
            g.standard_normal(out=out[a:b], dtype=np.float32)
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(fill, slabs))
    return out


def gaussian_field(cfg: int, k: int, shape, corr: float = 4.0) -> np.ndarray:
    """White N(0,1) noise filtered in Fourier space by exp(-|k|^2 corr^2 / 2),
    then standardised to zero mean and unit sample variance."""
    import scipy.fft as sfft
    workers = min(16, os.cpu_count() or 1)
    white = _normal_chunked(cfg, k, shape, workers)
    spec = sfft.rfftn(white, workers=workers)
    del white
    nz, ny, nx = shape
    c2 = corr * corr / 2
    fz = np.exp(-((2 * np.pi * np.fft.fftfreq(nz)) ** 2) * c2).astype(np.float32)[:, None, None]
    fy = np.exp(-((2 * np.pi * np.fft.fftfreq(ny)) ** 2) * c2).astype(np.float32)[None, :, None]
    fx = np.exp(-((2 * np.pi * np.fft.rfftfreq(nx)) ** 2) * c2).astype(np.float32)[None, None, :]
    spec *= fz
    spec *= fy
    spec *= fx
    spec[0, 0, 0] = 0                      # zero mean
    f = sfft.irfftn(spec, s=shape, workers=workers).astype(np.float32, copy=False)
    del spec
    rms = np.sqrt(np.einsum("i,i->", f.reshape(-1), f.reshape(-1), dtype=np.float64) / f.size)
    f *= np.float32(1.0 / rms)
    return f


# full sizes (the five configurations) and small sizes (parity runs: a few tiles
# plus a ragged tail, small enough for the oracle to finish in seconds)
FULL = {"options": 65536, "bonds": 1 << 20, "stencil2d": (2048, 2048),
        "poses": 1 << 22, "stencil3d": (512, 512, 512)}
SMALL = {"options": 65536, "bonds": 50021, "stencil2d": (67, 131),
         "poses": 40013, "stencil3d": (12, 20, 70)}


def make(name: str, size=None) -> Workload:
    """Build a workload.  ``size`` overrides the point count (pointwise) or the
    grid shape (stencils); "full" and "small" select the presets."""
    cfg = NAMES.index(name) + 1
    if size is None or size == "full":
        size = FULL[name]
    elif size == "small":
        size = SMALL[name]
    if name == "options":
        n = int(size)
        ranges = [(10, 200), (10, 200), (0, 0.1), (0.05, 0.6), (0.1, 5)]
        inputs = [_uniform(cfg, k, lo, hi, n) for k, (lo, hi) in enumerate(ranges)]
        dims, compute = [5, 64, 64, 1], "f32"
        ins, outs = pointwise_spec(n), pointwise_spec(n)
        outputs = [sentinel_like((n,))]
    elif name == "bonds":
        n = int(size)
        inputs = [_uniform(cfg, k, 0, 1, n) for k in range(9)]
        dims, compute = [9, 128, 128, 128, 1], "f32"
        ins, outs = pointwise_spec(n), pointwise_spec(n)
        outputs = [sentinel_like((n,))]
    elif name == "stencil2d":
        ny, nx = size
        inputs = [sinusoid_field(cfg, k, ny, nx) for k in range(4)]
        dims, compute = [36, 128, 128, 4], "f32"
        ins, outs = window2d_spec(ny, nx), point2d_spec(ny, nx)
        outputs = [sentinel_like((ny, nx)) for _ in range(4)]
    elif name == "poses":
        n = int(size)
        inputs = [_uniform(cfg, k, -math.pi, math.pi, n) for k in range(3)]
        inputs += [_uniform(cfg, k, -10, 10, n) for k in range(3, 6)]
        dims, compute = [6, 256, 256, 256, 1], "bf16"
        ins, outs = pointwise_spec(n), pointwise_spec(n)
        outputs = [sentinel_like((n,))]
    elif name == "stencil3d":
        shape = tuple(size)
        inputs = [gaussian_field(cfg, k, shape) for k in range(5)]
        dims, compute = [35, 512, 512, 5], "bf16"
        ins, outs = sevenpoint3d_spec(*shape), point3d_spec(*shape)
        outputs = [sentinel_like(shape) for _ in range(5)]
    else:
        raise KeyError(name)
    model = make_model(cfg, dims, compute)
    return Workload(name, cfg, compute, dims, ins, outs, inputs, outputs, model)


def sample_rows(n_points: int, k: int, seed_k: int = 999, must=None) -> np.ndarray:
    """A fixed seeded sample of ``k`` distinct sweep rows, always including
    ``must`` (e.g. every boundary cell), sorted."""
    g = rng(0, seed_k)
    base = np.asarray([] if must is None else must, np.int64)
    extra = g.choice(n_points, size=min(k, n_points), replace=False).astype(np.int64)
    rows = np.unique(np.concatenate([base, extra]))
    return rows


def edge_rows_3d(nz: int, ny: int, nx: int) -> np.ndarray:
    """Row numbers of every cell on the 12 edges of an nz x ny x nx grid."""
    cells = set()
    for a in (0, nz - 1):
        for b in (0, ny - 1):
            for c in range(nx):
                cells.add((a * ny + b) * nx + c)
        for c in (0, nx - 1):
            for b in range(ny):
                cells.add((a * ny + b) * nx + c)
    for b in (0, ny - 1):
        for c in (0, nx - 1):
            for a in range(nz):
                cells.add((a * ny + b) * nx + c)
    return np.asarray(sorted(cells), np.int64)


def edge_rows_2d(ny: int, nx: int) -> np.ndarray:
    cells = set()
    for a in (0, ny - 1):
        for c in range(nx):
            cells.add(a * nx + c)
    for c in (0, nx - 1):
        for a in range(ny):
            cells.add(a * nx + c)
    return np.asarray(sorted(cells), np.int64)


# ---- convolutional surrogates (Table IV model spaces) ----------------------
# * ``weather_cnn``  MiniWeather-like: 4 periodic state fields on an ny x nx
#   grid (sums of sinusoids, as ``stencil2d``); conv 5x5 4 -> 8 (circular,
#   ReLU), conv 3x3 8 -> 4 (circular); kernel sizes and channels from the
#   middle of the searched ranges (layer-1 kernel 2-8, 4-8 channels, layer-2
#   kernel 0-6).  Full size 2048 x 2048, the 2-D stencil's grid.
# * ``particle_cnn`` ParticleFilter-like: S video frames of H x W pixels (a
#   bright disc moving across a noisy background), conv 4x4 step 4 1 -> 8
#   (valid, ReLU), max-pool 2x2, fully connected 2048 -> 64 (ReLU) -> 2 (the
#   object's location).  Full size 1024 frames of 128 x 128.
CNN_NAMES = ("weather_cnn", "particle_cnn")
CNN_FULL = {"weather_cnn": (2048, 2048), "particle_cnn": (1024, 128, 128)}
CNN_SMALL = {"weather_cnn": (37, 150), "particle_cnn": (3, 128, 128)}


def conv_layer(cfg, k, cin, cout, kernel, padding="same", mode="circular", stride=(1, 1), act=RELU) -> dict:
    """He-normal weights N(0, 2/fan_in), biases U(-1/sqrt(fan_in), 1/sqrt(fan_in))."""
    fan = cin * kernel[0] * kernel[1]
    W = (rng(cfg, k).standard_normal((cout, cin) + tuple(kernel)) * math.sqrt(2.0 / fan)).astype(np.float32)
    b = rng(cfg, k + 1).uniform(-1 / math.sqrt(fan), 1 / math.sqrt(fan), cout).astype(np.float32)
    return {"kind": "conv", "out": cout, "kernel": tuple(kernel), "stride": tuple(stride), "padding": padding,
            "mode": mode, "act": act, "W": W, "b": b}


def linear_layer(cfg, k, fin, fout, act=RELU) -> dict:
    W = (rng(cfg, k).standard_normal((fout, fin)) * math.sqrt(2.0 / fin)).astype(np.float32)
    b = rng(cfg, k + 1).uniform(-1 / math.sqrt(fin), 1 / math.sqrt(fin), fout).astype(np.float32)
    return {"kind": "linear", "out": fout, "act": act, "W": W, "b": b}


def video_frames(cfg: int, k: int, S: int, H: int, W: int) -> np.ndarray:
    """S frames: background 0.4 + N(0, 0.05) noise and a disc of radius H/16
    and value 0.9 moving on a straight line across the frame."""
    g = rng(cfg, k)
    f = (0.4 + g.normal(0.0, 0.05, (S, H, W))).astype(np.float32)
    y0, x0 = g.uniform(0.2, 0.8, 2) * (H, W)
    vy, vx = g.uniform(-1.0, 1.0, 2)
    r = H / 16
    yy = np.arange(H)[:, None]
    xx = np.arange(W)[None, :]
    for s in range(S):
        cy, cx = (y0 + vy * s) % H, (x0 + vx * s) % W
        f[s][(yy - cy) ** 2 + (xx - cx) ** 2 <= r * r] = 0.9
    return f


def cnn_model(name: str, size=None) -> dict:
    """The model of a convolutional workload alone (no input arrays)."""
    cfg = 10 + CNN_NAMES.index(name)
    size = CNN_FULL[name] if size in (None, "full") else CNN_SMALL[name] if size == "small" else size
    if name == "weather_cnn":
        ny, nx = size
        layers = [conv_layer(cfg, 100, 4, 8, (5, 5)), conv_layer(cfg, 110, 8, 4, (3, 3), act=IDENTITY)]
        return {"kind": "cnn", "in_channels": 4, "image": (ny, nx), "layers": layers, "compute": "f32"}
    S, H, W = size
    c1 = conv_layer(cfg, 100, 1, 8, (4, 4), padding="valid", mode="zeros", stride=(4, 4))
    h, w = (H - 4) // 4 + 1, (W - 4) // 4 + 1
    h, w = (h - 2) // 2 + 1, (w - 2) // 2 + 1
    layers = [c1, {"kind": "pool", "kernel": (2, 2), "act": IDENTITY},
              linear_layer(cfg, 110, h * w * 8, 64), linear_layer(cfg, 120, 64, 2, act=IDENTITY)]
    return {"kind": "cnn", "in_channels": 1, "image": (H, W), "layers": layers, "compute": "f32"}


def make_cnn(name: str, size=None) -> Workload:
    """A convolutional workload; ``model`` is ``{"kind": "cnn", "in_channels",
    "image": (rows, columns), "layers": [...]}`` (the layer dicts of
    ``conv_layer`` / ``linear_layer`` and ``{"kind": "pool", "kernel"}``)."""
    cfg = 10 + CNN_NAMES.index(name)
    if size is None or size == "full":
        size = CNN_FULL[name]
    elif size == "small":
        size = CNN_SMALL[name]
    model = cnn_model(name, size)
    if name == "weather_cnn":
        ny, nx = size
        inputs = [sinusoid_field(cfg, k, ny, nx) for k in range(4)]
        ins, outs = point2d_spec(ny, nx), point2d_spec(ny, nx)
        outputs = [sentinel_like((ny, nx)) for _ in range(4)]
        dims = [4, 4]
    elif name == "particle_cnn":
        S, H, W = size
        inputs = [video_frames(cfg, 0, S, H, W)]
        ins = {"rank": 3, "slices": [((0, 0, 0), (1, 1, 1))], "sweep": ((0, 0, 0), (S, H, W), (1, 1, 1)),
               "bnd": [NONE] * 3}
        outs = pointwise_spec(S)
        outputs = [sentinel_like((S,)) for _ in range(2)]
        dims = [1, 2]
    else:
        raise KeyError(name)
    return Workload(name, cfg, "f32", dims, ins, outs, inputs, outputs, model)


def cnn_flops_per_image(model) -> int:
    """Multiply-adds x 2 of one image through the stack (max-pool: none)."""
    H, W = model["image"]
    h, w, c = H, W, model["in_channels"]
    total = 0
    for ly in model["layers"]:
        if ly["kind"] == "conv":
            kh, kw = ly["kernel"]
            if ly.get("padding", "valid") == "valid":
                sh, sw = ly.get("stride", (1, 1))
                h, w = (h - kh) // sh + 1, (w - kw) // sw + 1
            total += 2 * h * w * ly["out"] * c * kh * kw
            c = ly["out"]
        elif ly["kind"] == "pool":
            kh, kw = ly["kernel"]
            sh, sw = ly.get("stride", ly["kernel"])
            h, w = (h - kh) // sh + 1, (w - kw) // sw + 1
        else:
            total += 2 * h * w * c * ly["out"]
            h, w, c = 1, 1, ly["out"]
    return total

#!/usr/bin/env python3
"""Benchmark of the surrogate-inference region on one MI355X.

One step = one pass of the whole hot path over the workload: the fused
gather -> MLP -> scatter (``hpacml_infer``) plus the collect records of the
region's inputs and outputs (``hpacml_collect_pair`` into a [B x F_in] input
record and a [B x F_out] output record, the two datasets a collected region
stores).  Inputs are synthetic, seeded and resident in HBM before the timed
region.  Prints one JSON line.

Default (no --workload): the headline is the 3-D stencil surrogate, a
512^3 grid x 5 fp32 fields, periodic 7-point window (35 features), MLP
35 -> 512 -> 512 -> 5 ReLU in bf16 with fp32 accumulation, the largest of the
five workloads and the one whose fused kernel is bound by the bf16 matrix
cores.  The other four workloads (option pricing, bond pricing, the 2-D
stencil, pose scoring) are measured in the same run and reported under
``configs``.

When one step's working set (fields, outputs, records) is smaller than the
256 MB Infinity Cache, consecutive steps rotate over identical copies of the
batch (>= 1 GiB together) so that every step reads its data from HBM.

``roofline.traffic`` is the HBM traffic per launch of the dominant kernel
from the committed rocprofv3 counter summary in ``profiles/``, used only while
the kernel's source hash still matches the one recorded there (else null).
"""
import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"f32": 157.3e12, "bf16": 2.5e15}   # dense MFMA peaks of MI355X, flop/s
VALU_F32_PEAK = 157.3e12                   # published fp32 vector peak (packed FMA; see the design notes)
HBM_PEAK = 8.0e12                          # bytes/s
IC_BYTES = 256 << 20                       # Infinity Cache
HEADLINE = "stencil3d"
OTHERS = ("options", "bonds", "stencil2d", "poses")

DESCRIPTION = {
    "options": "option pricing: 65,536 points, 5 SoA fp32 inputs, MLP 5-64-64-1 ReLU fp32, 1 output",
    "bonds": "bond pricing: 1,048,576 points, 9 SoA fp32 inputs U[0,1], MLP 9-128-128-128-1 ReLU fp32, "
             "1 output; collect records 9+1 values per point",
    "stencil2d": "2-D stencil: 2048x2048 grid x 4 fp32 fields, periodic 3x3 window (36 features), "
                 "MLP 36-128-128-4 ReLU fp32, 4 outputs per cell",
    "poses": "pose scoring: 4,194,304 poses, 6 fp32 inputs, MLP 6-256-256-256-1 ReLU, bf16 weights and "
             "activations with fp32 accumulate, 1 output",
    "stencil3d": "3-D stencil: 512^3 grid x 5 fp32 fields, periodic 7-point window (35 features), "
                 "MLP 35-512-512-5 ReLU, bf16 with fp32 accumulate, 5 outputs per cell",
    "weather_cnn": "convolutional 2-D step: 2048x2048 grid x 4 fp32 fields, conv 5x5 4->8 circular ReLU, "
                   "conv 3x3 8->4 circular, fp32, 4 outputs per cell",
    "particle_cnn": "convolutional frame estimate: 1024 frames of 128x128 fp32 pixels, conv 4x4/4 1->8 ReLU, "
                    "max-pool 2x2, FC 2048->64 ReLU, FC 64->2, fp32, 2 outputs per frame",
}


KERNEL_SOURCES = {
    "collect": ["collect.hip", "device.hpp", "kernels.hpp"],
    "mlp_f32": ["mlp_f32.hip", "device.hpp", "kernels.hpp"],
    "mlp_bf16r": ["mlp_bf16r.hip", "mlp_bf16r.hpp", "mlp_bf16r_h256_nh1.hip", "mlp_bf16r_h256_nh2.hip",
                  "mlp_bf16r_h256_nh3.hip", "device.hpp", "kernels.hpp"],
    "mlp_bf16": ["mlp_bf16.hip", "device.hpp", "kernels.hpp"],
    "mlp_generic": ["mlp_generic.hip", "device.hpp", "kernels.hpp"],
    "mlp_layers": ["mlp_layers.hip", "layers.hpp", "device.hpp"],
    "cnn_": ["cnn.hip", "cnn.hpp", "device.hpp", "kernels.hpp"],
}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def source_sha(variant):
    """Hash of the sources of the kernel family `variant` belongs to (the key
    under which profiles/*.txt record its counters), or None."""
    fam = next((k for k in KERNEL_SOURCES if variant.startswith(k)), None)
    if fam is None:
        return None
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[fam]:
        path = os.path.join(ROOT, "paper_2407_18352_amd", "csrc", f)
        if not os.path.exists(path):
            return None
        h.update(open(path, "rb").read())
    return h.hexdigest()[:16]


def recorded_traffic(variant, workload):
    """HBM bytes per launch of `variant` on `workload` from profiles/*.txt,
    if the kernel source is unchanged since the counters were taken."""
    sha = source_sha(variant)
    if sha is None:
        return None
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.txt"))):
        for line in open(path):
            if line.startswith("traffic_line "):
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                if kv.get("kernel") == variant and kv.get("workload") == workload and kv.get("source_sha256") == sha:
                    return {"bytes": int(kv["bytes"]), "fetch": int(kv["fetch"]), "write": int(kv["write"]),
                            "source": os.path.relpath(path, ROOT)}
    return None


def cnn_hbm_bound(w, wl) -> bool:
    """A convolutional workload is bound by HBM when moving its arrays once at
    the HBM peak takes longer than its flops at the fp32 vector peak."""
    H, W = w.model["image"]
    n_img = w.n_points // (H * W)
    fields_b = sum(a.nbytes for a in w.inputs) + sum(a.nbytes for a in w.outputs)
    return fields_b / HBM_PEAK > wl.cnn_flops_per_image(w.model) * n_img / VALU_F32_PEAK


def host_cpu():
    """(logical CPUs usable by this process, CPU model name)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return n, model


def scaled_errors(got, want):
    """Worst |g - o| / max(|o|, s) with s the oracle column's RMS, the
    normwise relative error, and the NaN count."""
    import numpy as np
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    s = np.sqrt(np.mean(want * want, axis=0, keepdims=True))
    s = np.where(s > 0, s, 1.0)
    worst = float(np.nanmax(np.abs(got - want) / np.maximum(np.abs(want), s))) if want.size else 0.0
    norm = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))
    return worst, norm, int(np.isnan(got).sum())


class Run:
    """One workload resident on the GPU, with its maps, model, records and
    the timing of `steps` steps after `warmup` untimed ones."""

    def __init__(self, name, args, rotate_small=True):
        import numpy as np
        import torch

        from paper_2407_18352_amd import _abi, api
        from paper_2407_18352_amd import workloads as wl

        self.name = name
        self.is_cnn = name in wl.CNN_NAMES
        t0 = time.time()
        w = wl.make_cnn(name) if self.is_cnn else wl.make(name)
        if getattr(args, "dims", None) and not self.is_cnn:
            # another model of the workload's model space (same inputs and outputs)
            dims = [int(x) for x in args.dims.split(",")]
            if dims[0] != w.dims[0] or dims[-1] != w.dims[-1] or len(dims) < 2:
                print("--dims must keep %d inputs and %d outputs" % (w.dims[0], w.dims[-1]), file=sys.stderr)
                sys.exit(2)
            w.dims = dims
            w.model = wl.make_model(w.cfg, dims, w.compute)
        self.w = w
        log("workload %s generated in %.1fs" % (name, time.time() - t0))

        fields_b = sum(a.nbytes for a in w.inputs) + sum(a.nbytes for a in w.outputs)
        self.alg_bytes = fields_b
        # the dominant kernel's roof: a convolutional stack whose flops take
        # less time at the fp32 vector peak than its arrays take at the HBM
        # peak is bound by HBM
        self.hbm_bound = self.is_cnn and cnn_hbm_bound(w, wl)
        self.model = api.CnnModel(w.model) if self.is_cnn else api.Model(w.model)
        sets = []
        per_set = fields_b
        for k in range(400):
            ins = [torch.from_numpy(a).cuda() for a in w.inputs]
            outs = [torch.from_numpy(a).cuda() for a in w.outputs]
            if args.inplace:
                if len(w.outputs) > len(ins) or any(o.shape != i.shape for o, i in zip(outs, ins)):
                    print("--inplace needs outputs shaped like the first inputs", file=sys.stderr)
                    sys.exit(2)
                outs = ins[:len(w.outputs)]
            mi = api.Map(w.in_spec, ins, _abi.TO)
            mo = api.Map(w.out_spec, outs, _abi.FROM)
            mo_rec = api.Map(w.out_spec, outs, _abi.TO)        # the outputs as a recorded map
            rec_in = torch.empty((mi.n_points, mi.n_features), device="cuda")
            rec_out = torch.empty((mo.n_points, mo.n_features), device="cuda")
            sets.append((ins, outs, mi, mo, mo_rec, rec_in, rec_out))
            per_set = fields_b + 4 * (mi.n_points * mi.n_features + mo.n_points * mo.n_features)
            if k == 0:
                # a step's working set under the Infinity Cache (or an
                # HBM-bound kernel): rotate over copies
                rotate = (rotate_small and per_set < IC_BYTES) or self.hbm_bound or args.rotate
            if not rotate or (k + 1) * per_set >= (1 << 30):
                break
        self.sets = sets
        self.per_set = per_set
        ins, outs, mi, mo, mo_rec, rec_in, rec_out = sets[0]
        self.ins, self.outs, self.mi, self.mo, self.rec_in = ins, outs, mi, mo, rec_in
        self.variant = api.variant(self.model, mi, mo)
        self.B, self.Fi, self.Fo, self.Bo = mi.n_points, mi.n_features, mo.n_features, mo.n_points
        self.stream = torch.cuda.current_stream()
        self.turn = 0
        self.api = api

    def step(self, ev=None):
        _, _, mi_k, mo_k, mo_rec_k, rec_in_k, rec_out_k = self.sets[self.turn % len(self.sets)]
        self.turn += 1
        api, stream = self.api, self.stream
        if ev is not None:
            ev[0].record(stream)
        api.infer(self.model, mi_k, mo_k, stream)
        if ev is not None:
            ev[1].record(stream)
        api.collect_pair(mi_k, rec_in_k, self.Fi, mo_rec_k, rec_out_k, self.Fo, stream)
        if ev is not None:
            ev[2].record(stream)

    def time_steps(self, steps, warmup):
        import numpy as np
        import torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(steps)]
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        start.record(self.stream)
        for k in range(steps):
            self.step(evs[k])
        stop.record(self.stream)
        torch.cuda.synchronize()
        self.wall = time.perf_counter() - wall0
        self.total_ms = start.elapsed_time(stop)
        self.ms_step = self.total_ms / steps
        self.infer_ms = [e[0].elapsed_time(e[1]) for e in evs]
        self.collect_ms = [e[1].elapsed_time(e[2]) for e in evs]
        self.infer_avg = float(np.mean(self.infer_ms))
        self.collect_avg = float(np.mean(self.collect_ms))
        # after the timed steps the last set holds this run's outputs; point
        # the parity check at them
        last = self.sets[(self.turn - 1) % len(self.sets)]
        self.outs = last[1]

    def rooflines(self):
        from paper_2407_18352_amd import workloads as wl
        w, B = self.w, self.B
        if self.is_cnn:
            H, W = w.model["image"]
            flop_launch = wl.cnn_flops_per_image(w.model) * (B // (H * W))
            peak, bound = VALU_F32_PEAK, "alu"
        else:
            flop_launch = w.flops_per_point * B
            peak, bound = PEAK[w.compute], "mfma"
        achieved = flop_launch / (self.infer_avg * 1e-3)
        if self.hbm_bound:
            peak, bound = HBM_PEAK, "hbm"
            achieved = self.alg_bytes / (self.infer_avg * 1e-3)
        self.flop_launch, self.peak = flop_launch, peak
        traffic = recorded_traffic(self.variant, self.name)
        # collect: every element of the mapped arrays read once, every record
        # word written once (in and out records)
        collect_bytes = (sum(a.nbytes for a in w.inputs) + 4 * B * self.Fi) + \
                        (sum(a.nbytes for a in w.outputs) + 4 * self.Bo * self.Fo)
        collect_traffic = recorded_traffic("collect", self.name)
        hb = self.hbm_bound
        roof = {"bound": bound, "achieved": achieved / (1e9 if hb else 1e12),
                "peak": peak / (1e9 if hb else 1e12), "unit": "GB/s" if hb else "TFLOP/s",
                "frac": achieved / peak, "traffic": traffic["bytes"] if traffic else None,
                "traffic_source": traffic["source"] if traffic else None,
                "algorithmic_hbm_bytes_per_launch": self.alg_bytes,
                "kernel": self.variant, "kernel_avg_ms": self.infer_avg,
                "algorithmic_flop_per_launch": flop_launch}
        croof = {"bound": "hbm", "achieved": collect_bytes / (self.collect_avg * 1e-3) / 1e9,
                 "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                 "frac": collect_bytes / (self.collect_avg * 1e-3) / HBM_PEAK,
                 "traffic": collect_traffic["bytes"] if collect_traffic else None,
                 "traffic_source": collect_traffic["source"] if collect_traffic else None,
                 "algorithmic_bytes_per_step": collect_bytes, "ms_per_step": self.collect_avg,
                 "kernels": "hpacml_collect_pair: the input map's and the output map's records"}
        return roof, croof

    def copies_note(self):
        n = len(self.sets)
        return {"count": n, "bytes_each": self.per_set,
                "note": "steps rotate over identical copies so that data comes from HBM, not the "
                        "256 MB Infinity Cache" if n > 1 else "every step on the same arrays (working set "
                        "larger than the Infinity Cache)" if self.per_set >= IC_BYTES else
                        "every step on the same arrays"}

    def parity(self, rows, threads=None):
        """Oracle outputs on `rows` (timed), compared with the GPU's outputs.
        Returns (worst scaled error, normwise, NaN count, oracle seconds)."""
        import numpy as np

        import oracle
        if threads:
            oracle.set_num_threads(threads)
        c0 = time.perf_counter()
        Y = oracle.infer_rows(self.w.in_spec, self.w.inputs, self.w.model, rows)
        sec = time.perf_counter() - c0
        got = np.stack([o.cpu().numpy().reshape(-1)[rows] for o in self.outs], 1)
        return scaled_errors(got, Y) + (sec,)

    def close(self):
        import torch
        for (_, _, mi, mo, mo_rec, _, _) in self.sets:
            mi.close(), mo.close(), mo_rec.close()
        self.model.close()
        self.sets = None
        self.ins = self.outs = self.rec_in = None
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def headline_cpu_baseline(run, args, result):
    """The oracle on the host cores: a seeded sample of the workload's rows
    (every grid-edge cell of a 3-D grid included), which also serves as the
    parity sample; then a 1-thread run on a part of it."""
    import numpy as np

    import oracle
    from paper_2407_18352_amd import workloads as wl
    w, B = run.w, run.B
    nproc, model_name = host_cpu()
    threads = oracle.num_threads()
    must = None
    if run.name == "stencil3d":
        must = wl.edge_rows_3d(*w.inputs[0].shape)
    elif run.name == "stencil2d":
        must = wl.edge_rows_2d(*w.inputs[0].shape)
    n_sample = min(B, args.parity_rows)
    rows = wl.sample_rows(B, n_sample, seed_k=998, must=must)
    worst, norm, nan, sec = run.parity(rows, threads)
    reps, cpu_s = 1, sec
    while cpu_s < args.cpu_seconds:
        c0 = time.perf_counter()
        oracle.infer_rows(w.in_spec, w.inputs, w.model, rows)
        cpu_s += time.perf_counter() - c0
        reps += 1
    # one thread: a prefix of the same sample, sized to ~1/3 of the target
    n1 = max(256, min(len(rows), int(len(rows) / max(sec * threads, 1e-9) * args.cpu_seconds / 3)))
    oracle.set_num_threads(1)
    c0 = time.perf_counter()
    oracle.infer_rows(w.in_spec, w.inputs, w.model, rows[:n1])
    s1 = time.perf_counter() - c0
    oracle.set_num_threads(threads)
    result["cpu_baseline"] = {
        "value": reps * len(rows) / cpu_s, "unit": "points/s", "cores": threads, "kind": "oracle",
        "sample": "%d of %d sweep rows (seeded%s) x %d passes, gather + MLP in fp64, %.1fs on %d threads"
                  % (len(rows), B, ", every grid-edge cell included" if must is not None else "", reps, cpu_s,
                     threads),
        "nproc": nproc, "cpu_model": model_name,
        "one_thread": {"value": n1 / s1, "unit": "points/s", "rows": int(n1), "seconds": s1}}
    result["parity_on_cpu_sample"] = {
        "rows": int(len(rows)), "edge_rows": int(0 if must is None else len(must)),
        "worst_scaled_error": worst, "normwise": norm, "nan": nan,
        "rtol": 1e-5 if w.compute == "f32" else 2e-2,
        "rule": "|g - o| <= rtol * max(|o|, s), s = RMS of the oracle's output column"}


def cnn_cpu_baseline(run, args, result):
    import numpy as np

    import oracle
    w, B = run.w, run.B
    H, W = w.model["image"]
    S = B // (H * W)
    c0 = time.perf_counter()
    X1 = oracle.gather(dict(w.in_spec, sweep=_first_images(w.in_spec, 1)), w.inputs)
    oracle.cnn(w.model, X1)
    per_img = time.perf_counter() - c0
    n_img = int(min(S, max(1, args.cpu_seconds / max(per_img, 1e-9))))
    X = oracle.gather(dict(w.in_spec, sweep=_first_images(w.in_spec, n_img)), w.inputs)
    reps, cpu_s = 0, 0.0
    while reps == 0 or cpu_s < args.cpu_seconds:
        c0 = time.perf_counter()
        Y = oracle.cnn(w.model, X)
        cpu_s += time.perf_counter() - c0
        reps += 1
    n_out = Y.shape[0]
    got = np.stack([o.cpu().numpy().reshape(-1)[:n_out] for o in run.outs], 1)
    worst, norm, nan = scaled_errors(got, Y)
    nproc, model_name = host_cpu()
    result["cpu_baseline"] = {"value": reps * n_img * H * W / cpu_s, "unit": "points/s",
                              "cores": oracle.num_threads(), "kind": "oracle",
                              "sample": "the first %d of %d images x %d passes, gather + convolutional model "
                                        "in fp64, %.1fs" % (n_img, S, reps, cpu_s),
                              "nproc": nproc, "cpu_model": model_name}
    result["parity_on_cpu_sample"] = {"worst_scaled_error": worst, "normwise": norm, "nan": nan, "rtol": 1e-5}


def other_config(name, args):
    """One of the other workloads: timed steps, rooflines and a parity check
    against the oracle (every row of the smaller workloads, a seeded sample of
    2^18 rows of pose scoring)."""
    from paper_2407_18352_amd import workloads as wl
    run = Run(name, args)
    run.time_steps(args.steps, args.warmup)
    roof, croof = run.rooflines()
    if run.B <= (1 << 22) and run.w.compute == "f32":
        rows = None
        import numpy as np
        rows = np.arange(run.B, dtype=np.int64)
    else:
        rows = wl.sample_rows(run.B, 1 << 18, seed_k=998)
    worst, norm, nan, sec = run.parity(rows)
    out = {"workload": DESCRIPTION[name], "dtype": run.w.compute, "points": run.B,
           "ms_per_step": run.ms_step, "points_per_s": run.B / (run.ms_step * 1e-3),
           "infer_ms": run.infer_avg, "kernel": run.variant,
           "roofline": {k: roof[k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic")},
           "collect": {"ms": run.collect_avg, "achieved_gbs": croof["achieved"], "frac": croof["frac"]},
           "batch_copies": run.copies_note(),
           "parity": {"rows": int(len(rows)), "worst_scaled_error": worst, "normwise": norm, "nan": nan,
                      "rtol": 1e-5 if run.w.compute == "f32" else 2e-2},
           "oracle_points_per_s": len(rows) / sec}
    if name == "options":
        out["note"] = ("a 65,536-point region is one short launch: the fused kernel and the 2.8 MB of records "
                       "are bound by launch and latency, not by the matrix cores or HBM")
    run.close()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None, choices=sorted(DESCRIPTION),
                    help="measure this workload alone (default: the 3-D stencil, with the other four MLP "
                         "workloads under configs)")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workloads")
    ap.add_argument("--dims", default=None,
                    help="layer widths of another model for the workload, e.g. 6,1024,512,256,1 (inputs and "
                         "outputs as the workload's; seeded He-normal weights)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-rotate", action="store_true",
                    help="keep every step on the same arrays even when they fit the Infinity Cache")
    ap.add_argument("--rotate", action="store_true",
                    help="rotate steps over copies of the batch whatever the working set")
    ap.add_argument("--graph-calls", type=int, default=0,
                    help="also time N inference calls captured in one HIP graph and replayed (no per-call "
                         "launch gaps), reported under graph_replay")
    ap.add_argument("--inplace", action="store_true",
                    help="write the outputs back into the input fields (a time step advanced in place: windowed "
                         "maps then run the snapshot pass); no oracle leg, the fields change every step")
    ap.add_argument("--phases", action="store_true",
                    help="also time the model on the composed input tensor stored as dense column arrays (a "
                         "gather with nothing to compose): the fused kernel's time minus that is the cost of "
                         "mapping (reported under phases; MLP workloads)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU work for the oracle sample")
    ap.add_argument("--parity-rows", type=int, default=1 << 20,
                    help="seeded rows in the oracle sample (grid-edge cells are added to it)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="before warm-up, run one device-to-device copy of this many MiB (a kernel of "
                         "known traffic, to scale HBM counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(see the sharding notes in the design document)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2407_18352_amd import api

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    name = args.workload or HEADLINE
    with_configs = args.workload is None and not args.no_configs and not args.dims
    if args.inplace:
        args.no_cpu_baseline = True

    run = Run(name, args, rotate_small=not args.no_rotate)

    if args.copy_calibration_mb:
        src = torch.empty(args.copy_calibration_mb << 18, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    run.time_steps(args.steps, args.warmup)
    log("%s: %.3f ms per step (infer %.3f ms)" % (name, run.ms_step, run.infer_avg))
    roof, croof = run.rooflines()
    B, Fi, Fo, Bo = run.B, run.Fi, run.Fo, run.Bo
    stream = run.stream
    result = {
        "metric": "surrogate points/sec (gather+MLP+scatter) and % of HBM / MFMA roofline",
        "value": B / (run.ms_step * 1e-3),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": run.ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": run.w.compute,
        "data": "synthetic (seeded generators; random-init He-normal weights)",
        "config": {"workload": DESCRIPTION[name] + ("; outputs written in place into the input fields"
                                                     if args.inplace else "")
                   + ("; model %s instead" % "-".join(str(d) for d in run.w.dims) if args.dims else ""),
                   "points": B, "features_in": Fi, "features_out": Fo, "output_points": Bo},
        "roofline": roof,
        "infer_points_per_s": B / (run.infer_avg * 1e-3),
        "infer_ms": {"mean": run.infer_avg, "median": float(np.median(run.infer_ms)),
                     "min": float(np.min(run.infer_ms))},
        "collect_roofline": croof,
        "wall_s_timed": run.wall,
        "batch_copies": run.copies_note(),
    }
    model, mi, mo = run.model, run.mi, run.mo
    hbm_bound, alg_bytes, flop_launch, peak = run.hbm_bound, run.alg_bytes, run.flop_launch, run.peak

    if args.graph_calls > 0:
        # N back-to-back hpacml_infer calls captured once on a side stream and
        # replayed: the kernel's throughput without host launch gaps
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            api.infer(model, mi, mo, side)          # outside capture: any lazy set-up happens here
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=side):
                for _ in range(args.graph_calls):
                    api.infer(model, mi, mo, side)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        per_call = e0.elapsed_time(e1) / args.graph_calls
        result["graph_replay"] = {"calls": args.graph_calls, "ms_per_call": per_call,
                                  "points_per_s": B / (per_call * 1e-3),
                                  "achieved_tflops": flop_launch / (per_call * 1e-3) / 1e12,
                                  "frac": (alg_bytes if hbm_bound else flop_launch) / (per_call * 1e-3) / peak}
        if hbm_bound:
            result["graph_replay"]["achieved_gbs"] = alg_bytes / (per_call * 1e-3) / 1e9

    if args.phases and not run.is_cnn:
        # mapping vs inference: the composed tensor (the input record) as F
        # contiguous column arrays under a pointwise map, outputs to Fo fresh
        # arrays, through the same fused kernel family
        from paper_2407_18352_amd import _abi
        rec_in = run.rec_in
        api.collect(mi, rec_in, Fi, stream)
        torch.cuda.synchronize()
        cols = [rec_in[:, f].contiguous() for f in range(Fi)]
        dense_out = [torch.empty(B, device="cuda") for _ in range(Fo)]
        pw = {"rank": 1, "slices": [((0,), (1,))], "sweep": ((0,), (B,), (1,)), "bnd": [0]}
        mci = api.Map(pw, cols, _abi.TO)
        mco = api.Map(pw, dense_out, _abi.FROM)
        reps = max(3, min(args.steps, 20))

        def timed(fn):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps

        # the three in turn over 5 rounds (medians), so that clock changes
        # during the run fall on all of them
        runs = {"dense": [], "fused": [], "gather": []}
        for rnd in range(6):
            d = timed(lambda: api.infer(model, mci, mco, stream))
            f = timed(lambda: api.infer(model, mi, mo, stream))
            c = timed(lambda: api.collect(mi, rec_in, Fi, stream))
            if rnd:
                runs["dense"].append(d)
                runs["fused"].append(f)
                runs["gather"].append(c)
        dense_ms, fused_ms, gather_ms = (float(np.median(runs[k])) for k in ("dense", "fused", "gather"))
        result["phases"] = {
            "fused_ms": fused_ms, "dense_columns_ms": dense_ms, "dense_columns_kernel": api.variant(model, mci, mco),
            "mapping_ms": fused_ms - dense_ms, "mapping_frac": (fused_ms - dense_ms) / fused_ms,
            "gather_alone_ms": gather_ms,
            "note": "back-to-back launches, medians of 5 interleaved rounds; mapping_ms = the fused region's "
                    "time minus the same model on the composed tensor stored as dense columns; "
                    "gather_alone_ms = the input map's collect"}
        del cols, dense_out
        mci.close()
        mco.close()

    if not args.no_cpu_baseline:
        if run.is_cnn:
            cnn_cpu_baseline(run, args, result)
        else:
            headline_cpu_baseline(run, args, result)
        log("oracle leg done")
    run.close()
    del run

    if with_configs:
        result["configs"] = {}
        for other in OTHERS:
            result["configs"][other] = other_config(other, args)
            c = result["configs"][other]
            log("%s: %.4f ms per step, %s frac %.3f, collect frac %.3f, parity %.2e"
                % (other, c["ms_per_step"], c["kernel"], c["roofline"]["frac"], c["collect"]["frac"],
                   c["parity"]["worst_scaled_error"]))

    print(json.dumps(result), flush=True)


def _first_images(spec, n):
    """The sweep of `spec` cut to its first n images (leading sweep dimension;
    a rank-2 sweep is one image)."""
    start, stop, step = (list(v) for v in spec["sweep"])
    if spec["rank"] > 2:
        stop[0] = min(stop[0], start[0] + n * step[0])
    return tuple(start), tuple(stop), tuple(step)


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the surrogate-inference region on one MI355X.

One step = one pass of the whole hot path over the workload: the fused
gather -> MLP -> scatter (``hpacml_infer``) plus the collect records of the
region's inputs and outputs (``hpacml_collect_pair`` into a [B x F_in] input
record and a [B x F_out] output record, the two datasets a collected region
stores).  Inputs are synthetic, seeded and resident in HBM before the timed
region.  Prints one JSON line.

``roofline.traffic`` is the HBM traffic per launch of the dominant kernel
from the committed rocprofv3 counter summary in ``profiles/``, used only while
the kernel's source hash still matches the one recorded there (else null).

Default workload: bond-pricing surrogate, 1,048,576 points, 9 SoA fp32 inputs,
MLP 9 -> 128 -> 128 -> 128 -> 1 (ReLU), fp32.
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
    "mlp_bf16": ["mlp_bf16.hip", "device.hpp", "kernels.hpp"],
    "mlp_generic": ["mlp_generic.hip", "device.hpp", "kernels.hpp"],
    "cnn_": ["cnn.hip", "cnn.hpp", "device.hpp", "kernels.hpp"],
}


def recorded_traffic(variant, workload):
    """HBM bytes per launch of `variant` on `workload` from profiles/*.txt,
    if the kernel source is unchanged since the counters were taken."""
    fam = next((k for k in KERNEL_SOURCES if variant.startswith(k)), None)
    if fam is None:
        return None
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[fam]:
        path = os.path.join(ROOT, "paper_2407_18352_amd", "csrc", f)
        if not os.path.exists(path):
            return None
        h.update(open(path, "rb").read())
    sha = h.hexdigest()[:16]
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="bonds", choices=sorted(DESCRIPTION))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--rotate", action="store_true",
                    help="rotate steps over copies of the batch so that small working sets come from HBM, "
                         "not the Infinity Cache")
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

    from paper_2407_18352_amd import _abi, api
    from paper_2407_18352_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    t0 = time.time()
    is_cnn = args.workload in wl.CNN_NAMES
    w = wl.make_cnn(args.workload) if is_cnn else wl.make(args.workload)
    print("[bench] workload %s generated in %.1fs" % (args.workload, time.time() - t0), file=sys.stderr, flush=True)

    # By default every step runs on the same arrays, as a region invoked from
    # an application's time loop does.  With --rotate, when one step's working
    # set (fields, outputs, records) is under the 256 MB Infinity Cache,
    # consecutive steps rotate over enough identical copies (>= 1 GiB
    # together) that every step reads its data from HBM, as a fresh batch would
    fields_b = sum(a.nbytes for a in w.inputs) + sum(a.nbytes for a in w.outputs)
    per_set = fields_b
    # the dominant kernel's roof: a convolutional stack whose flops take less
    # time at the fp32 vector peak than its arrays take at the HBM peak is
    # bound by HBM, and then every step reads a fresh copy of the batch
    # (rotation) so that the Infinity Cache does not serve it
    hbm_bound = is_cnn and cnn_hbm_bound(w, wl)
    rotate = args.rotate or hbm_bound
    model = api.CnnModel(w.model) if is_cnn else api.Model(w.model)
    sets = []
    for k in range(400):
        ins = [torch.from_numpy(a).cuda() for a in w.inputs]
        outs = [torch.from_numpy(a).cuda() for a in w.outputs]
        if args.inplace:
            if len(w.outputs) > len(ins) or any(o.shape != i.shape for o, i in zip(outs, ins)):
                print("--inplace needs outputs shaped like the first inputs", file=sys.stderr)
                sys.exit(2)
            outs = ins[:len(w.outputs)]
            args.no_cpu_baseline = True
        mi = api.Map(w.in_spec, ins, _abi.TO)
        mo = api.Map(w.out_spec, outs, _abi.FROM)
        mo_rec = api.Map(w.out_spec, outs, _abi.TO)        # the outputs as a recorded map
        rec_in = torch.empty((mi.n_points, mi.n_features), device="cuda")
        rec_out = torch.empty((mo.n_points, mo.n_features), device="cuda")
        sets.append((ins, outs, mi, mo, mo_rec, rec_in, rec_out))
        per_set = fields_b + 4 * (mi.n_points * mi.n_features + mo.n_points * mo.n_features)
        if not rotate or per_set >= (256 << 20) or (k + 1) * per_set >= (1 << 30):
            break
    n_sets = len(sets)
    ins, outs, mi, mo, mo_rec, rec_in, rec_out = sets[0]
    variant = api.variant(model, mi, mo)
    B, Fi, Fo, Bo = mi.n_points, mi.n_features, mo.n_features, mo.n_points
    stream = torch.cuda.current_stream()
    turn = [0]

    def step(ev=None):
        _, _, mi_k, mo_k, mo_rec_k, rec_in_k, rec_out_k = sets[turn[0] % n_sets]
        turn[0] += 1
        if ev is not None:
            ev[0].record(stream)
        api.infer(model, mi_k, mo_k, stream)
        if ev is not None:
            ev[1].record(stream)
        api.collect_pair(mi_k, rec_in_k, Fi, mo_rec_k, rec_out_k, Fo, stream)
        if ev is not None:
            ev[2].record(stream)

    if args.copy_calibration_mb:
        src = torch.empty(args.copy_calibration_mb << 18, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for k in range(args.steps):
        step(evs[k])
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(stop)
    infer_ms = [e[0].elapsed_time(e[1]) for e in evs]
    collect_ms = [e[1].elapsed_time(e[2]) for e in evs]
    ms_step = total_ms / args.steps
    infer_avg = float(np.mean(infer_ms))

    alg_bytes = sum(a.nbytes for a in w.inputs) + sum(a.nbytes for a in w.outputs)
    if is_cnn:
        H, W = w.model["image"]
        flop_launch = wl.cnn_flops_per_image(w.model) * (B // (H * W))
        peak, bound = VALU_F32_PEAK, "alu"
    else:
        flop_launch = w.flops_per_point * B
        peak, bound = PEAK[w.compute], "mfma"
    achieved = flop_launch / (infer_avg * 1e-3)
    if hbm_bound:
        peak, bound = HBM_PEAK, "hbm"
        achieved = alg_bytes / (infer_avg * 1e-3)
    traffic = recorded_traffic(variant, args.workload)
    # collect: every element of the mapped arrays read once, every record
    # word written once (in and out records)
    collect_bytes = (sum(a.nbytes for a in w.inputs) + 4 * B * Fi) + (sum(a.nbytes for a in w.outputs) + 4 * Bo * Fo)
    collect_avg = float(np.mean(collect_ms))
    collect_traffic = recorded_traffic("collect", args.workload)
    result = {
        "metric": "surrogate points/sec (gather+MLP+scatter) and % of HBM / MFMA roofline",
        "value": B / (ms_step * 1e-3),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.compute,
        "data": "synthetic (seeded generators; random-init He-normal weights)",
        "config": {"workload": DESCRIPTION[args.workload] + ("; outputs written in place into the input fields"
                                                              if args.inplace else ""),
                   "points": B, "features_in": Fi, "features_out": Fo, "output_points": Bo},
        "roofline": {"bound": bound, "achieved": achieved / (1e9 if hbm_bound else 1e12),
                     "peak": peak / (1e9 if hbm_bound else 1e12), "unit": "GB/s" if hbm_bound else "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic["bytes"] if traffic else None,
                     "traffic_source": traffic["source"] if traffic else None,
                     "algorithmic_hbm_bytes_per_launch": alg_bytes,
                     "kernel": variant, "kernel_avg_ms": infer_avg,
                     "algorithmic_flop_per_launch": flop_launch},
        "infer_points_per_s": B / (infer_avg * 1e-3),
        "infer_ms": {"mean": infer_avg, "median": float(np.median(infer_ms)), "min": float(np.min(infer_ms))},
        "collect_roofline": {"bound": "hbm", "achieved": collect_bytes / (collect_avg * 1e-3) / 1e9,
                             "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                             "frac": collect_bytes / (collect_avg * 1e-3) / HBM_PEAK,
                             "traffic": collect_traffic["bytes"] if collect_traffic else None,
                             "traffic_source": collect_traffic["source"] if collect_traffic else None,
                             "algorithmic_bytes_per_step": collect_bytes, "ms_per_step": collect_avg,
                             "kernels": "hpacml_collect_pair: the input map's and the output map's records"},
        "wall_s_timed": wall,
        "batch_copies": {"count": n_sets, "bytes_each": per_set,
                         "note": "steps rotate over identical copies so that data comes from HBM, not the "
                                 "256 MB Infinity Cache" if n_sets > 1 else "every step on the same arrays"},
    }

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

    if args.phases and not is_cnn:
        # mapping vs inference: the composed tensor (the input record) as F
        # contiguous column arrays under a pointwise map, outputs to Fo fresh
        # arrays, through the same fused kernel family
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

    if not args.no_cpu_baseline and is_cnn:
        import oracle
        # bounded sample: whole images (the oracle's unit), as many as fit the
        # CPU-time target, repeated until it is reached
        H, W = w.model["image"]
        S = B // (H * W)
        c0 = time.perf_counter()
        X1 = oracle.gather(dict(w.in_spec, sweep=_first_images(w.in_spec, 1)), w.inputs)
        Y1 = oracle.cnn(w.model, X1)
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
        got = np.stack([o.cpu().numpy().reshape(-1)[:n_out] for o in outs], 1).astype(np.float64)
        s = np.sqrt(np.mean(Y.astype(np.float64) ** 2, axis=0, keepdims=True))
        worst = float(np.max(np.abs(got - Y) / np.maximum(np.abs(Y), s)))
        result["cpu_baseline"] = {"value": reps * n_img * H * W / cpu_s, "unit": "points/s",
                                  "cores": oracle.num_threads(), "kind": "oracle",
                                  "sample": "the first %d of %d images x %d passes, gather + convolutional model "
                                            "in fp64, %.1fs" % (n_img, S, reps, cpu_s)}
        result["parity_on_cpu_sample"] = {"worst_scaled_error": worst, "rtol": 1e-5}
    elif not args.no_cpu_baseline:
        import oracle
        # bounded sample: as many seeded rows as fit the CPU-time target
        # (estimated from a short calibration run); when the whole batch takes
        # less, it is repeated until the target is reached
        n_cal = min(B, 4096)
        c0 = time.perf_counter()
        oracle.infer_rows(w.in_spec, w.inputs, w.model, np.arange(n_cal, dtype=np.int64))
        per_pt = (time.perf_counter() - c0) / n_cal
        n = int(min(B, max(n_cal, args.cpu_seconds / max(per_pt, 1e-12))))
        rows = wl.sample_rows(B, n, seed_k=998)
        reps, cpu_s = 0, 0.0
        while reps == 0 or cpu_s < args.cpu_seconds:
            c0 = time.perf_counter()
            Y = oracle.infer_rows(w.in_spec, w.inputs, w.model, rows)
            cpu_s += time.perf_counter() - c0
            reps += 1
        got = np.stack([o.cpu().numpy().reshape(-1)[rows] for o in outs], 1).astype(np.float64)
        s = np.sqrt(np.mean(Y.astype(np.float64) ** 2, axis=0, keepdims=True))
        worst = float(np.max(np.abs(got - Y) / np.maximum(np.abs(Y), s)))
        result["cpu_baseline"] = {"value": reps * len(rows) / cpu_s, "unit": "points/s",
                                  "cores": oracle.num_threads(), "kind": "oracle",
                                  "sample": "%d of %d sweep rows (seeded) x %d passes, gather + MLP in fp64, "
                                            "%.1fs" % (len(rows), B, reps, cpu_s)}
        result["parity_on_cpu_sample"] = {"worst_scaled_error": worst, "rtol": 1e-5 if w.compute == "f32" else 2e-2}

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

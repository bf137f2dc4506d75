"""The bench contract's host-side parts, on the CPU: one GPU only, the
roofline bound of the convolutional workloads, and the committed profile
summaries (each names the command that made it and carries parsable traffic
lines)."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + list(args), capture_output=True,
                          text=True, timeout=300)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_unknown_workload_is_an_argument_error():
    r = _bench("--workload", "no_such_workload")
    assert r.returncode == 2 and "invalid choice" in r.stderr


def test_convolutional_roofline_bounds():
    """The frame workload's 67 MB take longer at 8 TB/s than its 537 Mflop at
    157.3 TF/s (HBM-bound); the 2048^2 two-convolution step is the other way
    round (fp32 vector)."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2407_18352_amd import workloads as wl
    p = wl.make_cnn("particle_cnn", (64, 128, 128))
    assert bench.cnn_hbm_bound(p, wl)
    w = wl.make_cnn("weather_cnn", (256, 256))
    assert not bench.cnn_hbm_bound(w, wl)
    # the same rule by hand for the frame model: bytes/flops per frame
    H, W = p.model["image"]
    flops = wl.cnn_flops_per_image(p.model)
    assert 4 * H * W / 8.0e12 > flops / 157.3e12


def test_profiles_name_their_commands_and_parse():
    files = sorted(glob.glob(os.path.join(ROOT, "profiles", "*.txt")))
    assert files, "no profile summaries committed"
    kernels = set()
    for f in files:
        text = open(f).read()
        assert "rocprofv3" in text and "bench.py" in text, f
        assert "/root/reference" not in text and "_work" not in text, f
        for line in text.splitlines():
            if line.startswith("traffic_line "):
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                assert {"kernel", "workload", "bytes", "fetch", "write", "source_sha256"} <= set(kv), line
                assert int(kv["bytes"]) == pytest.approx(int(kv["fetch"]) + int(kv["write"]), abs=2)
                kernels.add((kv["kernel"], kv["workload"]))
    for name in ("bonds", "options", "stencil2d", "poses", "stencil3d", "weather_cnn", "particle_cnn"):
        assert ("collect", name) in kernels, name

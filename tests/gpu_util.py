"""Helpers shared by the GPU tests: run a workload through the HIP library
and compare with the oracle under the stated tolerance rule."""
import numpy as np

RTOL = {"f32": 1e-5, "bf16": 2e-2}


def require_gpu():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_18352_amd import _abi
    _abi.lib()          # raises loudly when the HIP library is missing


def to_dev(arrays):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in arrays]


def run_infer(w, repeat=1):
    """gather -> MLP -> scatter on the GPU; returns (outputs as numpy, variant)."""
    import torch
    from paper_2407_18352_amd import api, _abi
    ins = to_dev(w.inputs)
    outs = to_dev(w.outputs)
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, outs, _abi.FROM)
    model = api.Model(w.model)
    var = api.variant(model, mi, mo)
    for _ in range(repeat):
        api.infer(model, mi, mo)
    torch.cuda.synchronize()
    res = [o.cpu().numpy() for o in outs]
    mi.close(), mo.close(), model.close()
    return res, var


def run_collect(spec, arrays, ld=None, col=0, rows_total=None):
    import torch
    from paper_2407_18352_amd import api, _abi
    dev = to_dev(arrays)
    m = api.Map(spec, dev, _abi.TO)
    ld = m.n_features if ld is None else ld
    rec = torch.full((max(m.n_points, 1), ld), float("nan"), device="cuda")
    rec.view(torch.int32).fill_(-1)
    api.collect(m, rec[:, col:] if col else rec, ld)
    torch.cuda.synchronize()
    out = rec.cpu().numpy().view(np.uint32)
    m.close()
    return out


def parity_stats(got, want):
    """Tolerance rule: |g - o| <= rtol * max(|o|, s_g), s_g = RMS of the
    oracle output column g.  Returns (worst ratio err/max(|o|, s), normwise
    relative error, NaN count)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    s = np.sqrt(np.mean(want * want, axis=0, keepdims=True))
    s = np.where(s > 0, s, 1.0)
    scale = np.maximum(np.abs(want), s)
    ratio = np.abs(got - want) / scale
    nan = int(np.isnan(got).sum())
    norm = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-300))
    return float(np.nanmax(ratio)) if ratio.size else 0.0, norm, nan


def pure_relative(got, want):
    """Max |g - o| / |o| over the outputs with |o| >= s (s = the column RMS),
    where relative error is meaningful."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    s = np.sqrt(np.mean(want * want, axis=0, keepdims=True))
    mask = np.abs(want) >= s
    if not mask.any():
        return 0.0
    return float(np.max(np.abs(got - want)[mask] / np.abs(want)[mask]))


def assert_close(got, want, rtol, what=""):
    worst, norm, nan = parity_stats(got, want)
    assert nan == 0, "%s: %d NaN outputs" % (what, nan)
    assert worst <= rtol, "%s: worst scaled error %.3e > %.1e (normwise %.3e)" % (what, worst, rtol, norm)
    return worst, norm

"""hpacml_infer_noalloc through the C ABI: the same outputs as hpacml_infer,
bit for bit, on in-place regions whose snapshot record lives in the library's
fixed scratch array, on two calls in a row (the second smaller), and on a
region that needs no record; a record larger than the array is refused before
anything runs."""
import numpy as np
import pytest

from paper_2407_18352_amd import _abi, api
from paper_2407_18352_amd import workloads as wl
from gpu_util import require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def _noalloc(model, mi, mo):
    import torch
    st = torch.cuda.current_stream().cuda_stream
    return _abi.lib().hpacml_infer_noalloc(model.handle, mi.handle, mo.handle, st)


def _run_both(w, inplace):
    """Fields after hpacml_infer and after hpacml_infer_noalloc, each on its
    own copy of the same inputs."""
    import torch
    res = []
    model = api.Model(w.model)
    for use_noalloc in (False, True):
        ins = to_dev(w.inputs)
        outs = ins[:len(w.outputs)] if inplace else to_dev(w.outputs)
        mi = api.Map(w.in_spec, ins, _abi.TO)
        mo = api.Map(w.out_spec, outs, _abi.FROM)
        if use_noalloc:
            st = _noalloc(model, mi, mo)
            assert st == _abi.OK, st
        else:
            api.infer(model, mi, mo)
        torch.cuda.synchronize()
        res.append([t.cpu().numpy().copy() for t in (ins + ([] if inplace else outs))])
        variant = api.variant(model, mi, mo)
        mi.close(), mo.close()
    model.close()
    return res, variant


@pytest.mark.parametrize("name, sizes", [
    ("stencil2d", [(67, 131), (23, 40)]),        # fp32, 3x3 window written back into its fields
    ("stencil3d", [(12, 20, 70), (5, 9, 33)]),   # bf16, 7-point window written back
])
def test_noalloc_matches_infer_in_place_twice(name, sizes):
    for size in sizes:        # two calls in a row, the second on a smaller input
        w = wl.make(name, size)
        (a, b), variant = _run_both(w, inplace=True)
        assert variant.startswith("snapshot+"), variant
        for x, y in zip(a, b):
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), (name, size)


def test_noalloc_without_a_record_matches_infer():
    w = wl.make("bonds", 5003)
    (a, b), variant = _run_both(w, inplace=False)
    assert not variant.startswith("snapshot+")
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))


def test_noalloc_refuses_a_record_beyond_the_scratch_array():
    import torch
    # 1024 x 1024 cells x 36 features x 4 bytes = 151 MB > 64 MiB
    w = wl.make("stencil2d", (1024, 1024))
    ins = to_dev(w.inputs)
    before = [t.clone() for t in ins]
    mi = api.Map(w.in_spec, ins, _abi.TO)
    mo = api.Map(w.out_spec, ins[:4], _abi.FROM)
    model = api.Model(w.model)
    assert _noalloc(model, mi, mo) == _abi.E_RANGE
    torch.cuda.synchronize()
    for x, y in zip(ins, before):
        assert torch.equal(x, y)
    mi.close(), mo.close(), model.close()

"""Argument checks of the Python binding that need no device: host weight
arrays whose sizes do not match the model description are refused before
the library reads them through plain pointers."""
import numpy as np
import pytest

from paper_2407_18352_amd import _abi, api
from paper_2407_18352_amd import workloads as wl


def _reaches_library(spec, cls):
    """Correct sizes pass the binding's check (the library may then succeed,
    or fail without a device)."""
    try:
        cls(spec).close()
    except _abi.HpacmlError:
        pass


def test_mlp_weight_sizes_checked():
    spec = wl.make_model(3, [9, 32, 2], "f32")
    _reaches_library(spec, api.Model)
    bad = dict(spec, W=[spec["W"][0], spec["W"][1][:, :31]])
    with pytest.raises(ValueError, match="layer 1"):
        api.Model(bad)
    bad = dict(spec, b=[spec["b"][0][:31], spec["b"][1]])
    with pytest.raises(ValueError, match="layer 0"):
        api.Model(bad)
    bad = dict(spec, W=spec["W"][:1])
    with pytest.raises(ValueError, match="weight"):
        api.Model(bad)


@pytest.mark.parametrize("name", wl.CNN_NAMES)
def test_cnn_weight_sizes_checked(name):
    spec = wl.cnn_model(name, "small")
    _reaches_library(spec, api.CnnModel)
    i = next(k for k, ly in enumerate(spec["layers"]) if ly["kind"] != "pool")
    layers = [dict(ly) for ly in spec["layers"]]
    layers[i]["W"] = np.asarray(layers[i]["W"]).reshape(-1)[:-1]
    with pytest.raises(ValueError, match="layer %d" % i):
        api.CnnModel(dict(spec, layers=layers))
    layers = [dict(ly) for ly in spec["layers"]]
    j = len(layers) - 1
    layers[j]["b"] = np.concatenate([np.asarray(layers[j]["b"]).reshape(-1), [0.0]])
    with pytest.raises(ValueError, match="layer %d" % j):
        api.CnnModel(dict(spec, layers=layers))


def test_invalid_description_left_to_the_library_status():
    spec = wl.cnn_model("weather_cnn", "small")
    bad = dict(spec, layers=[dict(spec["layers"][0], kernel=(0, 3))] + spec["layers"][1:])
    with pytest.raises(_abi.HpacmlError) as e:
        api.CnnModel(bad)
    assert e.value.status == _abi.E_INVAL

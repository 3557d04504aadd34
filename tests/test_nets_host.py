"""The library's layer lists (used by the benchmark and the driver) describe
the same graphs as the oracle's networks (used by every parity test), layer by
layer and field by field, for all five workloads."""
import pytest

from oracle import nets as onets
from paper_2005_14038_amd import nets as lnets
from paper_2005_14038_amd import workloads

from stage_harness import to_layers


def _norm(d):
    # bias is a flag on both sides; eps a float
    return {k: (bool(v) if k == "bias" else v) for k, v in d.items()}


@pytest.mark.parametrize("name", ["tiny", "vgg19_s1", "vgg19", "resnet152_mid", "resnet152"])
def test_library_layer_lists_equal_the_oracle_graphs(name):
    lib = lnets.by_name(name)
    ora = onets.by_name(name)
    assert (lib.input_shape) == (ora.H, ora.W, ora.C)
    a = [_norm(d) for d in lib.layers]
    b = [_norm(d) for d in to_layers(ora)]
    assert len(a) == len(b)
    for i, (x, y) in enumerate(zip(a, b)):
        assert x == y, (name, i, x, y)
    assert lib.param_count() == ora.param_count()


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_workload_shapes_match_the_networks(name):
    wl = workloads.WORKLOADS[name]
    ora = onets.by_name(wl.net, **wl.net_kw)
    assert (wl.H, wl.W, wl.C) == (ora.H, ora.W, ora.C)
    assert wl.has_loss == ora.has_loss
    if ora.has_loss:
        assert wl.classes == ora.nodes[-1]["classes"]

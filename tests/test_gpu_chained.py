"""Every layer of real stage graphs checked element by element against the
oracle on the layer's own GPU inputs (see chained.py): the five workloads'
networks at reduced spatial size and 12 seeded random residual graphs, in
fp32 (max relative error 1e-3) and bf16 (2e-2)."""
import pytest

from chained import check_layers
from gpu_common import dev  # noqa: F401
from stage_harness import make_inputs, oracle_weights
from test_gpu_stage import SMALL, random_graph

pytestmark = pytest.mark.gpu


def _report(name, dtype, fails, n):
    assert n > 0
    msg = "\n".join(f"  layer {i}: {what}: error {e:.3e} (bound {t:.1e})"
                    for i, what, e, t in fails[:40])
    assert not fails, f"{name} {dtype}: {len(fails)} of {n} layer checks failed:\n{msg}"


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("name", list(SMALL))
def test_every_layer_of_the_workload_graphs(dev, name, dtype):  # noqa: F811
    mk, B, need_dx, _ = SMALL[name]
    net = mk()
    w = oracle_weights(net, 71, scale_bn=True)
    x, lab, dy = make_inputs(net, B, 72, dy_std=1e-3)
    fails, n = check_layers(net, B, w, x, lab, dy, need_dx, dtype)
    _report(name, dtype, fails, n)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("seed", range(12))
def test_every_layer_of_random_residual_graphs(dev, seed, dtype):  # noqa: F811
    net = random_graph(seed)
    B = 2 + seed % 2
    w = oracle_weights(net, 90 + seed, scale_bn=True)
    x, lab, dy = make_inputs(net, B, 91 + seed, dy_std=1e-3)
    fails, n = check_layers(net, B, w, x, lab, dy, True, dtype)
    _report(f"graph {seed}", dtype, fails, n)

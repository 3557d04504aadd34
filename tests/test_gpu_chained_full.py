"""Every layer of the full-size workloads checked element by element on
sampled outputs against the oracle fed with the layer's own GPU inputs (see
chained_full.py): the VGG-19 stage 1, the full VGG-19 and the ResNet-152
middle stage (with its input gradient) in fp32 at 1e-3, the full ResNet-152
in bf16 at 2e-2, batch 32, one minibatch in the benchmark's configuration."""
import numpy as np
import pytest

from chained_full import check_stage_sampled
from gpu_common import dev  # noqa: F401
from oracle import nets as onets
from paper_2005_14038_amd import workloads

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["vgg19_s1", "vgg19", "resnet152_mid", "resnet152"])
def test_every_layer_at_full_size(dev, name):  # noqa: F811
    wl = workloads.WORKLOADS[name]
    net = onets.by_name(wl.net, **wl.net_kw)
    layers = wl.builder().layers
    w0 = workloads.initial_weights(wl, layers)
    x, lab, dy = workloads.inputs(wl, net.out_shape, 0, 1)
    fails, n = check_stage_sampled(net, wl.batch, w0, x, lab, dy, wl.need_dx, wl.dtype,
                                   log=lambda m: print(f"{name}: {m}", flush=True))
    msg = "\n".join(f"  layer {i}: {what}: error {e:.3e} (bound {t:.1e})"
                    for i, what, e, t in fails[:40])
    assert n > 3 * len([nd for nd in net.nodes if nd["op"] == "conv"])
    assert not fails, f"{name}: {len(fails)} of {n} layer checks failed:\n{msg}"

"""The five stage workloads, as concrete sizes and WSP settings.

Inputs are synthetic stand-ins for ImageNet (the paper's dataset, Sec. 6):
images N(0, 1) of the paper's shape (224x224x3 at batch 32), labels uniform
over the classes, the upstream gradient of a middle stage N(0, 1e-3^2),
He-normal initial weights (biases 0, batch-norm gamma 1 and beta 0), all
drawn from the counter-based generator of ``seeded_inputs``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import seeded_inputs as si

from . import nets
from .hetpipe import HP_BN, HP_CONV, HP_FC

SEED = 20052014


@dataclass
class Workload:
    name: str
    net: str
    batch: int
    H: int
    W: int
    C: int
    N: int                 # virtual workers
    s_local: int           # wave length W = s_local + 1
    D: int                 # clock-distance bound
    waves: int
    lr: float
    dtype: str = "fp32"
    periods: list = field(default_factory=list)
    dy_std: float | None = None
    classes: int = 0
    net_kw: dict = field(default_factory=dict)
    seed: int = SEED
    # a middle stage hands the gradient of its input back to the previous
    # stage (Sec. 3), so its step computes dx; a first stage reads the image
    need_dx: bool = False

    def builder(self):
        return nets.by_name(self.net, **self.net_kw)

    @property
    def has_loss(self):
        return self.dy_std is None


WORKLOADS = {
    "tiny": Workload("tiny", "tiny", 4, 16, 16, 3, N=2, s_local=3, D=0, waves=3, lr=0.01,
                     classes=10, periods=[1, 1]),
    "vgg19_s1": Workload("vgg19_s1", "vgg19_s1", 32, 224, 224, 3, N=1, s_local=3, D=0, waves=3,
                         lr=0.01, dy_std=1e-3, periods=[1]),
    "vgg19": Workload("vgg19", "vgg19", 32, 224, 224, 3, N=4, s_local=3, D=0, waves=2, lr=0.01,
                      classes=1000, periods=[1, 1, 1, 1]),
    "resnet152_mid": Workload("resnet152_mid", "resnet152_mid", 32, 56, 56, 256, N=1, s_local=4,
                              D=0, waves=3, lr=0.1, dy_std=1e-3, periods=[1], need_dx=True),
    "resnet152": Workload("resnet152", "resnet152", 32, 224, 224, 3, N=4, s_local=3, D=1,
                          waves=5, lr=0.01, dtype="bf16", classes=1000, periods=[1, 1, 1, 2]),
}


def param_segments(layers):
    """(kind, count, fan_in) of each parameter segment in flat order."""
    segs = []
    for d in layers:
        k = d["kind"]
        if k == HP_CONV:
            fan = d["R"] * d["S"] * d["C"]
            segs.append(("w", d["K"] * fan, fan))
            if d.get("bias"):
                segs.append(("b", d["K"], None))
        elif k == HP_FC:
            segs.append(("w", d["K"] * d["C"], d["C"]))
            if d.get("bias"):
                segs.append(("b", d["K"], None))
        elif k == HP_BN:
            segs.append(("gamma", d["C"], None))
            segs.append(("beta", d["C"], None))
    return segs


def initial_weights(wl: Workload, layers) -> np.ndarray:
    return si.initial_weights(param_segments(layers), wl.seed)


def inputs(wl: Workload, out_shape, vw: int, q: int):
    """Host arrays (x, labels or None, dy or None) of minibatch q of VW vw."""
    B = wl.batch
    x = si.normal(si.stream_key(wl.seed, vw, q, si.T_X), B * wl.H * wl.W * wl.C)
    x = x.reshape(B, wl.H, wl.W, wl.C)
    if wl.has_loss:
        lab = si.labels(si.stream_key(wl.seed, vw, q, si.T_LABELS), B, wl.classes)
        return x, lab, None
    n = B * int(np.prod(out_shape))
    dy = si.normal(si.stream_key(wl.seed, vw, q, si.T_DY), n, wl.dy_std).reshape((B,) + tuple(out_shape))
    return x, None, dy

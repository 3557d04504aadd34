"""Run one stage step on the GPU (through the C ABI) and in the oracle on the
same seeded inputs."""
import numpy as np
import torch

import seeded_inputs as si
from oracle import nets as onets
from oracle import stage as ostage
from paper_2005_14038_amd import hetpipe as hp

KIND = {"conv": hp.HP_CONV, "fc": hp.HP_FC, "relu": hp.HP_RELU, "maxpool": hp.HP_MAXPOOL,
        "bn": hp.HP_BN, "add": hp.HP_ADD, "gap": hp.HP_GAP, "ce": hp.HP_SOFTMAX_CE}


def to_layers(net):
    """The oracle's layer graph as hp_layer dictionaries."""
    out = []
    for nd in net.nodes:
        k = nd["op"]
        d = dict(kind=KIND[k], in0=nd["in"])
        if k == "conv":
            d.update(C=nd["C"], K=nd["K"], R=nd["R"], S=nd["S"], stride=nd["stride"],
                     pad=nd["pad"], bias=nd["bias"])
        elif k == "fc":
            d.update(C=nd["IN"], K=nd["OUT"], bias=nd["bias"])
        elif k == "maxpool":
            d.update(R=nd["R"], S=nd["R"], stride=nd["stride"], pad=nd["pad"])
        elif k == "bn":
            d.update(C=nd["C"], eps=nd["eps"])
        elif k == "add":
            d.update(in1=nd["in2"])
        elif k == "ce":
            d.update(K=nd["classes"])
        out.append(d)
    return out


def oracle_weights(net, seed, scale_bn=False):
    segs = []
    for i, name, shape, fan in net.param_segments():
        n = int(np.prod(shape))
        segs.append(("w" if name == "w" else name, n, fan))
    w = si.initial_weights(segs, seed)
    if scale_bn:
        # move BN gamma/beta away from (1, 0) so their gradients are exercised
        off = 0
        for i, name, shape, fan in net.param_segments():
            n = int(np.prod(shape))
            if name in ("gamma", "beta"):
                r = si.normal(si.stream_key(seed, 1, off, si.T_PROBE), n, 0.2)
                w[off:off + n] = (1.0 if name == "gamma" else 0.0) + r
            off += n
    return w


def make_inputs(net, B, seed, q=1, dy_std=1.0):
    x = si.normal(si.stream_key(seed, 0, q, si.T_X), B * net.H * net.W * net.C)
    x = x.reshape(B, net.H, net.W, net.C)
    if net.has_loss:
        lab = si.labels(si.stream_key(seed, 0, q, si.T_LABELS), B, net.nodes[-1]["classes"])
        return x, lab, None
    shp = (B,) + tuple(net.out_shape)
    dy = si.normal(si.stream_key(seed, 0, q, si.T_DY), int(np.prod(shp)), dy_std).reshape(shp)
    return x, None, dy


def run_gpu(net, B, w, x, labels, dy, need_dx, dtype="fp32", dev="cuda:0"):
    st = hp.Stage(to_layers(net), B, net.H, net.W, net.C, dtype=dtype)
    assert st.P == len(w), (st.P, len(w))
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(dev)
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(dev)
    grad = torch.full((max(st.P, 1),), float("nan"), dtype=torch.float32, device=dev)
    dx = torch.full(x.shape, float("nan"), dtype=torch.float32, device=dev) if need_dx else None
    if net.has_loss:
        yshape = (B, net.nodes[-1]["classes"])
        y = torch.empty(yshape, dtype=torch.float32, device=dev)
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        lt = torch.from_numpy(np.ascontiguousarray(labels, np.int32)).to(dev)
        st.forward(wt, xt, y, lt, loss)
        st.backward(wt, None, dx, grad)
    else:
        y = torch.empty((B,) + tuple(net.out_shape), dtype=torch.float32, device=dev)
        loss = None
        st.forward(wt, xt, y)
        dyt = torch.from_numpy(np.ascontiguousarray(dy, np.float32)).to(dev)
        st.backward(wt, dyt, dx, grad)
    torch.cuda.synchronize()
    out = dict(y=y.cpu().numpy(), grad=grad.cpu().numpy()[:st.P],
               loss=float(loss.item()) if loss is not None else None,
               dx=dx.cpu().numpy() if dx is not None else None)
    st.close()
    return out


def run_oracle(net, w, x, labels, dy, need_dx, bf16=False):
    r = ostage.step(net, np.asarray(w, np.float64), x, labels=labels, dy=dy, need_dx=need_dx,
                    bf16=bf16)
    return r


def single(op_fn, H, W, C):
    """A one-purpose Net built by op_fn(net) -> None."""
    n = onets.Net("probe", H, W, C)
    op_fn(n)
    return n

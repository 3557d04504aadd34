"""Forward and backward of one pipeline stage (a layer graph) on the CPU.

TEST INFRASTRUCTURE ONLY (see the package docstring).

HetPipe's stage is a contiguous run of a CNN's layers executed on one GPU of a
virtual worker (Sec. 3, pipelined model parallelism): the forward pass of a
minibatch runs the layers in order, the backward pass runs them in reverse and
produces the weight gradients of the stage plus, when the stage is not the
first one, the gradient with respect to the stage input.  Forward and backward
of one minibatch use the same weight version (Sec. 4: w_p is kept until p's
backward pass).

Precision: everything is float64.  In bf16 mode every operand of a contraction
(conv / FC weights, their input activations, and the upstream gradients fed to
dgrad and wgrad) is rounded to bfloat16 first (``bf16.round_bf16``); BN, ReLU,
pooling, the residual add, the loss and the bias gradient (a plain sum of the
upstream gradient) stay in full precision.
"""
from __future__ import annotations

import numpy as np

from . import ops
from .bf16 import round_bf16


def unflatten(net, flat):
    """Split a flat parameter vector into {(node, name): array} views."""
    out = {}
    off = 0
    for i, name, shape, _ in net.param_segments():
        n = int(np.prod(shape))
        out[(i, name)] = np.asarray(flat[off:off + n], dtype=np.float64).reshape(shape)
        off += n
    assert off == len(flat), (off, len(flat))
    return out


def flatten_grads(net, grads):
    parts = []
    for i, name, shape, _ in net.param_segments():
        parts.append(np.asarray(grads[(i, name)], dtype=np.float64).reshape(-1))
    return np.concatenate(parts) if parts else np.zeros(0)


def forward(net, params_flat, x, labels=None, bf16=False):
    """Returns (values, loss, saved) where values[i] is node i's output."""
    prm = unflatten(net, params_flat)
    rnd = round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    x = np.asarray(x, np.float64)
    vals = []
    saved = {}
    loss = None

    def inp(j):
        return x if j < 0 else vals[j]

    for i, nd in enumerate(net.nodes):
        k = nd["op"]
        a = inp(nd["in"])
        if k == "conv":
            y = ops.conv_fwd(rnd(a), rnd(prm[(i, "w")]),
                             prm.get((i, "b")), nd["stride"], nd["pad"])
        elif k == "fc":
            y = ops.fc_fwd(rnd(a.reshape(a.shape[0], -1)), rnd(prm[(i, "w")]),
                           prm.get((i, "b")))
        elif k == "relu":
            y = ops.relu_fwd(a)
        elif k == "maxpool":
            y = ops.maxpool_fwd(a, nd["R"], nd["stride"], nd["pad"])
        elif k == "bn":
            y, mu, iv = ops.bn_fwd(a, prm[(i, "gamma")], prm[(i, "beta")], nd["eps"])
            saved[i] = (mu, iv)
        elif k == "add":
            y = a + inp(nd["in2"])
        elif k == "gap":
            y = ops.gap_fwd(a)
        elif k == "ce":
            assert labels is not None
            loss, dz = ops.softmax_ce(a, labels)
            saved[i] = dz
            y = np.zeros(0)
        else:
            raise ValueError(k)
        vals.append(y)
    return vals, loss, saved


def backward(net, params_flat, x, vals, saved, dy=None, need_dx=False, bf16=False):
    """Returns (flat weight gradient, dx or None).

    ``dy`` is the gradient at the stage output (None when the stage ends in the
    loss head).  The gradient of a value consumed by several nodes is the sum of
    what each consumer sends back."""
    prm = unflatten(net, params_flat)
    rnd = round_bf16 if bf16 else (lambda a: np.asarray(a, np.float64))
    x = np.asarray(x, np.float64)
    nn = len(net.nodes)
    grad_of = [None] * nn
    gx = None
    grads = {}

    def inp(j):
        return x if j < 0 else vals[j]

    def send(j, g):
        nonlocal gx
        if j < 0:
            gx = g if gx is None else gx + g
        else:
            grad_of[j] = g if grad_of[j] is None else grad_of[j] + g

    if not net.has_loss:
        assert dy is not None
        grad_of[nn - 1] = np.asarray(dy, np.float64)

    for i in range(nn - 1, -1, -1):
        nd = net.nodes[i]
        k = nd["op"]
        if k == "ce":
            send(nd["in"], saved[i])
            continue
        g = grad_of[i]
        if g is None:
            continue
        a = inp(nd["in"])
        wants_dx = nd["in"] >= 0 or need_dx
        if k == "conv":
            w = prm[(i, "w")]
            dw, _ = ops.conv_wgrad(rnd(a), rnd(g), nd["R"], nd["S"], nd["stride"],
                                   nd["pad"], False)
            grads[(i, "w")] = dw
            if nd["bias"]:
                # the bias gradient is a plain sum of dy, not a contraction: no rounding
                grads[(i, "b")] = g.reshape(-1, nd["K"]).sum(axis=0)
            if wants_dx:
                send(nd["in"], ops.conv_dgrad(rnd(g), rnd(w), nd["stride"], nd["pad"],
                                              a.shape[1], a.shape[2]))
        elif k == "fc":
            w = prm[(i, "w")]
            a2 = a.reshape(a.shape[0], -1)
            dw, _ = ops.fc_wgrad(rnd(a2), rnd(g), False)
            grads[(i, "w")] = dw
            if nd["bias"]:
                grads[(i, "b")] = g.sum(axis=0)
            if wants_dx:
                send(nd["in"], ops.fc_dgrad(rnd(g), rnd(w)).reshape(a.shape))
        elif k == "relu":
            send(nd["in"], ops.relu_bwd(a, g))
        elif k == "maxpool":
            send(nd["in"], ops.maxpool_bwd(a, g, nd["R"], nd["stride"], nd["pad"]))
        elif k == "bn":
            mu, iv = saved[i]
            dxx, dg, dbt = ops.bn_bwd(a, g, prm[(i, "gamma")], mu, iv)
            grads[(i, "gamma")] = dg
            grads[(i, "beta")] = dbt
            send(nd["in"], dxx)
        elif k == "add":
            send(nd["in"], g)
            send(nd["in2"], g)
        elif k == "gap":
            send(nd["in"], ops.gap_bwd(g, a.shape[1], a.shape[2]))
        else:
            raise ValueError(k)
    for i, name, shape, _ in net.param_segments():
        if (i, name) not in grads:          # a parameter no gradient reached
            grads[(i, name)] = np.zeros(shape)
    return flatten_grads(net, grads), (gx if need_dx else None)


def step(net, params_flat, x, labels=None, dy=None, need_dx=False, bf16=False):
    """One minibatch: forward then backward at the same weights.

    Returns dict(loss, y (stage output), grad (flat), dx)."""
    vals, loss, saved = forward(net, params_flat, x, labels, bf16)
    grad, dx = backward(net, params_flat, x, vals, saved, dy, need_dx, bf16)
    y = vals[-2] if net.has_loss else vals[-1]
    return dict(loss=loss, y=y, grad=grad, dx=dx)

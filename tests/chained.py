"""Layer-by-layer parity of a real stage graph: every layer of the graph is
checked element by element against the oracle's operator evaluated on that
layer's own inputs as the GPU holds them after one forward and backward pass
(hp_stage_layer_buffers), so a wiring error anywhere in the graph -- a lost
shortcut gradient, a ReLU mask applied to the wrong value, a gradient added
twice -- shows up at the layer where it happens, and the chaotic growth of
rounding differences along a deep graph (which a whole-stage comparison has
to allow for) does not enter.

For each layer the checks are:
  forward   the oracle's operator on the GPU's input values against the GPU's
            output value (through the consumer ReLU where the layer applies
            it itself);
  backward  for every value with a gradient buffer: the sum over its
            consumers of the oracle's backward of each consumer, fed with the
            consumer's output gradient as the GPU holds it (derived one layer
            on where no buffer holds it: a ReLU's mask, an add's pass-through)
            and the GPU's forward values, against the GPU's gradient;
  weights   the oracle's weight, bias and batch-norm parameter gradients from
            the GPU's input value and output gradient against the GPU's
            gradient vector.
In bf16 mode the contraction operands are rounded to bf16 as the GPU rounds
them: the GPU's fp32 values go through the same round-to-nearest-even.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import ops
from oracle import stage as ostage
from oracle.bf16 import round_bf16
from paper_2005_14038_amd import hetpipe as hp

from gpu_common import BF16_TOL, FP32_TOL, rel_err
from stage_harness import to_layers


def _consumers(net):
    cons = {}
    for c, nd in enumerate(net.nodes):
        cons.setdefault(nd["in"], []).append((c, 0))
        if nd["op"] == "add":
            cons.setdefault(nd["in2"], []).append((c, 1))
    return cons


def _shape(net, i, B):
    s = (net.H, net.W, net.C) if i < 0 else net.shapes[i]
    return (B,) + tuple(s)


def run_and_read(net, B, w, x, labels, dy, need_dx, dtype, devc="cuda:0"):
    """One forward + backward on the GPU; returns the GPU's values and
    gradients of every layer (None where the stage holds none), its flat
    weight gradient and its loss."""
    st = hp.Stage(to_layers(net), B, net.H, net.W, net.C, dtype=dtype)
    assert st.P == len(w), (st.P, len(w))
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(devc)
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(devc)
    grad = torch.full((max(st.P, 1),), float("nan"), dtype=torch.float32, device=devc)
    dx = torch.full(x.shape, float("nan"), dtype=torch.float32, device=devc) if need_dx else None
    loss = None
    if net.has_loss:
        y = torch.empty((B, net.nodes[-1]["classes"]), dtype=torch.float32, device=devc)
        lt = torch.from_numpy(np.ascontiguousarray(labels, np.int32)).to(devc)
        loss = torch.empty(1, dtype=torch.float32, device=devc)
        st.forward(wt, xt, y, lt, loss)
        st.backward(wt, None, dx, grad)
    else:
        y = torch.empty(_shape(net, len(net.nodes) - 1, B), dtype=torch.float32, device=devc)
        dyt = torch.from_numpy(np.ascontiguousarray(dy, np.float32)).to(devc)
        st.forward(wt, xt, y)
        st.backward(wt, dyt, dx, grad)
    torch.cuda.synchronize()
    V, G = {}, {}
    for i in range(-1, len(net.nodes)):
        vp, gp = st.layer_buffers(i)
        if i >= 0 and net.nodes[i]["op"] == "ce":
            assert vp is None and gp is None
            continue
        n = int(np.prod(_shape(net, i, B)))
        V[i] = hp.read_vector(vp, n).reshape(_shape(net, i, B)) if vp else None
        G[i] = hp.read_vector(gp, n).reshape(_shape(net, i, B)) if gp else None
    out = dict(V=V, G=G, grad=grad.cpu().numpy()[:st.P],
               loss=float(loss.item()) if loss is not None else None)
    st.close()
    return out


def check_layers(net, B, w, x, labels, dy, need_dx, dtype, gpu=None, tol=None):
    """Runs the stage on the GPU (unless `gpu` holds such a run) and returns
    the list of failures [(layer, what, error, tol)]; empty when every layer
    matches.  Also returns the number of checks made."""
    if gpu is None:
        gpu = run_and_read(net, B, w, x, labels, dy, need_dx, dtype)
    bf = dtype == "bf16"
    tol = tol if tol is not None else (BF16_TOL if bf else FP32_TOL)
    rnd = round_bf16 if bf else (lambda a: np.asarray(a, np.float64))
    prm = ostage.unflatten(net, np.asarray(w, np.float64))
    V = {k: (None if v is None else np.asarray(v, np.float64)) for k, v in gpu["V"].items()}
    G = {k: (None if v is None else np.asarray(v, np.float64)) for k, v in gpu["G"].items()}
    cons = _consumers(net)
    nodes = net.nodes
    n = len(nodes)
    fails, checks = [], [0]

    def cmp(i, what, a, r, exact=False, bound=None):
        checks[0] += 1
        a = np.asarray(a, np.float64)
        r = np.asarray(r, np.float64)
        if exact:
            if not np.array_equal(a, r):
                fails.append((i, what, float(np.max(np.abs(a - r))), 0.0))
            return
        if bound is not None:
            # a result that is exactly zero in exact arithmetic: both sides are
            # round-off, held to the bound of recursive summation
            e = float(np.max(np.abs(a - r) - bound))
            if e > 0:
                fails.append((i, what, e, 0.0))
            return
        e = rel_err(a, r)
        if e > tol:
            fails.append((i, what, e, tol))

    def val(j):
        if j < 0:
            return V[-1]
        if V.get(j) is not None:
            return V[j]
        return None

    def relu_of(i):
        """The ReLU consumer that holds node i's value when i applies it."""
        (c, _), = cons[i]
        assert nodes[c]["op"] == "relu", (i, c)
        return c

    bn_stats = {}

    def bn_saved(i):
        if i not in bn_stats:
            _, mu, iv = ops.bn_fwd(val(nodes[i]["in"]), prm[(i, "gamma")], prm[(i, "beta")],
                                   nodes[i]["eps"])
            bn_stats[i] = (mu, iv)
        return bn_stats[i]

    # ---------------------------------------------------------------- forward
    for i, nd in enumerate(nodes):
        k = nd["op"]
        if k == "ce":
            zl = val(nd["in"])
            lref, dz = ops.softmax_ce(zl, labels)
            cmp(i, "loss", np.array([gpu["loss"]]), np.array([lref]))
            cmp(i, "loss gradient", G[nd["in"]], dz)
            continue
        a = val(nd["in"])
        if k == "relu" and a is None:
            continue                            # applied by its producer: checked there
        assert a is not None, (i, "input value not held")
        if k == "conv":
            y = ops.conv_fwd(rnd(a), rnd(prm[(i, "w")]), prm.get((i, "b")), nd["stride"],
                             nd["pad"])
        elif k == "fc":
            y = ops.fc_fwd(rnd(a.reshape(B, -1)), rnd(prm[(i, "w")]), prm.get((i, "b")))
        elif k == "bn":
            y, _, _ = ops.bn_fwd(a, prm[(i, "gamma")], prm[(i, "beta")], nd["eps"])
        elif k == "add":
            y = a + val(nd["in2"])
        elif k == "relu":
            cmp(i, "relu forward", V[i], ops.relu_fwd(a), exact=True)
            continue
        elif k == "maxpool":
            cmp(i, "max-pool forward", V[i], ops.maxpool_fwd(a, nd["R"], nd["stride"], nd["pad"]),
                exact=True)
            continue
        elif k == "gap":
            y = ops.gap_fwd(a)
        else:
            raise ValueError(k)
        y = y.reshape(_shape(net, i, B))
        if V[i] is None:                       # the layer applies its consumer ReLU
            cmp(i, f"{k} + relu forward", V[relu_of(i)], ops.relu_fwd(y))
        else:
            cmp(i, f"{k} forward", V[i], y)

    # --------------------------------------------------------------- backward
    def bwd_to(c, slot, E):
        """The gradient consumer c sends to its input `slot` given its output
        gradient E (oracle operators on the GPU's forward values)."""
        nd = nodes[c]
        k = nd["op"]
        j = nd["in"] if slot == 0 else nd["in2"]
        sh = _shape(net, j, B)
        if k == "conv":
            return ops.conv_dgrad(rnd(E), rnd(prm[(c, "w")]), nd["stride"], nd["pad"], sh[1], sh[2])
        if k == "fc":
            return ops.fc_dgrad(rnd(E.reshape(B, -1)), rnd(prm[(c, "w")])).reshape(sh)
        if k == "relu":
            return ops.relu_bwd(V[c], E)        # V[c] > 0 exactly where its input is
        if k == "maxpool":
            return ops.maxpool_bwd(val(j), E, nd["R"], nd["stride"], nd["pad"])
        if k == "bn":
            mu, iv = bn_saved(c)
            dxx, _, _ = ops.bn_bwd(val(j), E, prm[(c, "gamma")], mu, iv)
            return dxx
        if k == "add":
            return E
        if k == "gap":
            return ops.gap_bwd(E.reshape(B, -1), sh[1], sh[2])
        if k == "ce":
            return ops.softmax_ce(val(j), labels)[1]
        raise ValueError(k)

    memo = {}

    def eff(i):
        """dL/d(value i) as the GPU has it: its buffer, or one layer on from
        the consumers' buffers where the stage keeps none."""
        if i in memo:
            return memo[i]
        if G.get(i) is not None:
            memo[i] = G[i]
            return memo[i]
        tot = None
        for c, slot in cons.get(i, []):
            if nodes[c]["op"] == "ce":
                g = ops.softmax_ce(val(i), labels)[1]
            else:
                Ec = eff(c)
                if Ec is None:
                    continue
                g = bwd_to(c, slot, Ec)
            tot = g if tot is None else tot + g
        memo[i] = tot
        return tot

    for j in range(-1, n):
        if j >= 0 and nodes[j]["op"] == "ce":
            continue
        if G.get(j) is None or (j == n - 1 and not net.has_loss):
            continue
        if any(nodes[c]["op"] == "ce" for c, _ in cons.get(j, [])):
            continue                            # the logits: checked with the loss
        ref = None
        for c, slot in cons.get(j, []):
            Ec = eff(c)
            if Ec is None:
                continue
            g = bwd_to(c, slot, Ec)
            ref = g if ref is None else ref + g
        assert ref is not None, (j, "a gradient buffer no consumer feeds")
        what = "input gradient" if j < 0 else f"gradient of {nodes[j]['op']} output"
        cmp(j, what, G[j], ref)

    # ---------------------------------------------------------------- weights
    off = 0
    readers = {}
    for c, nd in enumerate(nodes):
        readers.setdefault(nd["in"], []).append(nd["op"])
        if nd["op"] == "add":
            readers.setdefault(nd["in2"], []).append(nd["op"])
    got = np.asarray(gpu["grad"], np.float64)
    for i, name, shape, _ in net.param_segments():
        cnt = int(np.prod(shape))
        seg = got[off:off + cnt].reshape(shape)
        off += cnt
        nd = nodes[i]
        E = eff(i)
        if E is None:
            cmp(i, f"{name} gradient (unreached)", seg, np.zeros(shape), exact=True)
            continue
        a = val(nd["in"])
        if nd["op"] == "conv":
            if name == "w":
                ref, _ = ops.conv_wgrad(rnd(a), rnd(E), nd["R"], nd["S"], nd["stride"], nd["pad"],
                                        False)
                cmp(i, "conv weight gradient", seg, ref)
            else:
                E2 = E.reshape(-1, nd["K"])
                ref = E2.sum(axis=0)
                if all(op == "bn" for op in readers.get(i, ["-"])):
                    bound = 2 * E2.shape[0] * 2.0 ** -24 * np.abs(E2).sum(axis=0)
                    cmp(i, "conv bias gradient (exact zero)", seg, ref, bound=bound)
                else:
                    cmp(i, "conv bias gradient", seg, ref)
        elif nd["op"] == "fc":
            E2 = E.reshape(B, -1)
            if name == "w":
                ref, _ = ops.fc_wgrad(rnd(a.reshape(B, -1)), rnd(E2), False)
                cmp(i, "fc weight gradient", seg, ref)
            else:
                cmp(i, "fc bias gradient", seg, E2.sum(axis=0))
        elif nd["op"] == "bn":
            mu, iv = bn_saved(i)
            _, dg, dbt = ops.bn_bwd(a, E, prm[(i, "gamma")], mu, iv)
            cmp(i, f"batch-norm {name} gradient", seg, dg if name == "gamma" else dbt)
    return fails, checks[0]

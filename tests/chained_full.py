"""Layer-by-layer parity of a full-size stage on sampled outputs.

The same checks as chained.py -- every layer's forward output, every value's
gradient and every parameter gradient against the oracle's operator fed with
that layer's own inputs as the GPU holds them after one forward and backward
pass, element by element at 1e-3 (fp32) or 2e-2 (bf16) -- at the workloads'
full sizes.  Contractions are evaluated by the oracle only at sampled outputs
(one per 64 x 64 block of each output matrix, so every tile a kernel
computes, whole or cut, is represented, up to a cap per tensor); the
element-wise layers and batch norms are evaluated at the same samples from
per-channel statistics of the whole GPU tensors.  GPU buffers are read on
demand, so a whole ResNet-152 at batch 32 fits in host memory.
"""
from __future__ import annotations

import time

import numpy as np
import torch

from oracle import ops
from oracle import stage as ostage
from paper_2005_14038_amd import hetpipe as hp

from gpu_common import BF16_TOL, FP32_TOL, rel_err
from stage_harness import to_layers

BLOCK = 64


def rnd_bf16(a):
    """Round to the nearest bfloat16, ties to even, returned as float64: the
    rounding rule of oracle.bf16.round_bf16 on 32-bit words (finite values;
    test_chained_full_host pins the two equal)."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32).astype(np.float64)


def block_samples(rows, cols, rng, cap):
    """Flat indices of one element in every BLOCK x BLOCK block of a rows x cols
    matrix; above `cap` blocks a random subset that keeps the ragged last
    block row and column."""
    br, bc = -(-rows // BLOCK), -(-cols // BLOCK)
    bi = np.repeat(np.arange(br), bc)
    bj = np.tile(np.arange(bc), br)
    if bi.size > cap:
        edge = (bi == br - 1) | (bj == bc - 1)
        inner = np.flatnonzero(~edge)
        keep = np.concatenate([np.flatnonzero(edge),
                               rng.choice(inner, size=max(0, min(inner.size, cap - int(edge.sum()))),
                                          replace=False)])
        bi, bj = bi[keep], bj[keep]
    r0, c0 = bi * BLOCK, bj * BLOCK
    r = r0 + (rng.random(r0.size) * np.minimum(BLOCK, rows - r0)).astype(np.int64)
    c = c0 + (rng.random(c0.size) * np.minimum(BLOCK, cols - c0)).astype(np.int64)
    return np.unique(np.concatenate([r * cols + c, [0, rows * cols - 1]]))


def _consumers(net):
    cons = {}
    for c, nd in enumerate(net.nodes):
        cons.setdefault(nd["in"], []).append((c, 0))
        if nd["op"] == "add":
            cons.setdefault(nd["in2"], []).append((c, 1))
    return cons


class _Reader:
    """GPU buffers of the stage read on demand into host float32 arrays,
    with a bounded cache."""

    def __init__(self, st, net, B, limit=24e9):
        self.net, self.B, self.limit = net, B, limit
        self.ptr = {}
        for i in range(-1, len(net.nodes)):
            if i >= 0 and net.nodes[i]["op"] == "ce":
                continue
            self.ptr[i] = st.layer_buffers(i)
        self.cache = {}

    def shape(self, i):
        s = (self.net.H, self.net.W, self.net.C) if i < 0 else self.net.shapes[i]
        return (self.B,) + tuple(s)

    def _get(self, i, which):
        key = (i, which)
        if key in self.cache:
            v = self.cache.pop(key)
            self.cache[key] = v
            return v
        p = self.ptr[i][which]
        if not p:
            return None
        shp = self.shape(i)
        v = hp.read_vector(p, int(np.prod(shp))).reshape(shp)
        self.cache[key] = v
        while sum(a.nbytes for a in self.cache.values()) > self.limit and len(self.cache) > 1:
            self.cache.pop(next(iter(self.cache)))
        return v

    def value(self, i):
        return self._get(i, 0)

    def grad(self, i):
        return self._get(i, 1)


def check_stage_sampled(net, B, w, x, labels, dy, need_dx, dtype, cap=2048, seed=5,
                        log=lambda m: None, devc="cuda:0"):
    """Runs one forward + backward of the stage on the GPU and checks every
    layer on sampled outputs.  Returns (failures [(layer, what, err, tol)],
    number of checks)."""
    bf = dtype == "bf16"
    tol = BF16_TOL if bf else FP32_TOL
    rnd = rnd_bf16 if bf else (lambda a: np.asarray(a, np.float64))
    st = hp.Stage(to_layers(net), B, net.H, net.W, net.C, dtype=dtype)
    assert st.P == len(w)
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(devc)
    xt = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(devc)
    grad = torch.full((st.P,), float("nan"), dtype=torch.float32, device=devc)
    dxt = torch.full(x.shape, float("nan"), dtype=torch.float32, device=devc) if need_dx else None
    loss = None
    if net.has_loss:
        yt = torch.empty((B, net.nodes[-1]["classes"]), dtype=torch.float32, device=devc)
        lt = torch.from_numpy(np.ascontiguousarray(labels, np.int32)).to(devc)
        losst = torch.empty(1, dtype=torch.float32, device=devc)
        st.forward(wt, xt, yt, lt, losst)
        st.backward(wt, None, dxt, grad)
    else:
        yt = torch.empty((B,) + tuple(net.out_shape), dtype=torch.float32, device=devc)
        dyt = torch.from_numpy(np.ascontiguousarray(dy, np.float32)).to(devc)
        st.forward(wt, xt, yt)
        st.backward(wt, dyt, dxt, grad)
    torch.cuda.synchronize()
    if net.has_loss:
        loss = float(losst.item())
    gvec = grad.cpu().numpy().astype(np.float64)
    R = _Reader(st, net, B)
    try:
        return _check(net, B, w, labels, R, gvec, loss, rnd, tol, cap, seed, log)
    finally:
        st.close()


def _check(net, B, w, labels, R, gvec, loss, rnd, tol, cap, seed, log):
    prm = ostage.unflatten(net, np.asarray(w, np.float64))
    nodes = net.nodes
    n = len(nodes)
    cons = _consumers(net)
    rng = np.random.default_rng(seed)
    fails, checks = [], [0]
    t0 = time.time()

    def cmp(i, what, a, r, exact=False, bound=None):
        checks[0] += 1
        a = np.asarray(a, np.float64)
        r = np.asarray(r, np.float64)
        if exact:
            if not np.array_equal(a, r):
                fails.append((i, what, float(np.max(np.abs(a - r))), 0.0))
        elif bound is not None:
            e = float(np.max(np.abs(a - r) - bound))
            if e > 0:
                fails.append((i, what, e, 0.0))
        else:
            e = rel_err(a, r)
            if e > tol:
                fails.append((i, what, e, tol))

    def samples_of(shape):
        C = shape[-1]
        return block_samples(int(np.prod(shape)) // C, C, rng, cap)

    def fused_relu(i):
        """The consumer ReLU whose buffer holds node i's value, if i applies it."""
        if R.ptr[i][0] is not None:
            return None
        (c, _), = cons[i]
        assert nodes[c]["op"] == "relu"
        return c

    def val(j):
        v = R.value(j)
        assert v is not None, f"value of layer {j} is not held"
        return v

    rounded = {}

    def rval(j):
        """The value of j as a contraction operand (bf16-rounded in bf16 mode)."""
        k = ("v", j)
        if k not in rounded:
            rounded.clear()
            rounded[k] = rnd(val(j))
        return rounded[k]

    bn_cache = {}

    def bn_stats(i):
        """mean, invstd (biased variance) of batch norm i's input, fp64."""
        if i not in bn_cache:
            bn_cache.clear()
            xin = val(nodes[i]["in"])
            C = xin.shape[-1]
            x2 = xin.reshape(-1, C).astype(np.float64)
            mu = x2.mean(axis=0)
            var = ((x2 - mu) ** 2).mean(axis=0)
            bn_cache[i] = (mu, 1.0 / np.sqrt(var + nodes[i]["eps"]))
        return bn_cache[i]

    # ---------------------------------------------------------------- forward
    for i, nd in enumerate(nodes):
        k = nd["op"]
        if k == "ce":
            zl = val(nd["in"])
            lref, dz = ops.softmax_ce(zl, labels)
            cmp(i, "loss", [loss], [lref])
            cmp(i, "loss gradient", R.grad(nd["in"]), dz)
            continue
        if k == "relu" and R.ptr[nd["in"]][0] is None:
            continue                               # applied by its producer: checked there
        relu = fused_relu(i) if k in ("conv", "fc", "bn", "add") else None
        out = R.value(relu if relu is not None else i)
        shp = R.shape(i)
        if k == "conv":
            idx = samples_of(shp)
            ref = ops.conv_fwd_at(rval(nd["in"]), rnd(prm[(i, "w")]), prm.get((i, "b")),
                                  nd["stride"], nd["pad"], idx)
        elif k == "fc":
            idx = np.arange(int(np.prod(shp)))
            ref = ops.fc_fwd(rval(nd["in"]).reshape(B, -1), rnd(prm[(i, "w")]),
                             prm.get((i, "b"))).reshape(-1)
        elif k == "bn":
            idx = samples_of(shp)
            mu, iv = bn_stats(i)
            C = shp[-1]
            xin = val(nd["in"]).reshape(-1)[idx].astype(np.float64)
            ch = idx % C
            ref = prm[(i, "gamma")][ch] * (xin - mu[ch]) * iv[ch] + prm[(i, "beta")][ch]
        elif k == "add":
            idx = samples_of(shp)
            ref = (val(nd["in"]).reshape(-1)[idx].astype(np.float64) +
                   val(nd["in2"]).reshape(-1)[idx].astype(np.float64))
        elif k == "relu":
            cmp(i, "relu forward", out, np.maximum(val(nd["in"]), 0), exact=True)
            continue
        elif k == "maxpool":
            ref = ops.maxpool_fwd(val(nd["in"]), nd["R"], nd["stride"], nd["pad"])
            cmp(i, "max-pool forward", out, ref, exact=True)
            continue
        elif k == "gap":
            idx = np.arange(int(np.prod(shp)))
            ref = ops.gap_fwd(val(nd["in"])).reshape(-1)
        else:
            raise ValueError(k)
        if relu is not None:
            ref = np.maximum(ref, 0.0)
        cmp(i, f"{k}{' + relu' if relu is not None else ''} forward", out.reshape(-1)[idx], ref)
    log(f"forward checked ({time.time() - t0:.0f} s)")

    # --------------------------------------------------------------- backward
    full_memo = {}

    def eff_full(i):
        """dL/d(value i) as a whole tensor: the GPU's buffer, or, where none
        holds it, the ReLU consumer's buffer through the ReLU's mask (a batch
        norm or add that applies its ReLU)."""
        g = R.grad(i)
        if g is not None:
            return g
        if i in full_memo:
            return full_memo[i]
        cs = cons.get(i, [])
        if len(cs) == 1 and nodes[cs[0][0]]["op"] == "ce":
            return None
        tot = None
        for c, _ in cs:
            if nodes[c]["op"] == "relu":
                g = np.where(val(c) > 0, eff_full(c), np.float32(0))
            elif nodes[c]["op"] == "add":       # passes its gradient on unchanged
                g = eff_full(c)
            else:
                raise AssertionError(f"no whole gradient for layer {i}")
            tot = g if tot is None else tot + g
        if tot is None:
            raise AssertionError(f"no whole gradient for layer {i}")
        full_memo.clear()
        full_memo[i] = tot
        return tot

    def bwd_at(c, slot, j, idx):
        """What consumer c sends to its input j at the flat indices idx."""
        nd = nodes[c]
        k = nd["op"]
        sh = R.shape(j)
        if k == "conv":
            return ops.conv_dgrad_at(rnd(eff_full(c)), rnd(prm[(c, "w")]), nd["stride"], nd["pad"],
                                     sh[1], sh[2], idx)
        if k == "fc":
            return ops.fc_dgrad(rnd(eff_full(c).reshape(B, -1)),
                                rnd(prm[(c, "w")])).reshape(-1)[idx]
        if k == "relu":
            m = val(c).reshape(-1)[idx] > 0
            g = R.grad(c)
            inner = g.reshape(-1)[idx].astype(np.float64) if g is not None else grad_at(c, idx)
            return np.where(m, inner, 0.0)
        if k == "maxpool":
            return ops.maxpool_bwd(val(j), eff_full(c), nd["R"], nd["stride"],
                                   nd["pad"]).reshape(-1)[idx]
        if k == "bn":
            mu, iv = bn_stats(c)
            E = eff_full(c)
            C = sh[-1]
            x2 = val(j).reshape(-1, C).astype(np.float64)
            E2 = E.reshape(-1, C).astype(np.float64)
            xh = (x2 - mu) * iv
            M = x2.shape[0]
            s1, s2 = E2.sum(axis=0), (E2 * xh).sum(axis=0)
            ch = idx % C
            e_i = E.reshape(-1)[idx].astype(np.float64)
            xh_i = xh.reshape(-1)[idx]
            return prm[(c, "gamma")][ch] * iv[ch] * (e_i - s1[ch] / M - xh_i * s2[ch] / M)
        if k == "add":
            g = R.grad(c)
            if g is None and c in full_memo:
                g = full_memo[c]
            if g is None:
                try:
                    g = eff_full(c)
                except AssertionError:
                    return grad_at(c, idx)
            return g.reshape(-1)[idx].astype(np.float64)
        if k == "gap":
            C = sh[-1]
            HW = sh[1] * sh[2]
            E = eff_full(c).reshape(B, C).astype(np.float64)
            return E[idx // (HW * C), idx % C] / HW
        if k == "ce":
            return ops.softmax_ce(val(j), labels)[1].reshape(-1)[idx]
        raise ValueError(k)

    def grad_at(j, idx):
        tot = np.zeros(idx.size)
        for c, slot in cons.get(j, []):
            tot = tot + bwd_at(c, slot, j, idx)
        return tot

    for j in range(n - 1, -2, -1):
        if j >= 0 and nodes[j]["op"] == "ce":
            continue
        g = R.grad(j)
        if g is None or (j == n - 1 and not net.has_loss):
            continue
        if any(nodes[c]["op"] == "ce" for c, _ in cons.get(j, [])):
            continue                               # the logits: checked with the loss
        idx = samples_of(R.shape(j))
        ref = grad_at(j, idx)
        what = "input gradient" if j < 0 else f"gradient of {nodes[j]['op']} output"
        cmp(j, what, g.reshape(-1)[idx], ref)
    log(f"data gradients checked ({time.time() - t0:.0f} s)")

    # ---------------------------------------------------------------- weights
    readers = {}
    for c, nd in enumerate(nodes):
        readers.setdefault(nd["in"], []).append(nd["op"])
        if nd["op"] == "add":
            readers.setdefault(nd["in2"], []).append(nd["op"])
    off = 0
    for i, name, shape, _ in net.param_segments():
        cnt = int(np.prod(shape))
        seg = gvec[off:off + cnt]
        off += cnt
        nd = nodes[i]
        E = eff_full(i)
        if nd["op"] == "conv":
            if name == "w":
                idx = block_samples(shape[0], cnt // shape[0], rng, cap)
                ref = ops.conv_wgrad_at(rval(nd["in"]), rnd(E), nd["R"], nd["S"], nd["stride"],
                                        nd["pad"], idx)
                cmp(i, "conv weight gradient", seg[idx], ref)
            else:
                E2 = E.reshape(-1, nd["K"]).astype(np.float64)
                ref = E2.sum(axis=0)
                if all(op == "bn" for op in readers.get(i, ["-"])):
                    bound = 2 * E2.shape[0] * 2.0 ** -24 * np.abs(E2).sum(axis=0)
                    cmp(i, "conv bias gradient (exact zero)", seg, ref, bound=bound)
                else:
                    cmp(i, "conv bias gradient", seg, ref)
        elif nd["op"] == "fc":
            E2 = E.reshape(B, -1).astype(np.float64)
            if name == "w":
                idx = block_samples(shape[0], shape[1], rng, cap)
                a = rval(nd["in"]).reshape(B, -1)
                ref = (rnd(E2)[:, idx // shape[1]] * a[:, idx % shape[1]]).sum(axis=0)
                cmp(i, "fc weight gradient", seg[idx], ref)
            else:
                cmp(i, "fc bias gradient", seg, E2.sum(axis=0))
        elif nd["op"] == "bn":
            mu, iv = bn_stats(i)
            C = shape[0]
            x2 = val(nd["in"]).reshape(-1, C).astype(np.float64)
            E2 = E.reshape(-1, C).astype(np.float64)
            ref = (E2 * ((x2 - mu) * iv)).sum(axis=0) if name == "gamma" else E2.sum(axis=0)
            cmp(i, f"batch-norm {name} gradient", seg, ref)
    log(f"weight gradients checked ({time.time() - t0:.0f} s)")
    return fails, checks[0]

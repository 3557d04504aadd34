"""One virtual worker as a pipeline of k partitions on one GPU.

HetPipe runs a virtual worker (VW) as pipelined model parallelism over k GPUs
(Sec. 3, Sec. 4): the layers are cut into k consecutive partitions, up to N_m
minibatches are in the pipeline at once, and a new minibatch enters as soon as
an earlier one completes.  Here the k partitions share one GPU: partition q
runs on its own HIP stream, cross-partition order is carried by HIP events,
and every partition keeps one activation stash (stage object) per minibatch
it holds at once, as each minibatch's forward activations and weight version
must survive until its backward pass (Sec. 4).

Scheduling follows the rules of Sec. 4 (partition scheduling): on every
partition the forward tasks run in minibatch order, the backward tasks run in
minibatch order, and ready tasks are taken first-in first-out; on the last
partition a minibatch's forward and backward form one task.  The host cannot
observe readiness on the device, so the task order of every stream comes
from a discrete-event simulation of those rules with nominal task durations
(``schedule``); the device then executes each stream in that order and the
events enforce the data dependencies.

Weights follow the local-staleness rule of Sec. 4 exactly: minibatch q uses
the version with the local updates 1..q-N_m (N_m = W = s_local + 1), because
minibatch q enters only when q-N_m has completed and completions are in
order.  The WSP calls (hp_wsp_weights at entry, hp_wsp_local_update at
completion, push and pull at a wave end) are the same as for a sequential
VW, so the result is identical to running the minibatches one after another.
"""
from __future__ import annotations

import heapq
from dataclasses import dataclass

import torch

from .hetpipe import (HP_ADD, HP_BN, HP_CONV, HP_FC, HP_GAP, HP_MAXPOOL, HP_SOFTMAX_CE,
                      ParameterServer, Stage, VirtualWorker)


# ----------------------------------------------------------------- partitions

def _refs(d):
    r = [d.get("in0", -1)]
    if d["kind"] == HP_ADD:
        r.append(d.get("in1", -1))
    return r


def valid_cuts(layers):
    """Indices i such that cutting after layer i leaves exactly one tensor (the
    output of layer i) crossing the cut, and the loss head keeps a layer before
    it in its partition.  A conv and the batch norm reading it stay together:
    the batch norm takes its statistics from the conv's contraction, and a cut
    between them would change the order of those sums, so the pipeline would
    no longer reproduce the sequential stage bit for bit."""
    n = len(layers)
    # earliest layer referenced by any later layer
    cuts = []
    min_ref_after = [n] * (n + 1)
    for j in range(n - 1, -1, -1):
        r = min(_refs(layers[j]))
        min_ref_after[j] = min(min_ref_after[j + 1], r)
    for i in range(n - 1):
        if min_ref_after[i + 1] < i:
            continue
        if layers[-1]["kind"] == HP_SOFTMAX_CE and i == n - 2:
            continue
        if layers[i]["kind"] == HP_CONV and any(
                d["kind"] == HP_BN and d.get("in0", -1) == i for d in layers[i + 1:]):
            continue
        cuts.append(i)
    return cuts


def param_count(d):
    k = d["kind"]
    if k == HP_CONV:
        return d["K"] * d["R"] * d["S"] * d["C"] + (d["K"] if d.get("bias") else 0)
    if k == HP_FC:
        return d["K"] * d["C"] + (d["K"] if d.get("bias") else 0)
    if k == HP_BN:
        return 2 * d["C"]
    return 0


def layer_shapes(layers, H, W, C):
    """Per-image output shape of every layer (and -1: the input)."""
    shape = {-1: (H, W, C)}
    for i, d in enumerate(layers):
        h, w, c = shape[d.get("in0", -1)]
        k = d["kind"]
        if k == HP_CONV:
            shape[i] = ((h + 2 * d["pad"] - d["R"]) // d["stride"] + 1,
                        (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1, d["K"])
        elif k == HP_FC:
            shape[i] = (1, 1, d["K"])
        elif k == HP_MAXPOOL:
            shape[i] = ((h + 2 * d["pad"] - d["R"]) // d["stride"] + 1,
                        (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1, c)
        elif k == HP_GAP:
            shape[i] = (1, 1, c)
        elif k == HP_SOFTMAX_CE:
            shape[i] = (1, 1, 0)
        else:
            shape[i] = (h, w, c)
    return shape


def layer_costs(layers, H, W, C, batch):
    """Nominal forward + backward work of every layer: 6 FLOP per MAC of a
    contraction, 20 per output element of anything else."""
    shape = layer_shapes(layers, H, W, C)
    cost = []
    for i, d in enumerate(layers):
        h, w, c = shape[i]
        if d["kind"] == HP_CONV:
            cost.append(6.0 * batch * h * w * c * d["R"] * d["S"] * d["C"])
        elif d["kind"] == HP_FC:
            cost.append(6.0 * batch * d["K"] * d["C"])
        else:
            cost.append(20.0 * batch * h * w * max(c, 1))
    return cost


def balanced_cuts(layers, k, cost):
    """k-1 valid cuts minimising the largest partition cost (exact, by
    dynamic programming over the valid cut points)."""
    n = len(layers)
    pts = [-1] + valid_cuts(layers) + [n - 1]      # partition = (pts[a], pts[b]]
    if k > len(pts) - 1:
        raise ValueError(f"{k} partitions need {k - 1} cuts; only {len(pts) - 2} are valid")
    pre = [0.0]
    for c in cost:
        pre.append(pre[-1] + c)

    def seg(a, b):            # cost of layers pts[a]+1 .. pts[b]
        return pre[pts[b] + 1] - pre[pts[a] + 1]

    m = len(pts)
    INF = float("inf")
    best = [[INF] * m for _ in range(k + 1)]
    arg = [[-1] * m for _ in range(k + 1)]
    best[0][0] = 0.0
    for j in range(1, k + 1):
        for b in range(1, m):
            for a in range(b):
                if best[j - 1][a] == INF:
                    continue
                v = max(best[j - 1][a], seg(a, b))
                if v < best[j][b]:
                    best[j][b] = v
                    arg[j][b] = a
    cuts = []
    b = m - 1
    for j in range(k, 0, -1):
        a = arg[j][b]
        if j > 1:
            cuts.append(pts[a])
        b = a
    return sorted(cuts)


@dataclass
class Partition:
    layers: list        # renumbered layer dictionaries (-1 = the partition input)
    first: int          # index of the first layer in the full list
    last: int           # index of the last layer
    in_shape: tuple     # per-image input shape
    out_shape: tuple    # per-image output shape (of the last layer)
    p_off: int          # first parameter of the partition in the flat vector
    p_cnt: int


def split(layers, cuts, H, W, C):
    """Partitions of `layers` cut after each index in `cuts`."""
    ok = set(valid_cuts(layers))
    for c in cuts:
        if c not in ok:
            raise ValueError(f"cut after layer {c} leaves more than one tensor crossing it")
    shape = layer_shapes(layers, H, W, C)
    bounds = [-1] + sorted(cuts) + [len(layers) - 1]
    offs = [0]
    for d in layers:
        offs.append(offs[-1] + param_count(d))
    parts = []
    for a, b in zip(bounds[:-1], bounds[1:]):
        first = a + 1
        sub = []
        for j in range(first, b + 1):
            d = dict(layers[j])
            for key in ("in0", "in1"):
                if key in d:
                    r = d[key]
                    d[key] = -1 if r == a else r - first
            sub.append(d)
        parts.append(Partition(sub, first, b, shape[a], shape[b], offs[first],
                               offs[b + 1] - offs[first]))
    return parts


# ----------------------------------------------------------------- schedule

@dataclass(order=True)
class Task:
    start: float
    kind: str           # "F" forward, "FB" last partition forward+backward, "B" backward,
                        # "U" completion: local update (+ push / pull at a wave end)
    m: int              # minibatch (1-based)
    q: int              # partition (0-based; -1 for "U")
    end: float = 0.0


def schedule(k, W, total, d_fwd=None, d_bwd=None, d_upd=0.0):
    """Task order of a k-partition pipeline with up to W minibatches in flight
    (the rules of Sec. 4), simulated with per-partition forward / backward
    durations (default 1 and 2, the ratio the paper's pipeline figure
    assumes).  Minibatch m+W enters when minibatch m completes.  Among tasks
    ready on one partition the earliest-ready runs first; ties go to the older
    minibatch.  Returns the tasks in order of start time."""
    d_fwd = list(d_fwd) if d_fwd else [1.0] * k
    d_bwd = list(d_bwd) if d_bwd else [2.0] * k
    free = [0.0] * k
    queue = [[] for _ in range(k)]          # heap of (ready, m, kind) per partition
    next_f = [1] * k                        # forward order per partition
    next_b = [1] * k                        # backward order per partition
    out = []

    def ready(q, t, m, kind):
        heapq.heappush(queue[q], (t, m, 0 if kind != "F" else 1, kind))

    for m in range(1, min(W, total) + 1):
        ready(0, 0.0, m, "F" if k > 1 else "FB")
    done = 0
    while done < total:
        # the partition whose FIFO head can start first
        best = None
        for q in range(k):
            if not queue[q]:
                continue
            t, m, _, kind = queue[q][0]
            in_order = (m == next_f[q]) if kind in ("F", "FB") else (m == next_b[q])
            if not in_order:
                continue
            s = max(free[q], t)
            if best is None or (s, q) < (best[0], best[1]):
                best = (s, q)
        if best is None:
            raise RuntimeError("pipeline schedule stalled")
        s, q = best
        t, m, _, kind = heapq.heappop(queue[q])
        dur = d_fwd[q] + d_bwd[q] if kind == "FB" else (d_fwd[q] if kind == "F" else d_bwd[q])
        e = s + dur
        free[q] = e
        out.append(Task(s, kind, m, q, e))
        if kind in ("F", "FB"):
            next_f[q] += 1
        if kind in ("B", "FB"):
            next_b[q] += 1
        if kind == "F":
            ready(q + 1, e, m, "FB" if q + 1 == k - 1 else "F")
        elif q > 0:
            ready(q - 1, e, m, "B")
        else:                                  # minibatch m completed
            out.append(Task(e, "U", m, -1, e + d_upd))
            done += 1
            if m + W <= total:
                ready(0, e + d_upd, m + W, "F" if k > 1 else "FB")
    out.sort(key=lambda t: (t.start, t.kind != "U", t.q, t.m))
    return out


def stash_counts(k, W, d_fwd=None, d_bwd=None):
    """Largest number of minibatches that partition q holds at once between
    the start of their forward and the end of their backward pass, under the
    schedule above (Sec. 4: the first partition holds the most, the last one
    only the minibatch it is processing).  On one partition the forward and
    the backward tasks each run in minibatch order, so the minibatches held
    form a contiguous range and minibatch m can use stash m mod count."""
    total = 3 * W + 2 * k
    held = [0] * k
    most = [0] * k
    for t in schedule(k, W, total, d_fwd, d_bwd):
        if t.kind == "F":
            held[t.q] += 1
            most[t.q] = max(most[t.q], held[t.q])
        elif t.kind == "FB":
            most[t.q] = max(most[t.q], held[t.q] + 1)
        elif t.kind == "B":
            held[t.q] -= 1
    return most


# ----------------------------------------------------------------- driver

class PipelinedVW:
    """One VW of a stage list with a loss head, cut into partitions, under WSP
    with a parameter server in device memory (N = 1)."""

    def __init__(self, layers, batch, H, W, C, w0: torch.Tensor, s_local: int, lr: float,
                 data_fn, cuts, dtype="fp32", D=0, d_fwd=None, d_bwd=None):
        if layers[-1]["kind"] != HP_SOFTMAX_CE:
            raise ValueError("a pipelined VW needs the loss head in its last partition")
        self.parts = split(layers, cuts, H, W, C)
        self.k = len(self.parts)
        self.W = s_local + 1
        self.lr = lr if callable(lr) else (lambda n, q, _lr=lr: _lr)
        self.batch = batch
        self.data_fn = data_fn
        self.d_fwd, self.d_bwd = d_fwd, d_bwd
        dev = w0.device
        self.P = sum(p.p_cnt for p in self.parts)
        self.streams = [torch.cuda.Stream(device=dev) for _ in range(self.k)]
        self.ps_stream = torch.cuda.Stream(device=dev)
        # one stage object (activation stash) per minibatch a partition holds
        # at once: minibatch m uses stash (m - 1) mod slots[q]
        self.slots = stash_counts(self.k, self.W, d_fwd, d_bwd)
        self.stages = [[Stage(p.layers, batch, *p.in_shape, dtype=dtype, stream=s)
                        for _ in range(n)]
                       for p, s, n in zip(self.parts, self.streams, self.slots)]
        for p, st in zip(self.parts, self.stages):
            assert st[0].P == p.p_cnt, (st[0].P, p.p_cnt)
        self.acts = [[torch.empty((batch,) + tuple(p.out_shape), dtype=torch.float32, device=dev)
                      for _ in range(self.W)] for p in self.parts[:-1]]
        self.gx = [[torch.empty_like(a) for a in row] for row in self.acts]
        self.grads = [torch.empty(self.P, dtype=torch.float32, device=dev)
                      for _ in range(self.W)]
        self.loss = [torch.empty(1, dtype=torch.float32, device=dev) for _ in range(self.W)]
        torch.cuda.synchronize(dev)
        self.ps = ParameterServer(self.P, w0, 1, D, self.ps_stream)
        self.vw = VirtualWorker(self.ps, 0, s_local)
        torch.cuda.synchronize(dev)          # ring versions initialised on the server stream
        self.events = []
        self.wptr = {}
        self.inputs = {}
        self.done_ev = {}
        self.started = 0
        self.completed = 0

    def close(self):
        torch.cuda.synchronize()
        for row in self.stages:
            for st in row:
                st.close()
        self.vw.close()
        self.ps.close()

    # ---- helpers ----
    def _record(self, key, stream):
        ev = torch.cuda.Event()
        ev.record(stream)
        self.done_ev[key] = ev

    def _wait(self, stream, key):
        ev = self.done_ev.get(key)
        if ev is not None:
            stream.wait_event(ev)

    def _enter(self, m):
        """Minibatch m enters the pipeline: hp_wsp_weights (local staleness)."""
        self.events.append(("mb", 0, m, self.vw.version()))
        self.wptr[m] = self.vw.weights()
        self.inputs[m] = self.data_fn(0, m)
        self.started = m

    def run(self, waves):
        total = waves * self.W
        first = self.completed + 1
        tasks = schedule(self.k, self.W, total - self.completed, self.d_fwd, self.d_bwd)
        for t in tasks:
            t.m += first - 1
        for m in range(first, min(first + self.W, total + 1)):
            self._enter(m)
        for t in tasks:
            m, q = t.m, t.q
            slot = (m - 1) % self.W
            if t.kind == "U":
                self._complete(m, slot, total)
                continue
            part, s = self.parts[q], self.streams[q]
            st = self.stages[q][(m - 1) % self.slots[q]]
            w = self.wptr[m] + 4 * part.p_off
            grad = self.grads[slot][part.p_off:]
            x, labels, _ = self.inputs[m]
            if t.kind in ("F", "FB"):
                if q == 0:
                    self._wait(s, ("U", m - self.W))      # the ring slot is written
                else:
                    self._wait(s, ("F", m, q - 1))
                xin = x if q == 0 else self.acts[q - 1][slot]
                if t.kind == "F":
                    st.forward(w, xin, self.acts[q][slot])
                    self._record(("F", m, q), s)
                else:
                    st.forward(w, xin, None, labels, self.loss[slot])
                    st.backward(w, None, self.gx[q - 1][slot] if q > 0 else None, grad)
                    self._record(("B", m, q), s)
            else:
                self._wait(s, ("B", m, q + 1))
                st.backward(w, self.gx[q][slot], self.gx[q - 1][slot] if q > 0 else None, grad)
                self._record(("B", m, q), s)
        return self.events

    def _complete(self, m, slot, total):
        """Minibatch m completed: local update, push / pull at a wave end, then
        the next minibatch enters."""
        self._wait(self.ps_stream, ("B", m, 0))
        if m % self.W == 0:
            # local update + push + gate in one call (hp_wsp_wave_end)
            g0 = self.vw.state()["g"]
            ok = self.vw.wave_end(self.grads[slot], self.lr(0, m))
            s = self.vw.state()
            self.events.append(("push", 0, s["c"], self.ps.clock()))
            if not ok:
                raise RuntimeError("a single VW cannot be blocked by the clock bound")
            if s["g"] != g0:
                self.events.append(("pull", 0, s["g"]))
        else:
            self.vw.local_update(self.grads[slot], self.lr(0, m))
        self._record(("U", m), self.ps_stream)
        self.completed = m
        for key in [k for k in self.done_ev if k[1] == m and k[0] != "U"]:
            del self.done_ev[key]
        self.done_ev.pop(("U", m - self.W), None)
        del self.wptr[m]
        del self.inputs[m]
        if m + self.W <= total:
            self._enter(m + self.W)

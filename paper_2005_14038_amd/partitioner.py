"""Model partitioner of a virtual worker (HetPipe Sec. 4, model partitioning;
Sec. 6, partitioning algorithm).

Given the layers of a model, k possibly heterogeneous GPUs in pipeline order
and N_m minibatches in flight, choose k-1 cuts that minimise the largest
partition execution time while every partition fits its GPU's memory.

* Execution time of a partition = the summed computation time of its layers
  on its GPU plus the time to receive the activations entering it (forward)
  and the gradients entering it from the next partition (backward).  Layer
  times are measured on the MI355X (``profile``: HIP events around every
  kernel of a timed stage step, attributed to layers); another GPU type is a
  relative speed.  Transfer time = bytes / link bandwidth.
* Memory of a partition = its stashes (one stage object per minibatch it
  holds at once, ``pipeline.stash_counts``: the first partition holds N_m,
  the last one) times the per-layer buffers measured by the stage
  (``hp_stage_layer_bytes``) plus an upper bound of the stage-level buffers,
  plus its share of the weight state (the VW's N_m weight versions, the wave
  accumulator, the server copy and N_m gradient buffers) and the boundary
  activation / gradient buffers it hands to the next partition.
* The optimiser is an exact dynamic program over the valid cut points (a cut
  crosses a single tensor) instead of the paper's CPLEX model: best[j][b] =
  min over a of max(best[j-1][a], T_j(a, b)) subject to M_j(a, b) <= cap_j.
  With ``search_order`` it also tries every distinct order of the GPU types.
"""
from __future__ import annotations

import itertools
import math
from dataclasses import dataclass, field

import torch

from .hetpipe import HP_RELU, Stage
from .pipeline import layer_shapes, param_count, stash_counts, valid_cuts


@dataclass
class LayerProfile:
    fwd_ms: list          # per layer: forward device time on the profiled GPU
    bwd_ms: list          # per layer: backward device time (weight gradient included)
    mem: list             # per layer: device bytes of one stash of the layer's buffers
    shared: int           # stage-level bytes of the whole model's stage (an upper bound per partition)
    params: list          # per layer: parameter count
    out_bytes: list       # per layer: bytes of its fp32 output (what a cut after it transfers)
    dtype: str = "fp32"
    stage_ms: float = 0.0  # stage-level device time per step (bf16 weight copies)
    # per layer: the layer it reads (-1: model input), and the value buffer a
    # ReLU needs of its own when a cut separates it from the producer it is
    # fused into (its value otherwise aliases the producer's)
    inputs: list = field(default_factory=list)
    relu_value: list = field(default_factory=list)

    @property
    def n(self):
        return len(self.fwd_ms)


@dataclass
class GPUSpec:
    name: str
    speed: float = 1.0                 # throughput relative to the profiled GPU
    mem_bytes: float = math.inf


@dataclass
class PartitionPlan:
    cuts: list                         # layer indices after which the model is cut
    parts: list = field(default_factory=list)   # (first, last, gpu name, ms, bytes, stashes)
    bottleneck_ms: float = math.inf
    gpus: list = field(default_factory=list)


def profile(layers, batch, H, W, C, dtype="fp32", steps=3, warmup=1, seed=0, device="cuda"):
    """Per-layer device time and memory of the whole model as one stage on the
    current GPU: ``warmup`` untimed and ``steps`` timed forward+backward
    passes on seeded N(0, 1) inputs and N(0, 0.05) weights."""
    st = Stage(layers, batch, H, W, C, dtype=dtype)
    try:
        gen = torch.Generator(device="cpu").manual_seed(seed)
        dev = torch.device(device)
        w = (0.05 * torch.randn(st.P, generator=gen)).to(dev)
        x = torch.randn((batch, H, W, C), generator=gen).to(dev)
        grad = torch.empty(st.P, dtype=torch.float32, device=dev)
        oh, ow, oc = st.output_shape(-1)
        if st.has_loss:
            labels = torch.randint(0, oc, (batch,), generator=gen, dtype=torch.int32).to(dev)
            loss = torch.empty(1, dtype=torch.float32, device=dev)
            y = dy = None
        else:
            y = torch.empty((batch, oh, ow, oc), dtype=torch.float32, device=dev)
            dy = (1e-3 * torch.randn((batch, oh, ow, oc), generator=gen)).to(dev)

        def step():
            if st.has_loss:
                st.forward(w, x, None, labels, loss)
                st.backward(w, None, None, grad)
            else:
                st.forward(w, x, y)
                st.backward(w, dy, None, grad)
        for _ in range(warmup):
            step()
        torch.cuda.synchronize(dev)
        st.read_layer_timing()
        st.set_timing(True)
        for _ in range(steps):
            step()
        f, b = st.read_layer_timing()
        st.set_timing(False)
        mem, shared = st.layer_bytes()
    finally:
        torch.cuda.synchronize()
        st.close()
    shapes = layer_shapes(layers, H, W, C)
    out_bytes = [4 * batch * h * w_ * c for (h, w_, c) in (shapes[i] for i in range(len(layers)))]
    inputs = [d.get("in0", i - 1) for i, d in enumerate(layers)]
    relu_value = [out_bytes[i] if d["kind"] == HP_RELU and inputs[i] >= 0 else 0
                  for i, d in enumerate(layers)]
    return LayerProfile(fwd_ms=[v / steps for v in f[:-1]], bwd_ms=[v / steps for v in b[:-1]],
                        mem=list(mem), shared=int(shared),
                        params=[param_count(d) for d in layers], out_bytes=out_bytes,
                        dtype=dtype, stage_ms=(f[-1] + b[-1]) / steps,
                        inputs=inputs, relu_value=relu_value)


def partition_time(prof: LayerProfile, a, b, gpu: GPUSpec, link_GBps=None):
    """Execution time (ms) of layers a..b on `gpu`: computation plus the
    transfers into the partition (activations at a, gradients at b)."""
    t = (sum(prof.fwd_ms[a:b + 1]) + sum(prof.bwd_ms[a:b + 1])) / gpu.speed
    if link_GBps:
        if a > 0:
            t += prof.out_bytes[a - 1] / (link_GBps * 1e6)
        if b < prof.n - 1:
            t += prof.out_bytes[b] / (link_GBps * 1e6)
    return t


def stage_bytes(prof: LayerProfile, a, b):
    """Upper bound of the device bytes of one stage object of layers a..b:
    their buffers as measured in the whole model, a value buffer for a ReLU
    cut off from its producer, the whole model's stage-level buffers (its
    workspaces and weight copies cover any part's) and, in bf16, the copy of
    the partition input."""
    n = sum(prof.mem[a:b + 1]) + prof.shared
    if prof.relu_value:
        n += sum(prof.relu_value[i] for i in range(a, b + 1) if prof.inputs[i] < a)
    if prof.dtype == "bf16" and a > 0:
        n += prof.out_bytes[a - 1] // 2
    return n


def partition_memory(prof: LayerProfile, a, b, stashes, n_m):
    """Device bytes of layers a..b as one partition holding `stashes`
    minibatches, with N_m weight versions in flight."""
    stage = stage_bytes(prof, a, b)
    p = sum(prof.params[a:b + 1])
    weights = 4 * p * (2 * n_m + 2)                     # versions, gradients, u~, w_g
    boundary = 2 * n_m * prof.out_bytes[b] if b < prof.n - 1 else 0
    return stashes * stage + weights + boundary


def _dp(prof, pts, gpus, stashes, n_m, link_GBps):
    k, m = len(gpus), len(pts)
    INF = math.inf
    best = [[INF] * m for _ in range(k + 1)]
    arg = [[-1] * m for _ in range(k + 1)]
    best[0][0] = 0.0
    for j in range(1, k + 1):
        g = gpus[j - 1]
        for bi in range(1, m):
            for ai in range(bi):
                if best[j - 1][ai] == INF:
                    continue
                a, b = pts[ai] + 1, pts[bi]
                if partition_memory(prof, a, b, stashes[j - 1], n_m) > g.mem_bytes:
                    continue
                v = max(best[j - 1][ai], partition_time(prof, a, b, g, link_GBps))
                if v < best[j][bi]:
                    best[j][bi] = v
                    arg[j][bi] = ai
    if best[k][m - 1] == INF:
        return None
    cuts, bi = [], m - 1
    for j in range(k, 0, -1):
        ai = arg[j][bi]
        if j > 1:
            cuts.append(pts[ai])
        bi = ai
    return best[k][m - 1], sorted(cuts)


def partition(layers, prof: LayerProfile, gpus, n_m, link_GBps=None, search_order=False,
              d_fwd=None, d_bwd=None):
    """The cuts minimising the largest partition time subject to every
    partition fitting its GPU (None if no assignment fits)."""
    k = len(gpus)
    pts = [-1] + valid_cuts(layers) + [len(layers) - 1]
    if k > len(pts) - 1:
        raise ValueError(f"{k} partitions need {k - 1} cuts; only {len(pts) - 2} are valid")
    stashes = stash_counts(k, n_m, d_fwd, d_bwd)
    orders = [list(gpus)]
    if search_order:
        seen, orders = set(), []
        for perm in itertools.permutations(range(k)):
            key = tuple((gpus[i].name, gpus[i].speed, gpus[i].mem_bytes) for i in perm)
            if key not in seen:
                seen.add(key)
                orders.append([gpus[i] for i in perm])
    best = None
    for order in orders:
        r = _dp(prof, pts, order, stashes, n_m, link_GBps)
        if r is not None and (best is None or r[0] < best[0] - 1e-12):
            best = (r[0], r[1], order)
    if best is None:
        return None
    bott, cuts, order = best
    bounds = [-1] + cuts + [len(layers) - 1]
    plan = PartitionPlan(cuts=cuts, bottleneck_ms=bott, gpus=[g.name for g in order])
    for j in range(k):
        a, b = bounds[j] + 1, bounds[j + 1]
        plan.parts.append((a, b, order[j].name,
                           partition_time(prof, a, b, order[j], link_GBps),
                           partition_memory(prof, a, b, stashes[j], n_m), stashes[j]))
    return plan

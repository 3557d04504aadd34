"""Writes the full-size golden samples of one minibatch step of the VGG-19
stage 1, the full VGG-19 and the ResNet-152 middle stage (with its input
gradient): tests/golden/fullsize_<workload>.json.

Calls only the oracle (oracle.nets, oracle.stage: plain loops, fp64
accumulation) on inputs from the seeded generator (seeded_inputs, the same
draws the GPU tests make): minibatch 1 of virtual worker 0, He-normal
weights, images N(0, 1), labels uniform, the middle stages' upstream gradient
N(0, 1e-3^2).  Nothing here reads a GPU result.

Each tensor is viewed as the matrix its contraction writes (activations
[batch*H*W][C], conv weights [K][R*S*C], FC weights [out][in], vectors
[1][n]) and cut into 64 x 64 blocks; one element is drawn from every block
(up to a cap per tensor, always keeping the blocks on the ragged last row and
column of blocks), so every tile a kernel computes -- the cut ones and the
edge ones included -- has its outputs represented.  The file keeps, per
tensor, its shape, the largest magnitude over the whole tensor (the floor of
the error metric), the flat indices and the oracle's values.

With --sens it runs the oracle again on weights perturbed by a relative 1e-6
(seeded normal factors 1 + 1e-6 xi; about the fp32 round-off of a 2000-term
reduction, sqrt(2304) 2^-24 = 2.9e-6), once per perturbation seed, and
stores per tensor how far the oracle's own sampled values move, the largest
over the seeds: normwise ("sens") and element by element in the metric of
the comparison, max |r1 - r0| / max(|r0|, 1e-2 max|r0|) ("sens_elem").  That
is how much any fp32 implementation may differ from the exact result through
ReLU masks that a perturbation of that size flips at pre-activations next to
zero (gradients) and through the conditioning of a deep stage (outputs); one
perturbation is a noisy sample of it, hence several seeds.

  python tests/golden/make_fullsize.py [--sens] [workload ...]   (OMP threads: all)
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import seeded_inputs as si              # noqa: E402
from oracle import nets as onets        # noqa: E402
from oracle import stage as ostage      # noqa: E402

SEED = 20052014
BATCH = 32
# name: (network, classes or None, upstream-gradient std or None, input gradient)
WORKLOADS = {
    "vgg19_s1": ("vgg19_s1", None, 1e-3, False),
    "vgg19": ("vgg19", 1000, None, False),
    "resnet152_mid": ("resnet152_mid", None, 1e-3, True),
}
BLOCK = 64
CAP_MATRIX = 1024     # samples per weight matrix
CAP_VECTOR = 256      # samples per bias / batch-norm parameter vector
CAP_ACT = 4096        # samples per activation-shaped tensor


def sample(rows, cols, cap, rng):
    """Flat indices of one element per BLOCK x BLOCK block of a rows x cols
    matrix (at most `cap`, the ragged last block row and column always in)."""
    br, bc = -(-rows // BLOCK), -(-cols // BLOCK)
    blocks = [(i, j) for i in range(br) for j in range(bc)]
    edge = [b for b in blocks if b[0] == br - 1 or b[1] == bc - 1]
    inner = [b for b in blocks if not (b[0] == br - 1 or b[1] == bc - 1)]
    if len(blocks) > cap:
        keep = max(0, cap - len(edge))
        pick = rng.choice(len(inner), size=min(keep, len(inner)), replace=False)
        blocks = sorted(edge + [inner[k] for k in pick])
    out = []
    for i, j in blocks:
        r0, c0 = i * BLOCK, j * BLOCK
        r = r0 + int(rng.integers(0, min(BLOCK, rows - r0)))
        c = c0 + int(rng.integers(0, min(BLOCK, cols - c0)))
        out.append(r * cols + c)
    return sorted(set(out) | {0, rows * cols - 1})


def entry(a, rows, cols, cap, rng):
    a = np.asarray(a, np.float64).reshape(-1)
    idx = sample(rows, cols, cap, rng)
    return {"shape": [rows, cols], "absmax": float(np.max(np.abs(a))),
            "idx": idx, "val": [float(a[k]) for k in idx]}


SENS_REL = 1e-6
SENS_SEEDS = 2


def inputs(name):
    netname, classes, dy_std, need_dx = WORKLOADS[name]
    net = onets.by_name(netname)
    segs = [("w" if nm == "w" else nm, int(np.prod(shape)), fan)
            for _, nm, shape, fan in net.param_segments()]
    w0 = si.initial_weights(segs, SEED)
    x = si.normal(si.stream_key(SEED, 0, 1, si.T_X), BATCH * net.H * net.W * net.C)
    x = x.reshape(BATCH, net.H, net.W, net.C)
    lab = dy = None
    if classes:
        lab = si.labels(si.stream_key(SEED, 0, 1, si.T_LABELS), BATCH, classes)
    else:
        shp = (BATCH,) + tuple(net.out_shape)
        dy = si.normal(si.stream_key(SEED, 0, 1, si.T_DY), int(np.prod(shp)), dy_std).reshape(shp)
    return net, w0, x, lab, dy


def sampled(r, t, key):
    """The oracle result's values at the stored indices of tensor `key`."""
    idx = np.asarray(t["idx"], np.int64)
    if key.startswith("grad:"):
        return np.asarray(r["grad"], np.float64)[t["offset"] + idx]
    if key == "dx":
        return np.asarray(r["dx"], np.float64).reshape(-1)[idx]
    return np.asarray(r["y"], np.float64).reshape(-1)[idx]


def sens(name):
    path = os.path.join(HERE, f"fullsize_{name}.json")
    out = json.load(open(path))
    netname, classes, dy_std, need_dx = WORKLOADS[name]
    net, w0, x, lab, dy = inputs(name)
    for t in out["tensors"].values():
        t["sens"] = t["sens_elem"] = 0.0
    t0 = time.time()
    for j in range(SENS_SEEDS):
        xi = si.normal(si.stream_key(SEED, 0, j, si.T_PROBE), len(w0)).astype(np.float64)
        w1 = w0.astype(np.float64) * (1.0 + SENS_REL * xi)
        r = ostage.step(net, w1, x, labels=lab, dy=dy, need_dx=need_dx)
        for key, t in out["tensors"].items():
            r0 = np.asarray(t["val"], np.float64)
            r1 = sampled(r, t, key)
            nw = float(np.linalg.norm(r1 - r0) / max(np.linalg.norm(r0), 1e-300))
            el = float(np.max(np.abs(r1 - r0) / np.maximum(np.abs(r0), 1e-2 * t["absmax"])))
            t["sens"] = max(t["sens"], nw)
            t["sens_elem"] = max(t["sens_elem"], el)
    dt = time.time() - t0
    out["sens_rel"] = SENS_REL
    out["sens_seeds"] = SENS_SEEDS
    out["sens_oracle_seconds"] = round(dt, 1)
    with open(path, "w") as f:
        json.dump(out, f, separators=(",", ":"))
    print(f"{name}: perturbed oracle {dt:.0f} s -> sensitivities in {path}", flush=True)


def make(name):
    netname, classes, dy_std, need_dx = WORKLOADS[name]
    net, w0, x, lab, dy = inputs(name)
    t0 = time.time()
    r = ostage.step(net, w0.astype(np.float64), x, labels=lab, dy=dy, need_dx=need_dx)
    dt = time.time() - t0
    rng = np.random.default_rng(4242)
    out = {"workload": name, "network": netname, "batch": BATCH, "seed": SEED,
           "minibatch": 1, "vw": 0, "need_dx": need_dx,
           "source": "oracle.stage.step (fp64 accumulation) on seeded_inputs draws",
           "oracle_seconds": round(dt, 1), "tensors": {}}
    T = out["tensors"]
    y = np.asarray(r["y"], np.float64)
    if classes:
        out["loss"] = float(r["loss"])
        T["logits"] = entry(y, BATCH, classes, CAP_ACT, rng)
    else:
        T["y"] = entry(y, y.size // y.shape[-1], y.shape[-1], CAP_ACT, rng)
    off = 0
    for i, nm, shape, _ in net.param_segments():
        n = int(np.prod(shape))
        g = r["grad"][off:off + n]
        key = f"grad:{i}:{nm}"
        if len(shape) == 1:
            T[key] = entry(g, 1, n, CAP_VECTOR, rng)
        else:
            T[key] = entry(g, shape[0], n // shape[0], CAP_MATRIX, rng)
        T[key]["offset"] = off
        off += n
    if need_dx:
        dx = np.asarray(r["dx"], np.float64)
        T["dx"] = entry(dx, dx.size // dx.shape[-1], dx.shape[-1], CAP_ACT, rng)
    path = os.path.join(HERE, f"fullsize_{name}.json")
    with open(path, "w") as f:
        json.dump(out, f, separators=(",", ":"))
    print(f"{name}: oracle {dt:.0f} s, {sum(len(t['idx']) for t in T.values())} samples "
          f"-> {path}", flush=True)


if __name__ == "__main__":
    args = [a for a in sys.argv[1:] if not a.startswith("--")]
    for nm in args or list(WORKLOADS):
        (sens if "--sens" in sys.argv else make)(nm)

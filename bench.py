#!/usr/bin/env python3
"""Stage-step throughput of the HetPipe hot path on one MI355X.

One step = one minibatch of one virtual worker through the whole hot path:
weight-version select (hp_wsp_weights), stage forward, stage backward, local
update + wave accumulation, and at every wave end the push and the gated pull
against the parameter server in device memory.  Inputs (a pool of seeded
minibatches) are resident in HBM before the timed region starts.

Default workload: the full VGG-19 as a single-stage virtual worker (16 3x3
convolutions, FC 25088 -> 4096 -> 4096 -> 1000, softmax cross-entropy), batch
32 of 224x224x3 fp32 images, four virtual workers with s_local = 3 and clock
bound D = 0 -- the largest of the five workloads.

Prints one JSON line: metric, value = images/s over K timed steps run exactly
as a user runs them, the roofline of the dominant kernel class (the
implicit-GEMM contractions) and of the WSP update kernels, both from HIP
events around every launch during K further steps of the same schedule, and
the CPU oracle baseline.
"""
import argparse
import dataclasses
import hashlib
import json
import statistics
import os
import re
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2516.6}     # MI355X dense MFMA peaks
HBM_PEAK_GBS = 8000.0
METRIC = "stage-step images/sec (fwd+bwd+WSP update); % of MFMA peak, HBM GB/s"


def contraction_flops(layers, batch, H, W, C, need_dx=False):
    """Algorithmic FLOPs (2 per multiply-add) of one stage step's conv / FC
    contractions: forward, weight gradient, and data gradient except for a
    layer that reads the stage input when the stage needs no input gradient
    (a first stage: the image needs none)."""
    from paper_2005_14038_amd.hetpipe import HP_CONV, HP_FC
    shape = {-1: (H, W, C)}
    total = 0
    for i, d in enumerate(layers):
        h, w, c = shape[d.get("in0", i - 1)]
        k = d["kind"]
        if k == HP_CONV:
            P = (h + 2 * d["pad"] - d["R"]) // d["stride"] + 1
            Q = (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1
            macs = batch * P * Q * d["K"] * d["R"] * d["S"] * c
            total += 2 * macs * (2 if d.get("in0", i - 1) < 0 and not need_dx else 3)
            shape[i] = (P, Q, d["K"])
        elif k == HP_FC:
            macs = batch * d["K"] * d["C"]
            total += 2 * macs * (2 if d.get("in0", i - 1) < 0 and not need_dx else 3)
            shape[i] = (1, 1, d["K"])
        elif k == 4:   # max-pool
            P = (h + 2 * d["pad"] - d["R"]) // d["stride"] + 1
            Q = (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1
            shape[i] = (P, Q, c)
        elif k == 7:   # global average pool
            shape[i] = (1, 1, c)
        else:
            shape[i] = (h, w, c)
    return total


LAYER_NAMES = {1: "conv", 2: "fc", 3: "relu", 4: "maxpool", 5: "batchnorm", 6: "add",
               7: "gap", 8: "softmax_ce"}


def layer_work(layers, batch, H, W, C, need_dx=False):
    """Per layer: output shape and the algorithmic FLOP and bytes of its forward
    and backward passes (every tensor read or written once per pass, 4 bytes an
    element; a layer reading the stage input computes no data gradient unless
    the stage hands one back)."""
    shape = {-1: (H, W, C)}
    rows = []
    for i, d in enumerate(layers):
        src = d.get("in0", i - 1)
        h, w, c = shape[src]
        k = d["kind"]
        n_in = batch * h * w * c
        f_flop = b_flop = 0
        if k in (1, 2):
            if k == 1:
                P = (h + 2 * d["pad"] - d["R"]) // d["stride"] + 1
                Q = (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1
                out, wts = (P, Q, d["K"]), d["K"] * d["R"] * d["S"] * c
            else:
                out, wts = (1, 1, d["K"]), d["K"] * d["C"]
            n_out = batch * out[0] * out[1] * out[2]
            macs = n_out * (wts // d["K"])
            dgrad = src >= 0 or need_dx
            f_flop, b_flop = 2 * macs, 2 * macs * (2 if dgrad else 1)
            f_el = n_in + wts + n_out
            b_el = (n_out + n_in + wts) * (2 if dgrad else 1)
        else:
            if k == 4:
                out = ((h + 2 * d["pad"] - d["R"]) // d["stride"] + 1,
                       (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1, c)
            elif k == 7:
                out = (1, 1, c)
            else:
                out = (h, w, c)
            n_out = batch * out[0] * out[1] * out[2]
            if k == 6:                   # add: two inputs, gradient to both
                f_el, b_el = 2 * n_in + n_out, n_out + 2 * n_in
            elif k in (3, 4, 5):         # backward also reads the forward input
                f_el, b_el = n_in + n_out, n_out + 2 * n_in
            else:
                f_el, b_el = n_in + n_out, n_out + n_in
        shape[i] = out
        rows.append({"layer": i, "op": LAYER_NAMES.get(k, str(k)), "out": list(out),
                     "fwd_flop": f_flop, "bwd_flop": b_flop,
                     "fwd_bytes": 4 * f_el, "bwd_bytes": 4 * b_el})
    return rows


def per_layer_rooflines(rows, fwd_ms, bwd_ms, steps, peak_tflops):
    """Achieved fraction of the bounding peak per layer and pass, beside the
    roofline-attainable fraction min(1, AI * 8 TB/s / MFMA peak) of a
    contraction (element-wise layers are bound by HBM: attainable 1)."""
    out = []
    for r, tf, tb in zip(rows, fwd_ms, bwd_ms):
        for ph, t, fl, by in (("fwd", tf, r["fwd_flop"], r["fwd_bytes"]),
                              ("bwd", tb, r["bwd_flop"], r["bwd_bytes"])):
            ms = t / steps
            if ms <= 0:
                continue                 # done inside another layer's kernels
            e = {"layer": r["layer"], "op": r["op"], "pass": ph, "out": r["out"],
                 "ms": round(ms, 4), "GB/s": round(by / (ms * 1e-3) / 1e9, 1)}
            if fl:
                ai = fl / by
                e.update({"bound": "mfma" if ai * HBM_PEAK_GBS * 1e9 >= peak_tflops * 1e12 else "hbm",
                          "TFLOP/s": round(fl / (ms * 1e-3) / 1e12, 2),
                          "frac": round(fl / (ms * 1e-3) / (peak_tflops * 1e12), 4),
                          "hbm_frac": round(by / (ms * 1e-3) / (HBM_PEAK_GBS * 1e9), 4),
                          "attainable": round(min(1.0, ai * HBM_PEAK_GBS * 1e9 / (peak_tflops * 1e12)), 4)})
            else:
                e.update({"bound": "hbm", "frac": round(by / (ms * 1e-3) / (HBM_PEAK_GBS * 1e9), 4),
                          "attainable": 1.0})
            out.append(e)
    return out


def kernel_code_hash(path=None):
    """Hash of the contraction kernels' code: igemm.hip with its comments and
    whitespace removed, so that a change to a comment keeps stored counter
    figures valid and a change to the code does not."""
    p = path or os.path.join(ROOT, "paper_2005_14038_amd", "csrc", "igemm.hip")
    src = open(p, encoding="utf-8").read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)     # block comments
    src = re.sub(r"//[^\n]*", " ", src)                  # line comments
    code = " ".join(src.split())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per step of the contraction kernels from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    p = os.path.join(ROOT, "profiles", f"igemm_{workload}_traffic.json")
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("igemm_code_sha256_16") != kernel_code_hash():
        return None
    return d.get("bytes_per_step")


# Algorithmic HBM bytes per parameter of each WSP update kernel (fp32):
#   local update starting a wave: read g, w_newest; write w_new, u~     16 B
#   other local updates:          read g, w_newest, u~; write w_new, u~  20 B
#   wave push:                    read w_g, u~; write w_g                12 B
#   pull:                         read w_g; write the ring slot           8 B
#   fused wave end that pulls:    read g, u~, w_g; write u~, w_g, slot   24 B
#   fused wave end, no pull:      read g, w_newest, u~, w_g;
#                                 write w_new, u~, w_g                   28 B
# (a wave of one minibatch reads no u~: 4 B less for the fused wave ends)
UPDATE_BYTES_PER_PARAM = {"update_first": 16, "update": 20, "push": 12, "pull": 8,
                          "wave_end_pull": 24, "wave_end": 28}


def update_roofline(P, ms, launches):
    """HBM roofline of the WSP update kernels over the timed steps (device
    time from HIP events around every launch on the server's stream)."""
    per = {}
    tot_b = tot_ms = 0.0
    for k, b in UPDATE_BYTES_PER_PARAM.items():
        if launches[k]:
            nbytes = b * P * launches[k]
            per[k] = {"launches": launches[k], "avg_us": round(ms[k] * 1e3 / launches[k], 2),
                      "GB/s": round(nbytes / (ms[k] * 1e-3) / 1e9, 1)}
            tot_b += nbytes
            tot_ms += ms[k]
    if not tot_ms:
        return None
    achieved = tot_b / (tot_ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "params": P, "kernels": per}


def cpu_baseline(wl, layers, out_shape, images):
    """The oracle (plain C loops, fp64 accumulation, OpenMP) on the first
    `images` images of minibatch 1: forward + backward of the stage and the
    local update."""
    import numpy as np
    from oracle import nets as onets
    from oracle import stage as ostage
    from oracle import wsp as owsp
    from paper_2005_14038_amd import workloads
    onet = onets.by_name(wl.net, **wl.net_kw)
    w0 = workloads.initial_weights(wl, layers)
    x, lab, dy = workloads.inputs(wl, out_shape, 0, 1)
    x1 = x[:images]
    lab1 = lab[:images] if lab is not None else None
    dy1 = dy[:images] if dy is not None else None
    t0 = time.perf_counter()
    r = ostage.step(onet, w0.astype(np.float64), x1, labels=lab1, dy=dy1, bf16=(wl.dtype == "bf16"))
    sim = owsp.WSP(w0, 1, wl.s_local, 0, wl.lr, lambda n, q, w: r["grad"].astype(np.float32))
    sim._minibatch(0, 1)
    dt = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    return {"value": round(images / dt, 4), "unit": "images/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "sample": f"{images} image(s) of minibatch 1 ({wl.name}): oracle stage forward + "
                      f"backward + local update, {dt:.1f} s"}


def single_thread_baseline(args):
    """The oracle's sample on one thread and one image, timed in a child
    process (OpenMP fixes its thread count when the library loads)."""
    cmd = [sys.executable, os.path.abspath(__file__), "--cpu-baseline-only",
           "--workload", args.workload, "--cpu-images", "1"]
    if args.dtype is not None:
        cmd += ["--dtype", args.dtype]
    r = subprocess.run(cmd, env=dict(os.environ, OMP_NUM_THREADS="1"), capture_output=True,
                       text=True, timeout=1800)
    if r.returncode != 0:
        raise RuntimeError("single-thread oracle sample failed:\n" + r.stderr[-2000:])
    d = json.loads(r.stdout.strip().splitlines()[-1])
    return {"value": d["value"], "unit": d["unit"], "cores": d["cores"], "sample": d["sample"]}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def run_pipeline(args, wl, dev):
    """Throughput of one virtual worker run as a K-partition pipeline (K HIP
    streams, up to W = s_local + 1 minibatches in flight, cut at block
    boundaries by nominal work or by the partitioner on measured per-layer
    times and memory), against K = 1 in the same process.
    A step is one minibatch; the timed region covers whole waves after one
    warm-up wave, so pipeline fill and drain are included once."""
    import torch
    from paper_2005_14038_amd import workloads
    from paper_2005_14038_amd.pipeline import PipelinedVW, balanced_cuts, layer_costs
    b = wl.builder()
    layers = b.layers
    if not wl.has_loss:
        sys.exit("--pipeline needs a workload with a loss head (tiny, vgg19, resnet152)")
    w0 = torch.from_numpy(workloads.initial_weights(wl, layers)).to(dev)
    pool = {}

    def data(n, q):
        j = (q - 1) % args.pool
        if j not in pool:
            x, lab, _ = workloads.inputs(wl, None, 0, j + 1)
            pool[j] = (torch.from_numpy(x).to(dev), torch.from_numpy(lab).to(dev), None)
        return pool[j]

    W = wl.s_local + 1
    waves = max(1, -(-args.steps // W))
    result = {}
    plan_info = None
    for k in (1, args.pipeline):
        if k == 1:
            cuts = []
        elif args.partition == "measured":
            # the partitioner on this GPU's measured per-layer times and memory,
            # K partitions on K GPUs of this type (288 GB each)
            from paper_2005_14038_amd import partitioner as pt
            prof = pt.profile(layers, wl.batch, wl.H, wl.W, wl.C, dtype=wl.dtype, steps=3)
            plan = pt.partition(layers, prof, [pt.GPUSpec("MI355X", 1.0, 288e9)] * k, W)
            cuts = plan.cuts
            plan_info = {"predicted_bottleneck_ms": round(plan.bottleneck_ms, 4),
                         "parts": [{"layers": [a, b], "ms": round(ms, 4),
                                    "GB": round(mem / 1e9, 3), "stashes": nst}
                                   for a, b, _, ms, mem, nst in plan.parts]}
        else:
            cuts = balanced_cuts(layers, k, layer_costs(layers, wl.H, wl.W, wl.C, wl.batch))
        pv = PipelinedVW(layers, wl.batch, wl.H, wl.W, wl.C, w0, wl.s_local, wl.lr, data, cuts,
                         dtype=wl.dtype)
        pv.run(1)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pv.run(1 + waves)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        result[k] = (waves * W * wl.batch / dt, dt * 1e3 / (waves * W), cuts)
        pv.close()
        del pv
        torch.cuda.empty_cache()
    K = args.pipeline
    value, ms, cuts = result[K]
    out = {
        "metric": "pipelined virtual worker images/sec (fwd+bwd+WSP update, K partitions on "
                  "K streams of one GPU)",
        "value": round(value, 3), "unit": "images/s", "n_gpus": 1, "steps": waves * W,
        "warmup": W, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if wl.dtype == "fp32" else "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: batch {wl.batch} x {wl.H}x{wl.W}x{wl.C}, one virtual "
                               f"worker, N_m = {W}, {K} partitions cut after layers {cuts}",
                   "global_batch": wl.batch, "parallelism": f"pipeline {K} streams, one GPU"},
        "one_partition": {"value": round(result[1][0], 3), "ms_per_step": round(result[1][1], 4)},
        "partition": args.partition,
    }
    if plan_info:
        out["partition_plan"] = plan_info
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--workload", default="vgg19")
    ap.add_argument("--pool", type=int, default=2, help="distinct minibatches resident in HBM")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=2,
                    help="images of the oracle's bounded CPU sample")
    ap.add_argument("--cpu-single-thread", action="store_true",
                    help="also time the oracle on one thread, on one image (a child process "
                         "with OMP_NUM_THREADS=1, started before this one touches the GPU)")
    ap.add_argument("--cpu-baseline-only", action="store_true",
                    help="time only the oracle's bounded CPU sample, without the GPU, and "
                         "print it as one JSON line")
    ap.add_argument("--per-layer", action="store_true",
                    help="add each layer's forward and backward time, achieved fraction of its "
                         "bounding peak and roofline-attainable fraction (from the kernel-timing "
                         "pass)")
    ap.add_argument("--dtype", choices=["fp32", "bf16"], default=None,
                    help="contraction mode (default: the workload's); bf16 rounds the "
                         "contraction operands and keeps fp32 master weights")
    ap.add_argument("--partition", choices=["work", "measured"], default="work",
                    help="with --pipeline: cut by nominal work, or by the partitioner on "
                         "per-layer times and memory measured on this GPU")
    ap.add_argument("--pipeline", type=int, default=0, metavar="K",
                    help="run one virtual worker as a K-partition pipeline on K streams "
                         "(workloads with a loss head) instead of the stage step")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the multi-VW data-parallel layer is simulated on a "
              "single MI355X (virtual workers take turns on it); --gpus must be 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.cpu_baseline_only:
        from oracle import nets as onets
        from paper_2005_14038_amd import workloads
        wl = workloads.WORKLOADS[args.workload]
        if args.dtype is not None:
            wl = dataclasses.replace(wl, dtype=args.dtype)
        out_shape = onets.by_name(wl.net, **wl.net_kw).out_shape
        print(json.dumps(cpu_baseline(wl, wl.builder().layers, out_shape, args.cpu_images)),
              flush=True)
        return
    single = None
    if args.cpu_single_thread and not args.no_cpu_baseline and not args.pipeline:
        single = single_thread_baseline(args)

    import torch
    from paper_2005_14038_amd import workloads
    from paper_2005_14038_amd.driver import WSPDriver
    from paper_2005_14038_amd.hetpipe import Stage

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    wl = workloads.WORKLOADS[args.workload]
    if args.dtype is not None:
        wl = dataclasses.replace(wl, dtype=args.dtype)
    if args.pipeline:
        return run_pipeline(args, wl, dev)
    b = wl.builder()
    layers = b.layers
    st = Stage(layers, wl.batch, wl.H, wl.W, wl.C, dtype=wl.dtype)
    out_shape = st.output_shape(-1)
    w0 = torch.from_numpy(workloads.initial_weights(wl, layers)).to(dev)

    pool = {}
    for n in range(wl.N):
        for j in range(args.pool):
            x, lab, dy = workloads.inputs(wl, out_shape, n, j + 1)
            pool[(n, j)] = tuple(torch.from_numpy(a).to(dev) if a is not None else None
                                 for a in (x, lab, dy))

    def data(n, q):
        return pool[(n, (q - 1) % args.pool)]

    drv = WSPDriver(st, w0, wl.N, wl.s_local, wl.D, wl.lr, data, periods=wl.periods,
                    need_dx=wl.need_dx)
    order = []

    def next_vw():
        cand = [n for n in range(wl.N) if not drv.blocked[n]]
        return min(cand, key=lambda m: (drv.t[m], m))

    for _ in range(args.warmup):
        drv.minibatch(next_vw())
    torch.cuda.synchronize()

    # timed region: K steps exactly as a user runs them (no per-kernel
    # instrumentation; one event between steps gives the per-wave repeats)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        n = next_vw()
        order.append(n)
        drv.minibatch(n)
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = evs[0].elapsed_time(evs[-1])
    W = wl.s_local + 1
    wave_rates = [wl.batch * W / (evs[i].elapsed_time(evs[i + W]) * 1e-3)
                  for i in range(0, args.steps - W + 1, W)]

    # kernel-timing pass: K more steps of the same schedule with HIP events
    # recorded around every launch on the stream it is issued to (the library's
    # stage and server timers); the per-kernel-class device times give the
    # rooflines.  The events themselves cost a few microseconds per launch,
    # which is why the throughput above is measured without them.
    st.read_timing()                      # discard
    drv.ps.read_timing()
    st.set_timing(True)
    drv.ps.set_timing(True)
    for _ in range(args.steps):
        drv.minibatch(next_vw())
    torch.cuda.synchronize()
    ms, launches = st.read_timing()
    if args.per_layer:
        # the same records give either view: K more steps for the per-layer one
        for _ in range(args.steps):
            drv.minibatch(next_vw())
        layer_fwd_ms, layer_bwd_ms = st.read_layer_timing()
    st.set_timing(False)
    ums, ulaunch = drv.ps.read_timing()
    drv.ps.set_timing(False)

    ms_step = max(wall, ev_ms / 1e3) * 1e3 / args.steps
    value = wl.batch * args.steps / (max(wall, ev_ms / 1e3))
    flops_step = contraction_flops(layers, wl.batch, wl.H, wl.W, wl.C, need_dx=wl.need_dx)
    gemm_ms_step = ms["contraction"] / args.steps
    achieved = flops_step / (gemm_ms_step * 1e-3) / 1e12
    peak = PEAK_TFLOPS[wl.dtype]
    traffic = measured_traffic(args.workload)
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if wl.dtype == "fp32" else "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: batch {wl.batch} x {wl.H}x{wl.W}x{wl.C}, "
                               f"{wl.N} virtual worker(s), s_local {wl.s_local}, D {wl.D}"
                               + (", input gradient" if wl.need_dx else ""),
                   "global_batch": wl.batch, "parallelism": "single GPU, simulated VWs"},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": traffic,
                     "frac_of_bf16_peak": round(achieved / PEAK_TFLOPS["bf16"], 4),
                     "kernel": "implicit-GEMM conv/FC contractions (all launches of a step)",
                     "timing": f"HIP events around every launch, {args.steps} further steps",
                     "flop_per_step": flops_step, "ms_per_step": round(gemm_ms_step, 4),
                     "launches_per_step": launches["contraction"] / args.steps},
        "other_kernels_ms_per_step": round(ms["other"] / args.steps, 4),
        "repeats": ({"per": f"wave of {W} minibatches (HIP events between timed steps)",
                     "n": len(wave_rates), "unit": "images/s",
                     "median": round(statistics.median(wave_rates), 3),
                     "min": round(min(wave_rates), 3), "max": round(max(wave_rates), 3),
                     "rates": [round(v, 1) for v in wave_rates]}
                    if wave_rates else None),
        "wsp_update_roofline": update_roofline(st.P, ums, ulaunch),
    }
    if args.per_layer:
        out["per_layer"] = per_layer_rooflines(layer_work(layers, wl.batch, wl.H, wl.W, wl.C,
                                                          need_dx=wl.need_dx),
                                               layer_fwd_ms, layer_bwd_ms, args.steps, peak)
    drv.close()
    st.close()
    torch.cuda.synchronize()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, layers, out_shape, args.cpu_images)
        if single is not None:
            out["cpu_baseline"]["single_thread"] = single
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

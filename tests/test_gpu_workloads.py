"""The five workloads at their full sizes, in the launch configuration the
benchmark uses.

  * Tiny CNN: the complete WSP run (2 virtual workers x 3 waves) against the
    oracle -- event log bit-exact, every weight version, u~ and w_g within
    1e-3.
  * Every workload: the full WSP run through the C ABI with the real stage
    at full size; the event log (waves, clocks, pulls, blocks, version
    vectors) must equal the oracle's for the same schedule bit for bit, and
    every loss / gradient must be finite.
  * Every distinct conv / FC geometry of every workload, at batch 32 and full
    spatial size, as a one-layer stage (in the workload's precision, and the
    VGG-19 ones in bf16 too): outputs of forward, data gradient and weight
    gradient sampled once in every 64 x 64 block of each output matrix (so in
    every tile a kernel computes, whole or cut) against the oracle evaluated
    element by element.
  * VGG-19 stage 1 and full VGG-19 (no batch-norm, so images are
    independent): the complete forward output of image 0 of the batch
    against the oracle run on that image alone.
"""
import zlib

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import nets as onets
from oracle import ops as oops
from oracle import stage as ostage
from oracle import wsp as owsp
from paper_2005_14038_amd import hetpipe as hp
from paper_2005_14038_amd import workloads
from paper_2005_14038_amd.driver import WSPDriver

from gpu_common import BF16_TOL, FP32_TOL, assert_close, dev, rel_err  # noqa: F401

pytestmark = pytest.mark.gpu


def _device_data(wl, out_shape, devc):
    cache = {}

    def data(n, q):
        key = (n, q)
        if key not in cache:
            cache.clear()
            x, lab, dy = workloads.inputs(wl, out_shape, n, q)
            cache[key] = tuple(torch.from_numpy(a).to(devc) if a is not None else None
                               for a in (x, lab, dy))
        return cache[key]
    return data


def test_tiny_complete_wsp_run(dev):  # noqa: F811
    wl = workloads.WORKLOADS["tiny"]
    b = wl.builder()
    st = hp.Stage(b.layers, wl.batch, wl.H, wl.W, wl.C)
    out_shape = st.output_shape(-1)
    w0 = workloads.initial_weights(wl, b.layers)
    drv = WSPDriver(st, torch.from_numpy(w0).to(dev), wl.N, wl.s_local, wl.D, wl.lr,
                    _device_data(wl, out_shape, dev), periods=wl.periods)
    drv.run(wl.waves)
    torch.cuda.synchronize()

    onet = onets.tiny()

    def grad(n, q, w):
        x, lab, _ = workloads.inputs(wl, out_shape, n, q)
        return ostage.step(onet, w.astype(np.float64), x, labels=lab)["grad"].astype(np.float32)

    ref = owsp.WSP(w0, wl.N, wl.s_local, wl.D, wl.lr, grad, periods=wl.periods)
    ref.run(wl.waves)
    assert drv.events == ref.events
    assert_close(hp.read_vector(drv.ps.weights_ptr(), st.P), ref.wg, FP32_TOL, "w_g")
    for n in range(wl.N):
        ring, stride, ut = drv.vws[n].buffers()
        for s in range(wl.s_local + 1):
            assert_close(hp.read_vector(ring + 4 * s * stride, st.P), ref.ring[n][s], FP32_TOL,
                         f"VW {n} ring slot {s}")
        assert_close(hp.read_vector(ut, st.P), ref.ut[n], FP32_TOL, f"VW {n} u~")
    drv.close()
    st.close()


@pytest.mark.parametrize("name", ["tiny", "vgg19_s1", "vgg19", "resnet152_mid", "resnet152"])
def test_workload_event_log_and_finiteness(dev, name):  # noqa: F811
    wl = workloads.WORKLOADS[name]
    b = wl.builder()
    st = hp.Stage(b.layers, wl.batch, wl.H, wl.W, wl.C, dtype=wl.dtype)
    out_shape = st.output_shape(-1)
    w0 = workloads.initial_weights(wl, b.layers)
    assert st.P == len(w0) == onets.by_name(wl.net).param_count()
    losses = []

    def check(n, q, drv):
        g = drv.grad[:st.P]
        assert torch.isfinite(g).all().item(), (n, q)
        if wl.need_dx:
            assert torch.isfinite(drv.dx).all().item() and drv.dx.abs().max().item() > 0, (n, q)
        if wl.has_loss:
            losses.append(float(drv.loss.item()))

    drv = WSPDriver(st, torch.from_numpy(w0).to(dev), wl.N, wl.s_local, wl.D, wl.lr,
                    _device_data(wl, out_shape, dev), periods=wl.periods, on_minibatch=check,
                    need_dx=wl.need_dx)
    drv.run(wl.waves)
    torch.cuda.synchronize()
    # the bookkeeping does not depend on the gradient values: compare with the
    # oracle's simulation of the same schedule
    ref = owsp.WSP(np.zeros(1, np.float32), wl.N, wl.s_local, wl.D, wl.lr,
                   lambda n, q, w: np.zeros(1, np.float32), periods=wl.periods)
    ref.run(wl.waves)
    assert drv.events == ref.events
    if name == "resnet152":
        assert any(e[0] == "block" for e in drv.events)   # the clock bound did bind
    if wl.has_loss:
        assert all(np.isfinite(losses)) and min(losses) > 0
    drv.close()
    st.close()


# ---------------------------------------------------------------- layer shapes

def _geometries(name):
    """Distinct (conv or fc) layer geometries of a workload's network, with the
    input shape each one sees."""
    wl = workloads.WORKLOADS[name]
    net = onets.by_name(wl.net)
    seen = {}
    for i, nd in enumerate(net.nodes):
        if nd["op"] not in ("conv", "fc"):
            continue
        src = net._shape(nd["in"])
        if len(src) == 1:                      # FC or pooled vector input
            src = (1, 1, src[0])
        first = nd["in"] < 0
        if nd["op"] == "conv":
            key = ("conv", src, nd["K"], nd["R"], nd["stride"], nd["pad"], nd["bias"], first)
        else:
            key = ("fc", src, nd["OUT"], 1, 1, 0, nd["bias"], first)
        seen.setdefault(key, i)
    return [(name, k) for k in seen]


GEOMS = [g for n in ["vgg19_s1", "vgg19", "resnet152_mid", "resnet152"] for g in _geometries(n)]
_seen_ids = set()
GEOMS_UNIQ = []
# every geometry in its workload's precision, and the VGG-19 ones in bf16 too
# (the precision the bf16 contraction kernels run them in when asked)
for _dt_of in (lambda n: workloads.WORKLOADS[n].dtype,
               lambda n: "bf16" if n.startswith("vgg") else None):
    for _g in GEOMS:
        _dt = _dt_of(_g[0])
        _k = (_dt,) + _g[1]
        if _dt is not None and _k not in _seen_ids:
            _seen_ids.add(_k)
            GEOMS_UNIQ.append((_dt,) + _g)


def _gid(g):
    dt, name, (op, src, K, R, st, pad, bias, first) = g
    return f"{name}-{dt}-{op}{R}x{R}s{st}-{src[0]}x{src[1]}x{src[2]}-{K}"


def tile_samples(rows, cols, rng, block=64):
    """Flat indices of one element in every block x block block of a rows x
    cols matrix: every output tile a contraction kernel computes (whole or
    cut, ragged edge tiles included; every tile is a union of such blocks)
    has at least one of its outputs checked."""
    br, bc = -(-rows // block), -(-cols // block)
    r0 = np.repeat(np.arange(br) * block, bc)
    c0 = np.tile(np.arange(bc) * block, br)
    r = r0 + (rng.random(r0.size) * np.minimum(block, rows - r0)).astype(np.int64)
    c = c0 + (rng.random(c0.size) * np.minimum(block, cols - c0)).astype(np.int64)
    return np.unique(np.concatenate([r * cols + c, [0, rows * cols - 1]]))


@pytest.mark.parametrize("geom", GEOMS_UNIQ, ids=[_gid(g) for g in GEOMS_UNIQ])
def test_full_size_layer_sampled(dev, geom):  # noqa: F811
    dtype, name, key = geom
    seed = 1000 + zlib.crc32(_gid(geom).encode()) % 1000
    _layer_sampled(dev, dtype, workloads.WORKLOADS[name].batch, key, seed)


# bf16 geometries on the 256 x 128 direct-to-LDS tiles (at least 512 output
# columns, 16384 rows and a reduction of 2304): ragged last row of tiles and
# image borders; cut tiles (520 tiles: a partial last round); the data
# gradient on them; 25 taps (the per-row tap masks)
H16D_GEOMS = [
    (64, ("conv", (17, 17, 256), 512, 3, 1, 1, True, False)),
    (130, ("conv", (16, 16, 256), 512, 3, 1, 1, False, False)),
    (64, ("conv", (17, 17, 512), 256, 3, 1, 1, False, False)),
    (64, ("conv", (17, 17, 128), 512, 5, 1, 2, False, False)),
]


@pytest.mark.parametrize("bg", H16D_GEOMS, ids=[f"B{b}-" + _gid(("bf16", "t", g)).split("-", 2)[2]
                                                for b, g in H16D_GEOMS])
def test_direct_lds_tile_layer_sampled(dev, bg):  # noqa: F811
    B, key = bg
    _layer_sampled(dev, "bf16", B, key, 4000 + B + key[2] + key[3])


def _layer_sampled(dev, dtype, B, key, seed):
    """One conv or FC layer on the GPU (forward and backward), checked on one
    sampled output per 64 x 64 block of each output matrix against the
    oracle on the same (for bf16: bf16-rounded) operands."""
    op, src, K, R, stride, pad, bias, first = key
    H, W, C = src
    n = onets.Net("layer", H, W, C)
    if op == "conv":
        n.conv(-1, C, K, R, stride, pad, bias=bias)
    else:
        n.fc(-1, H * W * C, K, bias=bias)
    segs = [("w" if nm == "w" else nm, int(np.prod(s)), f) for _, nm, s, f in n.param_segments()]
    w = si.initial_weights(segs, seed)
    if bias:
        w[-K:] = si.normal(si.stream_key(seed, 0, 0, si.T_PROBE), K, 0.1)
    x = si.normal(si.stream_key(seed, 0, 1, si.T_X), B * H * W * C).reshape(B, H, W, C)
    out = n.out_shape
    dy = si.normal(si.stream_key(seed, 0, 1, si.T_DY), B * int(np.prod(out)), 1e-3)
    dy = dy.reshape((B,) + tuple(out))
    layers = [dict(kind=hp.HP_CONV, in0=-1, C=C, K=K, R=R, S=R, stride=stride, pad=pad,
                   bias=bias)] if op == "conv" else \
        [dict(kind=hp.HP_FC, in0=-1, C=H * W * C, K=K, bias=bias)]
    stg = hp.Stage(layers, B, H, W, C, dtype=dtype)
    wt = torch.from_numpy(w).to(dev)
    xt = torch.from_numpy(x).to(dev)
    y = torch.empty((B,) + tuple(out), dtype=torch.float32, device=dev)
    grad = torch.empty(stg.P, dtype=torch.float32, device=dev)
    dx = torch.empty_like(xt)
    stg.forward(wt, xt, y)
    stg.backward(wt, torch.from_numpy(dy).to(dev), dx, grad)
    torch.cuda.synchronize()
    yg, gg, dxg = y.cpu().numpy(), grad.cpu().numpy(), dx.cpu().numpy()
    stg.close()

    bf = dtype == "bf16"
    from oracle.bf16 import round_bf16
    rnd = round_bf16 if bf else (lambda a: np.asarray(a, np.float64))
    tol = BF16_TOL if bf else FP32_TOL
    rng = np.random.default_rng(5)
    if op == "conv":
        wk = w[:K * R * R * C].reshape(K, R, R, C)
        xo = x
        geo = (stride, pad)
    else:
        wk = w[:K * H * W * C].reshape(K, 1, 1, H * W * C)
        xo = x.reshape(B, 1, 1, H * W * C)
        geo = (1, 0)
    dyo = dy.reshape(B, 1, 1, K) if op == "fc" else dy
    xr, wr, dyr = rnd(xo), rnd(wk), rnd(dyo)
    bvec = w[-K:].astype(np.float64) if bias else None

    # forward [B*P*Q][K], weight gradient [K][R*S*C], data gradient [B*H*W][C]
    idx = tile_samples(yg.size // K, K, rng)
    ref = oops.conv_fwd_at(xr, wr, bvec, geo[0], geo[1], idx)
    _cmp(yg.reshape(-1)[idx], ref, tol, "forward")
    idx = tile_samples(K, wr[0].size, rng)
    ref = oops.conv_wgrad_at(xr, dyr, wr.shape[1], wr.shape[2], geo[0], geo[1], idx)
    _cmp(gg[:K * wr[0].size][idx], ref, tol, "weight gradient")
    if bias:
        # the whole bias gradient (in fp32 mode the weight-gradient kernel's
        # appended column)
        ref = dy.reshape(-1, K).astype(np.float64).sum(0)
        _cmp(gg[-K:], ref, tol, "bias gradient")
    cin = xo.shape[-1]
    idx = tile_samples(dxg.size // cin, cin, rng)
    ref = oops.conv_dgrad_at(dyr, wr, geo[0], geo[1], xo.shape[1], xo.shape[2], idx)
    _cmp(dxg.reshape(-1)[idx], ref, tol, "data gradient")


def _cmp(a, r, tol, what):
    e = rel_err(a, r)
    assert e <= tol, f"{what}: max relative error {e:.3e} > {tol:.1e} on sampled outputs"


@pytest.mark.parametrize("name", ["vgg19_s1", "vgg19"])
def test_full_size_forward_of_image0(dev, name):  # noqa: F811
    wl = workloads.WORKLOADS[name]
    b = wl.builder()
    st = hp.Stage(b.layers, wl.batch, wl.H, wl.W, wl.C)
    out_shape = st.output_shape(-1)
    w0 = workloads.initial_weights(wl, b.layers)
    x, lab, dy = workloads.inputs(wl, out_shape, 0, 1)
    y = torch.empty((wl.batch,) + (tuple(out_shape) if not wl.has_loss else (wl.classes,)),
                    dtype=torch.float32, device=dev)
    wt = torch.from_numpy(w0).to(dev)
    if wl.has_loss:
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        st.forward(wt, torch.from_numpy(x).to(dev), y, torch.from_numpy(lab).to(dev), loss)
    else:
        st.forward(wt, torch.from_numpy(x).to(dev), y)
    torch.cuda.synchronize()
    got = y[0].cpu().numpy()
    st.close()
    onet = onets.by_name(wl.net)
    vals, _, _ = ostage.forward(onet, w0.astype(np.float64), x[:1],
                                labels=lab[:1] if lab is not None else None)
    ref = vals[-2] if onet.has_loss else vals[-1]
    assert_close(got.reshape(-1), ref.reshape(-1), FP32_TOL, f"{name} image-0 output")

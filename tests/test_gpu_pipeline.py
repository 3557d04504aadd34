"""The pipelined virtual worker (k partitions on k HIP streams of one GPU, up
to N_m minibatches in flight, HetPipe Sec. 4) against the sequential virtual
worker and the oracle.

The pipeline only reorders work: every minibatch still reads the ring version
with the local updates 1..q-N_m, so weights, u~ and w_g must be bit-identical
to the sequential run of the same minibatches, and the event log (versions,
pushes, pulls) must equal the oracle's.
"""
import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import nets as onets
from oracle import stage as ostage
from oracle import wsp as owsp
from paper_2005_14038_amd import hetpipe as hp
from paper_2005_14038_amd import nets, workloads
from paper_2005_14038_amd import pipeline as pl
from paper_2005_14038_amd.driver import WSPDriver

from gpu_common import FP32_TOL, assert_close, dev  # noqa: F401

pytestmark = pytest.mark.gpu


def _data(builder, B, seed, classes, devc):
    H, W, C = builder.input_shape
    cache = {}

    def data(n, q):
        if (n, q) not in cache:
            x = si.normal(si.stream_key(seed, n, q, si.T_X), B * H * W * C).reshape(B, H, W, C)
            lab = si.labels(si.stream_key(seed, n, q, si.T_LABELS), B, classes)
            cache[(n, q)] = (torch.from_numpy(x).to(devc), torch.from_numpy(lab).to(devc), None)
        return cache[(n, q)]
    return data


def _split_events(ev):
    mb = sorted(e for e in ev if e[0] == "mb")
    rest = [e for e in ev if e[0] != "mb"]
    return mb, rest


def _run_both(builder, B, w0, s_local, lr, waves, k, dtype, data, devc):
    H, W, C = builder.input_shape
    cost = pl.layer_costs(builder.layers, H, W, C, B)
    cuts = pl.balanced_cuts(builder.layers, k, cost) if k > 1 else []
    wt = torch.from_numpy(w0).to(devc)
    pv = pl.PipelinedVW(builder.layers, B, H, W, C, wt, s_local, lr, data, cuts, dtype=dtype)
    pv.run(waves)
    torch.cuda.synchronize()
    st = hp.Stage(builder.layers, B, H, W, C, dtype=dtype)
    drv = WSPDriver(st, wt, 1, s_local, 0, lr, data)
    drv.run(waves)
    torch.cuda.synchronize()
    return pv, drv, st


def _assert_same_state(pv, drv, P, W):
    a = hp.read_vector(pv.ps.weights_ptr(), P)
    b = hp.read_vector(drv.ps.weights_ptr(), P)
    assert np.array_equal(a, b), "w_g differs from the sequential run"
    ra, sa, ua = pv.vw.buffers()
    rb, sb, ub = drv.vws[0].buffers()
    for s in range(W):
        assert np.array_equal(hp.read_vector(ra + 4 * s * sa, P), hp.read_vector(rb + 4 * s * sb, P)), s
    assert np.array_equal(hp.read_vector(ua, P), hp.read_vector(ub, P))


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_tiny_pipeline_equals_sequential_and_oracle(dev, k):  # noqa: F811
    wl = workloads.WORKLOADS["tiny"]
    b = nets.tiny()
    w0 = workloads.initial_weights(wl, b.layers)
    data = _data(b, wl.batch, wl.seed, wl.classes, dev)
    pv, drv, st = _run_both(b, wl.batch, w0, wl.s_local, wl.lr, 3, k, "fp32", data, dev)
    assert pv.k == k
    _assert_same_state(pv, drv, st.P, wl.s_local + 1)
    mb_p, rest_p = _split_events(pv.events)
    mb_s, rest_s = _split_events(drv.events)
    assert mb_p == mb_s and rest_p == rest_s

    # the oracle: the same WSP run with oracle gradients
    onet = onets.tiny()

    def grad(n, q, w):
        x, lab, _ = data(n, q)
        return ostage.step(onet, w.astype(np.float64), x.cpu().numpy(),
                           labels=lab.cpu().numpy())["grad"].astype(np.float32)

    ref = owsp.WSP(w0, 1, wl.s_local, 0, wl.lr, grad)
    ref.run(3)
    mb_o, rest_o = _split_events(ref.events)
    assert mb_p == mb_o and rest_p == rest_o
    assert_close(hp.read_vector(pv.ps.weights_ptr(), st.P), ref.wg, FP32_TOL, "w_g")
    pv.close()
    drv.close()
    st.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_small_resnet_pipeline_equals_sequential(dev, dtype):  # noqa: F811
    # stem + two groups of bottlenecks (a projection block each) + head, cut
    # at block boundaries into three partitions; batch-norm, residual fan-out
    # and (bf16) the operand copies all cross partitions
    b = nets.resnet152(H=32, W=32, classes=10, groups=[(16, 2, 1), (32, 2, 2)])
    B = 8
    segs = workloads.param_segments(b.layers)
    w0 = si.initial_weights(segs, 77)
    data = _data(b, B, 78, 10, dev)
    pv, drv, st = _run_both(b, B, w0, 2, 0.05, 2, 3, dtype, data, dev)
    _assert_same_state(pv, drv, st.P, 3)
    assert _split_events(pv.events) == _split_events(drv.events)
    pv.close()
    drv.close()
    st.close()


def test_window_full_is_an_error(dev):  # noqa: F811
    # W minibatches may be in flight; the (W+1)-th start is a protocol error
    w0 = torch.zeros(16, device=dev)
    ps = hp.ParameterServer(16, w0, 1, 0)
    vw = hp.VirtualWorker(ps, 0, 2)
    torch.cuda.synchronize()
    ptrs = [vw.weights() for _ in range(3)]
    assert len(set(ptrs)) == 3
    assert vw.state()["in_flight"] == 3
    with pytest.raises(hp.HPError):
        vw.weights()
    g = torch.ones(16, device=dev)
    vw.local_update(g, 0.5)                  # completes the oldest (minibatch 1)
    assert vw.state()["in_flight"] == 2 and vw.state()["p"] == 1
    assert vw.weights() == ptrs[0]           # minibatch 4 reuses minibatch 1's slot
    torch.cuda.synchronize()
    vw.close()
    ps.close()


def random_builder(seed):
    """A seeded small residual network with a loss head (convs with and
    without batch norm and ReLU, identity and projection shortcuts, fan-out of
    one value into two convs, max-pools)."""
    rng = np.random.default_rng(8000 + seed)
    H = int(rng.choice([8, 12]))
    b = nets.Builder(H, H, int(rng.choice([8, 16])))
    cur = -1
    for _ in range(int(rng.integers(2, 5))):
        C = b.shape[cur][2]
        kind = str(rng.choice(["plain", "res", "proj", "pool", "fan"]))
        if kind == "pool" and b.shape[cur][0] < 4:
            kind = "plain"
        if kind == "plain":
            R = int(rng.choice([1, 3]))
            a = b.conv(cur, int(rng.choice([8, 16, 24])), R, 1, R // 2,
                       bias=bool(rng.integers(0, 2)))
            if rng.random() < 0.7:
                a = b.bn(a)
            if rng.random() < 0.7:
                a = b.relu(a)
            cur = a
        elif kind in ("res", "proj"):
            K = C if kind == "res" else int(rng.choice([8, 16, 32]))
            mid = int(rng.choice([8, 16]))
            x = b.relu(b.bn(b.conv(cur, mid, 1)))
            x = b.relu(b.bn(b.conv(x, mid, 3, 1, 1)))
            x = b.bn(b.conv(x, K, 1))
            sc = cur if K == C and kind == "res" else b.bn(b.conv(cur, K, 1))
            cur = b.relu(b.add(x, sc) if rng.random() < 0.5 else b.add(sc, x))
        elif kind == "pool":
            cur = b.maxpool(cur, 2, 2)
        else:
            K = int(rng.choice([8, 16]))
            cur = b.relu(b.add(b.bn(b.conv(cur, K, 3, 1, 1)), b.bn(b.conv(cur, K, 1))))
    b.ce(b.fc(b.gap(cur), 10))
    return b


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("seed", range(8))
def test_random_graph_pipeline_equals_sequential(dev, seed, dtype):  # noqa: F811
    # random valid cuts of a random residual network: the pipelined VW must
    # reproduce the sequential one bit for bit
    b = random_builder(seed)
    H, W, C = b.input_shape
    rng = np.random.default_rng(9000 + seed)
    valid = pl.valid_cuts(b.layers)
    k = min(len(valid) + 1, int(rng.integers(2, 5)))
    cuts = sorted(int(c) for c in rng.choice(valid, size=k - 1, replace=False)) if k > 1 else []
    B = 4
    w0 = si.initial_weights(workloads.param_segments(b.layers), 100 + seed)
    data = _data(b, B, 101 + seed, 10, dev)
    wt = torch.from_numpy(w0).to(dev)
    pv = pl.PipelinedVW(b.layers, B, H, W, C, wt, 2, 0.05, data, cuts, dtype=dtype)
    pv.run(2)
    torch.cuda.synchronize()
    st = hp.Stage(b.layers, B, H, W, C, dtype=dtype)
    drv = WSPDriver(st, wt, 1, 2, 0, 0.05, data)
    drv.run(2)
    torch.cuda.synchronize()
    assert pv.k == k, (pv.k, k, cuts)
    _assert_same_state(pv, drv, st.P, 3)
    assert _split_events(pv.events) == _split_events(drv.events)
    pv.close()
    drv.close()
    st.close()

"""Degenerate shapes through the C ABI against the oracle: a single pixel, a
kernel larger than the image, a stride larger than the kernel (pixels no
output reads), one input or output channel, batch 1, batch-norm over a
single value per channel, and a pooling window that is mostly padding."""
import numpy as np
import pytest

from gpu_common import BF16_TOL, FP32_TOL, assert_close, dev  # noqa: F401
from stage_harness import make_inputs, oracle_weights, run_gpu, run_oracle, single

pytestmark = pytest.mark.gpu

CONV = [
    # N, H, W, C, K, R, stride, pad, bias
    (1, 1, 1, 5, 7, 3, 1, 1, True),      # one pixel: only the centre tap is inside
    (2, 2, 2, 8, 8, 3, 1, 1, False),     # kernel larger than the image
    (2, 5, 5, 4, 3, 1, 2, 0, True),      # stride 2 > kernel 1: odd pixels get no gradient
    (3, 6, 6, 1, 1, 3, 1, 1, True),      # one input and one output channel
    (1, 7, 7, 16, 32, 7, 2, 3, False),   # batch 1, stem-like 7x7 stride 2
    (2, 3, 3, 8, 16, 3, 3, 0, False),    # one output pixel
]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("case", CONV, ids=[str(c[:8]) for c in CONV])
def test_degenerate_conv(dev, case, dtype):  # noqa: F811
    N, H, W, C, K, R, st, pad, bias = case
    net = single(lambda n: n.conv(-1, C, K, R, st, pad, bias=bias), H, W, C)
    w = oracle_weights(net, 61)
    if bias:
        w[-K:] = np.linspace(-1, 1, K)
    x, _, dy = make_inputs(net, N, 62)
    g = run_gpu(net, N, w, x, None, dy, True, dtype)
    r = run_oracle(net, w, x, None, dy, True, bf16=(dtype == "bf16"))
    tol = FP32_TOL if dtype == "fp32" else BF16_TOL
    assert_close(g["y"], r["y"], tol, "forward")
    assert_close(g["grad"], r["grad"], tol, "weight gradient")
    assert_close(g["dx"], r["dx"], tol, "data gradient")
    if st > R:
        # inputs no output reads receive exactly zero gradient
        skipped = np.ones((H, W), bool)
        skipped[::st, ::st] = False
        assert np.all(g["dx"][:, skipped, :] == 0)


def test_fc_batch_one(dev):  # noqa: F811
    net = single(lambda n: n.fc(-1, 33, 9), 1, 1, 33)
    w = oracle_weights(net, 63)
    w[-9:] = np.linspace(-0.5, 0.5, 9)
    x, _, dy = make_inputs(net, 1, 64)
    g = run_gpu(net, 1, w, x, None, dy, True)
    r = run_oracle(net, w, x, None, dy, True)
    for key in ("y", "grad", "dx"):
        assert_close(g[key], r[key], FP32_TOL, key)


def test_batchnorm_over_one_value(dev):  # noqa: F811
    # batch 1, one pixel: every channel's mean is its value and its variance
    # is 0, so y = beta and the data gradient vanishes
    C = 16
    net = single(lambda n: n.bn(-1, C), 1, 1, C)
    w = oracle_weights(net, 65, scale_bn=True)
    x, _, dy = make_inputs(net, 1, 66)
    g = run_gpu(net, 1, w, x, None, dy, True)
    r = run_oracle(net, w, x, None, dy, True)
    assert_close(g["y"], r["y"], FP32_TOL, "forward")
    np.testing.assert_allclose(g["y"].reshape(-1), w[C:2 * C], rtol=0, atol=1e-6)
    assert_close(g["grad"], r["grad"], FP32_TOL, "gamma/beta gradient")
    assert np.abs(g["dx"]).max() <= 1e-6


def test_pool_window_mostly_padding(dev):  # noqa: F811
    net = single(lambda n: n.maxpool(-1, 3, 2, 1), 1, 1, 6)
    x, _, dy = make_inputs(net, 2, 67)
    g = run_gpu(net, 2, np.zeros(0, np.float32), x, None, dy, True)
    r = run_oracle(net, np.zeros(0), x, None, dy, True)
    np.testing.assert_array_equal(g["y"], r["y"].astype(np.float32))
    np.testing.assert_array_equal(g["dx"], r["dx"].astype(np.float32))


def test_wave_of_one_with_a_pipeline(dev):  # noqa: F811
    # s_local = 0: one minibatch in flight, every minibatch is a wave
    import torch
    from paper_2005_14038_amd import nets, workloads
    from paper_2005_14038_amd import pipeline as pl
    from paper_2005_14038_amd import hetpipe as hp
    from paper_2005_14038_amd.driver import WSPDriver
    import seeded_inputs as si
    b = nets.tiny()
    wl = workloads.WORKLOADS["tiny"]
    w0 = torch.from_numpy(workloads.initial_weights(wl, b.layers)).to(dev)

    def data(n, q):
        x = si.normal(si.stream_key(5, n, q, si.T_X), 4 * 16 * 16 * 3).reshape(4, 16, 16, 3)
        lab = si.labels(si.stream_key(5, n, q, si.T_LABELS), 4, 10)
        return torch.from_numpy(x).to(dev), torch.from_numpy(lab).to(dev), None
    pv = pl.PipelinedVW(b.layers, 4, 16, 16, 3, w0, 0, 0.01, data, [1, 2])
    pv.run(5)
    st = hp.Stage(b.layers, 4, 16, 16, 3)
    drv = WSPDriver(st, w0, 1, 0, 0, 0.01, data)
    drv.run(5)
    torch.cuda.synchronize()
    assert np.array_equal(hp.read_vector(pv.ps.weights_ptr(), st.P),
                          hp.read_vector(drv.ps.weights_ptr(), st.P))
    assert sorted(e for e in pv.events if e[0] == "mb") == \
        sorted(e for e in drv.events if e[0] == "mb")
    pv.close(); drv.close(); st.close()

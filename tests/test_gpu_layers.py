"""Per-operator parity of the HIP kernels against the oracle, through the C ABI.

Each case is a small stage holding the operator under test, run once forward
and backward on the GPU and in the oracle on the same seeded inputs.  Shapes
span several MFMA tiles with ragged tails, strides 1 and 2, paddings 0, 1 and
3, channel counts that are and are not multiples of 4, and split reductions.
"""
import numpy as np
import pytest

from gpu_common import BF16_TOL, FP32_TOL, assert_close, dev  # noqa: F401
from stage_harness import make_inputs, oracle_weights, run_gpu, run_oracle, single

pytestmark = pytest.mark.gpu

CONV = [
    # N, H, W, C, K, R, stride, pad, bias
    (2, 9, 9, 8, 16, 3, 1, 1, True),
    (2, 13, 11, 5, 7, 3, 2, 1, False),     # C % 4 != 0: scalar staging
    (3, 8, 8, 3, 8, 3, 1, 1, True),        # an image-input first layer
    (2, 10, 10, 16, 32, 1, 1, 0, False),
    (2, 9, 9, 12, 20, 1, 2, 0, False),     # projection shortcut shape
    (1, 15, 15, 3, 8, 7, 2, 3, False),     # ResNet stem shape
    (4, 20, 18, 64, 136, 3, 1, 1, True),   # several 128x128 tiles, ragged N
    (2, 30, 30, 32, 64, 3, 1, 1, True),    # 256x64 tile configuration
    (16, 4, 4, 256, 40, 3, 1, 1, False),   # long reduction, split-K in wgrad
    # bf16 on k-major operands (reduction channels a multiple of the k tile)
    (2, 15, 13, 64, 72, 3, 2, 1, False),   # strided, padded forward
    (2, 11, 9, 72, 128, 3, 1, 1, False),   # data gradient, 3x3 taps, ragged N
    (3, 7, 7, 64, 64, 1, 1, 0, False),     # 1x1 both ways, ragged M
    (8, 14, 14, 256, 256, 3, 1, 1, False), # split reduction both ways
    (4, 9, 7, 64, 128, 1, 1, 0, False),    # weight gradient on the 128x64 tile (N = 64)
    (2, 15, 13, 32, 64, 3, 2, 1, False),   # stride-2 data gradient, 128x64 tile, odd sizes
    (2, 14, 14, 64, 128, 1, 2, 0, False),  # stride-2 1x1 projection shape
    (2, 16, 12, 128, 128, 3, 2, 1, False), # stride-2 data gradient, 128x128 tile
    # fp32 FAST instantiations (forward with C, stride-1 data gradient with K,
    # weight gradient with Q a multiple of 16) and their neighbours
    (2, 32, 32, 16, 32, 3, 1, 1, True),    # all three FAST; bias column in the weight gradient
    (3, 17, 48, 32, 48, 3, 1, 1, False),   # FAST weight gradient across images, ragged M
    (16, 16, 16, 64, 64, 3, 1, 1, False),  # FAST weight gradient cut into reduction chunks
    (2, 33, 35, 16, 24, 3, 2, 1, False),   # FAST forward, strided data and weight gradients
    (2, 12, 12, 20, 16, 3, 1, 1, False),   # C % 16 != 0 forward, FAST data gradient
    (2, 14, 14, 16, 32, 7, 1, 3, False),   # FAST 7 x 7 taps (the largest the tap stepping takes)
    (2, 12, 12, 16, 32, 5, 1, 2, True),    # FAST 5 x 5 taps
]


def conv_net(c):
    N, H, W, C, K, R, st, pad, bias = c
    return single(lambda n: n.conv(-1, C, K, R, st, pad, bias=bias), H, W, C), N


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("case", CONV, ids=[str(c[:8]) for c in CONV])
def test_conv(dev, case, dtype):  # noqa: F811
    net, B = conv_net(case)
    w = oracle_weights(net, 11)
    if case[-1]:
        w[-case[4]:] = np.linspace(-1, 1, case[4])      # non-zero bias
    x, _, dy = make_inputs(net, B, 12)
    g = run_gpu(net, B, w, x, None, dy, True, dtype)
    r = run_oracle(net, w, x, None, dy, True, bf16=(dtype == "bf16"))
    tol = FP32_TOL if dtype == "fp32" else BF16_TOL
    assert_close(g["y"], r["y"], tol, "forward")
    assert_close(g["grad"], r["grad"], tol, "weight gradient")
    assert_close(g["dx"], r["dx"], tol, "data gradient")


def random_conv(seed):
    """A seeded conv geometry: taps 1, 3 or 5, stride 1 or 2, any legal padding,
    channel counts on and off the vector and k-tile multiples, ragged maps;
    shrunk until the layer is at most 40 M multiply-adds."""
    rng = np.random.default_rng(4000 + seed)
    R = int(rng.choice([1, 3, 3, 5]))
    st = int(rng.choice([1, 1, 2]))
    pad = int(rng.integers(0, R // 2 + 1))
    C = int(rng.choice([3, 5, 8, 16, 24, 64, 72, 128]))
    K = int(rng.choice([8, 20, 64, 96, 136, 256]))
    H, W = int(rng.integers(R, 19)), int(rng.integers(R, 19))
    N = int(rng.integers(1, 5))
    bias = bool(rng.integers(0, 2))

    def macs():
        P = (H + 2 * pad - R) // st + 1
        Q = (W + 2 * pad - R) // st + 1
        return N * P * Q * K * C * R * R

    while macs() > 40e6 and (N > 1 or H > R or W > R):
        if N > 1:
            N -= 1
        else:
            H, W = max(R, H - 2), max(R, W - 2)
    return (N, H, W, C, K, R, st, pad, bias)


RANDOM_CONV = [random_conv(s) for s in range(40)]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("case", RANDOM_CONV, ids=[f"rnd{i}-{c[:8]}" for i, c in enumerate(RANDOM_CONV)])
def test_conv_random_geometry(dev, case, dtype):  # noqa: F811
    test_conv(dev, case, dtype)


# the last two: a 32-image fully connected weight gradient of 64 x 256 tiles
# that the fixed grid walks more than once (1024 tiles, 512 workgroups at most),
# and 33 images, one past the batch that kernel takes
FC = [(4, 1, 1, 37, 50), (32, 2, 3, 16, 96), (5, 3, 3, 64, 260), (32, 1, 1, 4096, 4096),
      (33, 1, 1, 256, 128)]


@pytest.mark.parametrize("case", FC)
def test_fc(dev, case):  # noqa: F811
    B, H, W, C, OUT = case
    net = single(lambda n: n.fc(-1, H * W * C, OUT), H, W, C)
    w = oracle_weights(net, 21)
    w[-OUT:] = np.linspace(-0.5, 0.5, OUT)
    x, _, dy = make_inputs(net, B, 22)
    g = run_gpu(net, B, w, x, None, dy, True)
    r = run_oracle(net, w, x, None, dy, True)
    assert_close(g["y"], r["y"], FP32_TOL, "forward")
    assert_close(g["grad"], r["grad"], FP32_TOL, "weight gradient")
    assert_close(g["dx"], r["dx"], FP32_TOL, "data gradient")


def random_fc(seed):
    """A seeded FC geometry: batch 1-32, an input flattened from a small map,
    output widths on and off the tile edges."""
    rng = np.random.default_rng(3000 + seed)
    return (int(rng.integers(1, 33)), int(rng.integers(1, 4)), int(rng.integers(1, 4)),
            int(rng.choice([1, 3, 16, 37, 64, 130])), int(rng.choice([1, 10, 64, 100, 257, 1000])))


RANDOM_FC = [random_fc(s) for s in range(12)]


@pytest.mark.parametrize("case", RANDOM_FC, ids=[f"rnd{i}-{c}" for i, c in enumerate(RANDOM_FC)])
def test_fc_random_geometry(dev, case):  # noqa: F811
    test_fc(dev, case)


POOL = [(2, 8, 8, 4, 2, 2, 0), (2, 9, 7, 6, 3, 2, 1), (1, 11, 11, 64, 3, 2, 1)]


@pytest.mark.parametrize("case", POOL)
def test_maxpool_and_unfused_relu(dev, case):  # noqa: F811
    B, H, W, C, R, st, pad = case

    def build(n):
        a = n.maxpool(-1, R, st, pad)
        n.relu(a)
    net = single(build, H, W, C)
    x, _, dy = make_inputs(net, B, 31)
    g = run_gpu(net, B, np.zeros(0, np.float32), x, None, dy, True)
    r = run_oracle(net, np.zeros(0), x, None, dy, True)
    # max-pool and ReLU select values: the forward is exact
    np.testing.assert_array_equal(g["y"], r["y"].astype(np.float32))
    if st >= R:
        # each input is in at most one window: its gradient is one dy value
        np.testing.assert_array_equal(g["dx"], r["dx"].astype(np.float32))
    else:
        # an input sums dy over the k <= ceil(R/st)^2 windows whose first
        # maximum it is; an fp32 sum of k terms in any order is within
        # (k-1) 2^-24 sum|g| of the exact sum, and the routing depends on x
        # alone, so the oracle on |dy| gives sum|g| per element
        k = (-(-R // st)) ** 2
        s_abs = run_oracle(net, np.zeros(0), x, None, np.abs(dy), True)["dx"]
        err = np.abs(g["dx"].astype(np.float64) - r["dx"])
        bound = (k - 1) * 2.0 ** -24 * s_abs * (1 + 1e-6)
        assert np.all(err <= bound), \
            f"data gradient: worst excess {np.max(err - bound):.3e} over the fp32 summation bound"


def random_pool(seed):
    """A seeded max-pool geometry: windows 2 or 3, strides 1-3 (overlapping,
    tiling and gapped windows), padding up to half the window, ragged maps,
    channel counts on and off the vector width."""
    rng = np.random.default_rng(5000 + seed)
    R = int(rng.choice([2, 3]))
    st = int(rng.integers(1, 4))
    pad = int(rng.integers(0, R // 2 + 1))
    H, W = int(rng.integers(R, 21)), int(rng.integers(R, 21))
    if seed % 4 == 0:                     # windows that tile the map exactly
        st, pad = R, 0
        H, W = R * max(1, H // R), R * max(1, W // R)
    return (int(rng.integers(1, 5)), H, W, int(rng.choice([1, 3, 4, 8, 64, 130])), R, st, pad)


RANDOM_POOL = [random_pool(s) for s in range(24)]


@pytest.mark.parametrize("case", RANDOM_POOL, ids=[f"rnd{i}-{c}" for i, c in enumerate(RANDOM_POOL)])
def test_maxpool_random_geometry(dev, case):  # noqa: F811
    test_maxpool_and_unfused_relu(dev, case)


def test_maxpool_ties_route_to_first(dev):  # noqa: F811
    net = single(lambda n: n.maxpool(-1, 2, 2, 0), 4, 4, 2)
    x = np.zeros((1, 4, 4, 2), np.float32)
    dy = np.arange(1, 9, dtype=np.float32).reshape(1, 2, 2, 2)
    g = run_gpu(net, 1, np.zeros(0, np.float32), x, None, dy, True)
    r = run_oracle(net, np.zeros(0), x, None, dy, True)
    np.testing.assert_array_equal(g["dx"], r["dx"].astype(np.float32))


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("shape", [(4, 6, 6, 8), (2, 33, 33, 64), (32, 7, 7, 130)])
def test_batchnorm(dev, shape, relu):  # noqa: F811
    B, H, W, C = shape

    def build(n):
        a = n.bn(-1, C)
        if relu:
            n.relu(a)
    net = single(build, H, W, C)
    w = oracle_weights(net, 41, scale_bn=True)
    x, _, dy = make_inputs(net, B, 42)
    x = 0.5 + 2.0 * x                              # non-zero mean, non-unit variance
    g = run_gpu(net, B, w, x, None, dy, True)
    r = run_oracle(net, w, x, None, dy, True)
    assert_close(g["y"], r["y"], FP32_TOL, "forward")
    assert_close(g["grad"], r["grad"], FP32_TOL, "gamma/beta gradient")
    assert_close(g["dx"], r["dx"], FP32_TOL, "data gradient")


# conv -> batch norm -> ReLU: the batch norm takes its statistics from the
# conv's contraction (whole tiles in the epilogue, cut tiles in the cut-tile
# reduction); shapes with whole tiles only, with tiles cut 18 ways, and ragged
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("case", [(4, 32, 32, 64, 128, 1, 1, 0), (2, 14, 14, 256, 64, 3, 1, 1),
                                  (3, 9, 7, 64, 96, 3, 1, 1)])
def test_conv_batchnorm_statistics_from_the_contraction(dev, case, dtype):  # noqa: F811
    B, H, W, C, K, R, st, pad = case

    def build(n):
        n.relu(n.bn(n.conv(-1, C, K, R, st, pad), K))
    net = single(build, H, W, C)
    w = oracle_weights(net, 81, scale_bn=True)
    x, _, dy = make_inputs(net, B, 82)
    g = run_gpu(net, B, w, x, None, dy, True, dtype)
    r = run_oracle(net, w, x, None, dy, True, bf16=(dtype == "bf16"))
    tol = FP32_TOL if dtype == "fp32" else BF16_TOL
    assert_close(g["y"], r["y"], tol, "forward")
    assert_close(g["grad"], r["grad"], tol, "weight, gamma, beta gradients")
    assert_close(g["dx"], r["dx"], tol, "data gradient")


RANDOM_CONV_BN = [random_conv(100 + s)[:8] for s in range(16)]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("case", RANDOM_CONV_BN,
                         ids=[f"rnd{i}-{c}" for i, c in enumerate(RANDOM_CONV_BN)])
def test_conv_batchnorm_random_geometry(dev, case, dtype):  # noqa: F811
    test_conv_batchnorm_statistics_from_the_contraction(dev, case, dtype)


def test_residual_add_fans_out_to_the_input(dev):  # noqa: F811
    # y = relu(bn(conv(x)) + x): the input gradient sums the branch and the skip
    def build(n):
        a = n.bn(n.conv(-1, 16, 16, 3, 1, 1), 16)
        n.relu(n.addn(a, -1))
    net = single(build, 10, 10, 16)
    w = oracle_weights(net, 51, scale_bn=True)
    x, _, dy = make_inputs(net, 3, 52)
    g = run_gpu(net, 3, w, x, None, dy, True)
    r = run_oracle(net, w, x, None, dy, True)
    assert_close(g["y"], r["y"], FP32_TOL, "forward")
    assert_close(g["grad"], r["grad"], FP32_TOL, "weight gradient")
    assert_close(g["dx"], r["dx"], FP32_TOL, "data gradient")


@pytest.mark.parametrize("classes", [10, 1000])
def test_gap_fc_softmax_ce(dev, classes):  # noqa: F811
    def build(n):
        a = n.gap(-1)
        a = n.fc(a, 48, classes)
        n.ce(a, classes)
    net = single(build, 5, 5, 48)
    w = oracle_weights(net, 61)
    x, lab, _ = make_inputs(net, 8, 62)
    g = run_gpu(net, 8, w, x, lab, None, True)
    r = run_oracle(net, w, x, lab, None, True)
    assert abs(g["loss"] - r["loss"]) <= FP32_TOL * abs(r["loss"])
    assert_close(g["y"], r["y"], FP32_TOL, "logits")
    assert_close(g["grad"], r["grad"], FP32_TOL, "weight gradient")
    assert_close(g["dx"], r["dx"], FP32_TOL, "data gradient")

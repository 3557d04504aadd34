"""Pins of the oracle's stage operators against things other than itself.

Each test ties one oracle routine to a library routine, a closed form, an
identity or a hand-worked example, so that a dropped term, a wrong sign or
index, or a transposed operand in ``oracle.c`` fails at least one of them.
"""
import numpy as np
import pytest
import scipy.signal
import scipy.special
import torch

from oracle import ops
from oracle.bf16 import round_bf16

rng = np.random.default_rng(12345)


def _scipy_conv(x, w, b, stride, pad):
    """Multi-channel cross-correlation assembled from scipy.signal.correlate2d."""
    N, H, W, C = x.shape
    K, R, S, _ = w.shape
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    full = np.zeros((N, H + 2 * pad - R + 1, W + 2 * pad - S + 1, K))
    for n in range(N):
        for k in range(K):
            acc = 0.0
            for c in range(C):
                acc = acc + scipy.signal.correlate2d(xp[n, :, :, c], w[k, :, :, c], mode="valid")
            full[n, :, :, k] = acc
    y = full[:, ::stride, ::stride, :]
    if b is not None:
        y = y + b
    return y


CONV_CASES = [
    # N, H, W, C, K, R, stride, pad
    (2, 7, 6, 3, 4, 3, 1, 1),
    (1, 9, 9, 5, 3, 3, 2, 1),
    (2, 8, 8, 4, 6, 1, 1, 0),
    (1, 8, 7, 4, 6, 1, 2, 0),
    (1, 11, 11, 3, 2, 7, 2, 3),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_fwd_matches_scipy(case):
    N, H, W, C, K, R, st, pad = case
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((K, R, R, C))
    b = rng.standard_normal(K)
    y = ops.conv_fwd(x, w, b, st, pad)
    ref = _scipy_conv(x, w, b, st, pad)
    assert y.shape == ref.shape
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_conv_1x1_is_matmul():
    x = rng.standard_normal((3, 5, 4, 7))
    w = rng.standard_normal((6, 1, 1, 7))
    y = ops.conv_fwd(x, w, None, 1, 0)
    ref = x.reshape(-1, 7) @ w.reshape(6, 7).T
    np.testing.assert_allclose(y.reshape(-1, 6), ref, rtol=1e-12, atol=1e-12)


def test_conv_hand_example():
    # 1 image, 1 channel, 4x4 input 0..15, 3x3 all-ones kernel, pad 1:
    # every output is the sum of the in-range 3x3 neighbourhood.
    x = np.arange(16, dtype=np.float64).reshape(1, 4, 4, 1)
    w = np.ones((1, 3, 3, 1))
    y = ops.conv_fwd(x, w, None, 1, 1)[0, :, :, 0]
    expect = np.array([[10, 18, 24, 18],
                       [27, 45, 54, 39],
                       [51, 81, 90, 63],
                       [42, 66, 72, 50]], dtype=np.float64)
    np.testing.assert_array_equal(y, expect)
    # a centred delta kernel is the identity
    d = np.zeros((1, 3, 3, 1)); d[0, 1, 1, 0] = 1.0
    np.testing.assert_array_equal(ops.conv_fwd(x, d, None, 1, 1), x)
    # an off-centre delta shifts: w[0,0,0] picks x[p-1, q-1]
    d = np.zeros((1, 3, 3, 1)); d[0, 0, 0, 0] = 1.0
    y = ops.conv_fwd(x, d, None, 1, 1)[0, :, :, 0]
    assert y[0, 0] == 0 and y[1, 1] == x[0, 0, 0, 0] and y[3, 2] == x[0, 2, 1, 0]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_dgrad_adjoint(case):
    """<conv(x), dy> = <x, dgrad(dy)> for the bias-free convolution."""
    N, H, W, C, K, R, st, pad = case
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((K, R, R, C))
    y = ops.conv_fwd(x, w, None, st, pad)
    dy = rng.standard_normal(y.shape)
    dx = ops.conv_dgrad(dy, w, st, pad, H, W)
    assert dx.shape == x.shape
    lhs = np.sum(y * dy)
    rhs = np.sum(x * dx)
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_wgrad_adjoint(case):
    """<dw(x, dy), v> = <conv_v(x), dy> and db = sum of dy."""
    N, H, W, C, K, R, st, pad = case
    x = rng.standard_normal((N, H, W, C))
    v = rng.standard_normal((K, R, R, C))
    y = ops.conv_fwd(x, v, None, st, pad)
    dy = rng.standard_normal(y.shape)
    dw, db = ops.conv_wgrad(x, dy, R, R, st, pad, True)
    lhs = np.sum(dw * v)
    rhs = np.sum(y * dy)
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))
    np.testing.assert_allclose(db, dy.reshape(-1, K).sum(0), rtol=1e-12, atol=1e-12)


def test_conv_finite_differences():
    N, H, W, C, K, R, st, pad = 1, 5, 5, 2, 3, 3, 2, 1
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((K, R, R, C))
    b = rng.standard_normal(K)
    y = ops.conv_fwd(x, w, b, st, pad)
    dy = rng.standard_normal(y.shape)
    f = lambda xx, ww, bb: np.sum(ops.conv_fwd(xx, ww, bb, st, pad) * dy)
    dx = ops.conv_dgrad(dy, w, st, pad, H, W)
    dw, db = ops.conv_wgrad(x, dy, R, R, st, pad, True)
    h = 1e-6
    for idx in [(0, 0, 0, 0), (0, 2, 3, 1), (0, 4, 4, 0)]:
        e = np.zeros_like(x); e[idx] = h
        fd = (f(x + e, w, b) - f(x - e, w, b)) / (2 * h)
        assert abs(fd - dx[idx]) < 1e-6 * max(1, abs(fd))
    for idx in [(0, 0, 0, 0), (2, 1, 2, 1), (1, 2, 0, 1)]:
        e = np.zeros_like(w); e[idx] = h
        fd = (f(x, w + e, b) - f(x, w - e, b)) / (2 * h)
        assert abs(fd - dw[idx]) < 1e-6 * max(1, abs(fd))
    e = np.zeros_like(b); e[1] = h
    fd = (f(x, w, b + e) - f(x, w, b - e)) / (2 * h)
    assert abs(fd - db[1]) < 1e-6 * max(1, abs(fd))


def test_conv_sampled_entry_points_agree():
    N, H, W, C, K, R, st, pad = 2, 9, 8, 5, 4, 3, 2, 1
    x = rng.standard_normal((N, H, W, C))
    w = rng.standard_normal((K, R, R, C))
    b = rng.standard_normal(K)
    y = ops.conv_fwd(x, w, b, st, pad)
    idx = rng.choice(y.size, 20, replace=False)
    np.testing.assert_array_equal(ops.conv_fwd_at(x, w, b, st, pad, idx), y.reshape(-1)[idx])
    dy = rng.standard_normal(y.shape)
    dx = ops.conv_dgrad(dy, w, st, pad, H, W)
    idx = rng.choice(dx.size, 20, replace=False)
    np.testing.assert_array_equal(ops.conv_dgrad_at(dy, w, st, pad, H, W, idx), dx.reshape(-1)[idx])
    dw, _ = ops.conv_wgrad(x, dy, R, R, st, pad, False)
    idx = rng.choice(dw.size, 20, replace=False)
    np.testing.assert_array_equal(ops.conv_wgrad_at(x, dy, R, R, st, pad, idx), dw.reshape(-1)[idx])


def test_fc_matches_matmul():
    x = rng.standard_normal((4, 3, 2, 5))       # flattened (h, w, c) -> 30
    w = rng.standard_normal((7, 30))
    b = rng.standard_normal(7)
    x2 = x.reshape(4, 30)
    np.testing.assert_allclose(ops.fc_fwd(x, w, b), x2 @ w.T + b, rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal((4, 7))
    np.testing.assert_allclose(ops.fc_dgrad(dy, w), dy @ w, rtol=1e-12, atol=1e-12)
    dw, db = ops.fc_wgrad(x, dy, True)
    np.testing.assert_allclose(dw, dy.T @ x2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, dy.sum(0), rtol=1e-12, atol=1e-12)


def test_maxpool_matches_sliding_window():
    x = rng.standard_normal((2, 9, 7, 3))
    # 3x3 stride 2 pad 1 (the ResNet stem pool): pad with -inf, library max
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)), constant_values=-np.inf)
    win = np.lib.stride_tricks.sliding_window_view(xp, (3, 3), axis=(1, 2))
    ref = win.max(axis=(-1, -2))[:, ::2, ::2, :]
    np.testing.assert_array_equal(ops.maxpool_fwd(x, 3, 2, 1), ref)
    # 2x2 stride 2 on an even map = reshape + max
    x = rng.standard_normal((2, 8, 6, 4))
    ref = x.reshape(2, 4, 2, 3, 2, 4).max(axis=(2, 4))
    np.testing.assert_array_equal(ops.maxpool_fwd(x, 2, 2, 0), ref)


def test_maxpool_backward_routes_to_first_max():
    # all-equal windows: the gradient goes to the first tap in row-major order
    x = np.zeros((1, 4, 4, 1))
    dy = np.arange(1, 5, dtype=np.float64).reshape(1, 2, 2, 1)
    dx = ops.maxpool_bwd(x, dy, 2, 2, 0)[0, :, :, 0]
    expect = np.zeros((4, 4))
    expect[0, 0], expect[0, 2], expect[2, 0], expect[2, 2] = 1, 2, 3, 4
    np.testing.assert_array_equal(dx, expect)
    # overlapping 3x3/2 windows: a shared maximum collects both gradients
    x = np.zeros((1, 3, 3, 1)); x[0, 1, 1, 0] = 5.0
    dy = np.array([7.0, 11.0, 13.0, 17.0]).reshape(1, 2, 2, 1)
    dx = ops.maxpool_bwd(x, dy, 3, 2, 1)
    assert dx[0, 1, 1, 0] == 7 + 11 + 13 + 17 and np.count_nonzero(dx) == 1


def test_maxpool_finite_differences():
    x = rng.standard_normal((1, 6, 6, 2))
    y = ops.maxpool_fwd(x, 3, 2, 1)
    dy = rng.standard_normal(y.shape)
    dx = ops.maxpool_bwd(x, dy, 3, 2, 1)
    f = lambda xx: np.sum(ops.maxpool_fwd(xx, 3, 2, 1) * dy)
    h = 1e-7
    for idx in np.ndindex(x.shape):
        e = np.zeros_like(x); e[idx] = h
        fd = (f(x + e) - f(x - e)) / (2 * h)
        assert abs(fd - dx[idx]) < 1e-6


def test_bn_identities_and_gradients():
    x = 3.0 + 2.0 * rng.standard_normal((4, 5, 3, 6))
    C = 6
    gamma = np.ones(C); beta = np.zeros(C)
    eps = 1e-5
    y, mu, iv = ops.bn_fwd(x, gamma, beta, eps)
    xm = x.reshape(-1, C)
    np.testing.assert_allclose(mu, xm.mean(0), rtol=1e-12)
    var = xm.var(0)
    np.testing.assert_allclose(iv, 1 / np.sqrt(var + eps), rtol=1e-12)
    ym = y.reshape(-1, C)
    np.testing.assert_allclose(ym.mean(0), 0, atol=1e-12)
    np.testing.assert_allclose(ym.var(0), var / (var + eps), rtol=1e-10)
    # affine part
    gamma = rng.standard_normal(C); beta = rng.standard_normal(C)
    y2, _, _ = ops.bn_fwd(x, gamma, beta, eps)
    np.testing.assert_allclose(y2, gamma * y + beta, rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal(x.shape)
    dx, dg, dbt = ops.bn_bwd(x, dy, gamma, mu, iv)
    np.testing.assert_allclose(dbt, dy.reshape(-1, C).sum(0), rtol=1e-12)
    np.testing.assert_allclose(dg, (dy * y).reshape(-1, C).sum(0), rtol=1e-10, atol=1e-12)
    # per channel the input gradient sums to zero
    np.testing.assert_allclose(dx.reshape(-1, C).sum(0), 0, atol=1e-10)
    f = lambda xx, gg, bb: np.sum(ops.bn_fwd(xx, gg, bb, eps)[0] * dy)
    h = 1e-6
    for idx in [(0, 0, 0, 0), (3, 4, 2, 5), (1, 2, 1, 3)]:
        e = np.zeros_like(x); e[idx] = h
        fd = (f(x + e, gamma, beta) - f(x - e, gamma, beta)) / (2 * h)
        assert abs(fd - dx[idx]) < 1e-6 * max(1, abs(fd))
    for c in [0, 4]:
        e = np.zeros(C); e[c] = h
        fd = (f(x, gamma + e, beta) - f(x, gamma - e, beta)) / (2 * h)
        assert abs(fd - dg[c]) < 1e-6 * max(1, abs(fd))
        fd = (f(x, gamma, beta + e) - f(x, gamma, beta - e)) / (2 * h)
        assert abs(fd - dbt[c]) < 1e-6 * max(1, abs(fd))


def test_softmax_ce():
    z = rng.standard_normal((5, 7)) * 3
    lab = np.array([0, 6, 3, 3, 1], np.int32)
    loss, dz = ops.softmax_ce(z, lab)
    ref = np.mean(scipy.special.logsumexp(z, axis=1) - z[np.arange(5), lab])
    assert abs(loss - ref) < 1e-12
    np.testing.assert_allclose(dz.sum(1), 0, atol=1e-15)
    sm = scipy.special.softmax(z, axis=1)
    onehot = np.eye(7)[lab]
    np.testing.assert_allclose(dz, (sm - onehot) / 5, rtol=1e-12, atol=1e-15)
    h = 1e-6
    for idx in [(0, 0), (2, 3), (4, 6)]:
        e = np.zeros_like(z); e[idx] = h
        fd = (ops.softmax_ce(z + e, lab)[0] - ops.softmax_ce(z - e, lab)[0]) / (2 * h)
        assert abs(fd - dz[idx]) < 1e-8
    # large logits stay finite (max-subtracted)
    loss, dz = ops.softmax_ce(z + 1000.0, lab)
    assert np.isfinite(loss) and abs(loss - ref) < 1e-9


def test_relu_gap():
    x = np.array([-1.0, 0.0, 2.0, -0.0, 3.5])
    np.testing.assert_array_equal(ops.relu_fwd(x), [0, 0, 2, 0, 3.5])
    np.testing.assert_array_equal(ops.relu_bwd(x, np.ones(5)), [0, 0, 1, 0, 1])
    x = rng.standard_normal((2, 3, 4, 5))
    np.testing.assert_allclose(ops.gap_fwd(x), x.mean(axis=(1, 2)), rtol=1e-12)
    dy = rng.standard_normal((2, 5))
    dx = ops.gap_bwd(dy, 3, 4)
    assert np.allclose(np.sum(dx * x), np.sum(dy * ops.gap_fwd(x)))


def test_bf16_rounding():
    one = 1.0
    ulp = 2.0 ** -7
    vals = np.array([one, one + ulp / 2, one + 1.5 * ulp, one + ulp / 2 + 2 ** -20,
                     -3.0 - ulp, 65504.0, 1e-30, 0.0, -0.0])
    out = round_bf16(vals)
    assert out[0] == 1.0
    assert out[1] == 1.0                      # tie -> even mantissa (0)
    assert out[2] == one + 2 * ulp            # tie -> even mantissa (2)
    assert out[3] == one + ulp                # above the tie rounds up
    ref = torch.tensor(vals, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(out, ref)
    x = rng.standard_normal(10000).astype(np.float32) * 100
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x), ref)

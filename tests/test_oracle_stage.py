"""Pins of the oracle's layer-graph executor (forward + backward of a stage).

Finite differences of the whole stage in float64 tie the backward pass to the
forward pass for every node kind, including gradient fan-out at residual adds;
the parameter counts of the standard architectures pin the layer graphs.
"""
import numpy as np
import pytest

from oracle import nets, stage
from oracle.bf16 import round_bf16

rng = np.random.default_rng(777)


def test_parameter_counts_of_the_standard_networks():
    # VGG-19 and ResNet-152 parameter counts are the standard ones; the paper
    # quotes their fp32 sizes as 548 MB and 230 MB (Sec. 6.3).
    assert nets.tiny().param_count() == 11642
    assert nets.vgg19_s1().param_count() == 2325568
    v = nets.vgg19().param_count()
    r = nets.resnet152().param_count()
    assert v == 143667240 and r == 60192808
    assert round(v * 4 / 2 ** 20) == 548
    assert round(r * 4 / 2 ** 20) == 230
    assert nets.resnet152_mid().param_count() == 42953728
    assert nets.vgg19_s1().out_shape == (56, 56, 256)
    assert nets.resnet152_mid().out_shape == (14, 14, 1024)


def _mini_resnet():
    """Stem + one projected bottleneck (stride 2) + one identity bottleneck."""
    n = nets.Net("mini", 12, 12, 3)
    a = n.relu(n.bn(n.conv(-1, 3, 4, 3, 2, 1), 4))
    a = n.maxpool(a, 3, 2, 1)
    a, c = nets._bottleneck(n, a, 4, 2, 2, True)
    a, c = nets._bottleneck(n, a, c, 2, 1, False)
    a = n.gap(a)
    a = n.fc(a, c, 5)
    n.ce(a, 5)
    return n


def _mini_vgg_stage():
    n = nets.Net("minivgg", 8, 8, 3)
    a = n.relu(n.conv(-1, 3, 4, 3, 1, 1, bias=True))
    a = n.maxpool(a, 2, 2)
    a = n.relu(n.conv(a, 4, 5, 3, 1, 1, bias=True))
    return n


def _init(net, scale=0.5):
    return rng.standard_normal(net.param_count()) * scale


def _fd_check(net, params, x, labels, dy, need_dx, n_checks=12):
    def f(p, xx):
        vals, loss, _ = stage.forward(net, p, xx, labels)
        if net.has_loss:
            return loss
        return float(np.sum(vals[-1] * dy))

    out = stage.step(net, params, x, labels=labels, dy=dy, need_dx=need_dx)
    g = out["grad"]
    h = 1e-6
    idx = rng.choice(params.size, n_checks, replace=False)
    for i in idx:
        e = np.zeros_like(params); e[i] = h
        fd = (f(params + e, x) - f(params - e, x)) / (2 * h)
        assert abs(fd - g[i]) < 2e-6 * max(1.0, abs(fd)), (i, fd, g[i])
    if need_dx:
        for _ in range(6):
            j = tuple(rng.integers(0, s) for s in x.shape)
            e = np.zeros_like(x); e[j] = h
            fd = (f(params, x + e) - f(params, x - e)) / (2 * h)
            assert abs(fd - out["dx"][j]) < 2e-6 * max(1.0, abs(fd)), (j, fd)
    return out


def test_tiny_stage_finite_differences():
    net = nets.tiny(8, 8)
    p = _init(net, 0.3)
    x = rng.standard_normal((3, 8, 8, 3))
    lab = np.array([1, 9, 4], np.int32)
    _fd_check(net, p, x, lab, None, need_dx=True)


def test_resnet_block_finite_differences():
    net = _mini_resnet()
    p = _init(net, 0.5)
    # BN gammas/betas at a generic point
    x = rng.standard_normal((2, 12, 12, 3))
    lab = np.array([0, 3], np.int32)
    _fd_check(net, p, x, lab, None, need_dx=True, n_checks=20)


def test_stage_without_loss_head_finite_differences():
    net = _mini_vgg_stage()
    p = _init(net, 0.4)
    x = rng.standard_normal((2, 8, 8, 3))
    dy = rng.standard_normal((2,) + net.out_shape)
    _fd_check(net, p, x, None, dy, need_dx=True)


def test_residual_fanout_sums_both_paths():
    # y = relu(bn(conv(x))) + x has d<y,dy>/dx = (branch gradient) + dy
    n = nets.Net("fan", 5, 5, 2)
    a = n.bn(n.conv(-1, 2, 2, 1), 2)
    n.addn(a, -1)
    p = _init(n, 0.7)
    x = rng.standard_normal((2, 5, 5, 2))
    dy = rng.standard_normal((2, 5, 5, 2))
    out = stage.step(n, p, x, dy=dy, need_dx=True)
    # remove the skip path: gradient through the branch alone
    n2 = nets.Net("branch", 5, 5, 2)
    n2.bn(n2.conv(-1, 2, 2, 1), 2)
    out2 = stage.step(n2, p, x, dy=dy, need_dx=True)
    np.testing.assert_allclose(out["dx"], out2["dx"] + dy, rtol=1e-12, atol=1e-12)


def test_first_layer_dgrad_skipped_when_not_needed():
    net = _mini_vgg_stage()
    p = _init(net)
    x = rng.standard_normal((1, 8, 8, 3))
    dy = rng.standard_normal((1,) + net.out_shape)
    a = stage.step(net, p, x, dy=dy, need_dx=False)
    b = stage.step(net, p, x, dy=dy, need_dx=True)
    assert a["dx"] is None
    np.testing.assert_array_equal(a["grad"], b["grad"])


def test_bf16_mode_within_rounding_bound():
    """bf16 operands with exact accumulation differ from the fp64 result by at
    most sum |x||w| * 2 * 2^-8 (each operand carries relative error <= 2^-8)."""
    n = nets.Net("one", 6, 6, 4)
    n.conv(-1, 4, 3, 3, 1, 1, bias=False)
    p = _init(n, 1.0)
    x = rng.standard_normal((2, 6, 6, 4))
    y64 = stage.forward(n, p, x)[0][-1]
    y16 = stage.forward(n, p, x, bf16=True)[0][-1]
    w = p.reshape(3, 3, 3, 4)
    from oracle import ops
    bound = ops.conv_fwd(np.abs(x), np.abs(w), None, 1, 1) * (2 * 2.0 ** -8 + 2.0 ** -16)
    assert np.all(np.abs(y16 - y64) <= bound)
    assert np.any(y16 != y64)
    # the bf16 result is exactly the fp64 contraction of the rounded operands
    y_r = ops.conv_fwd(round_bf16(x), round_bf16(w), None, 1, 1)
    np.testing.assert_array_equal(y16, y_r)

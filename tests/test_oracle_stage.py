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


def _forward_macs_per_image(net):
    """Multiply-adds of one image's forward pass, summed over the conv and FC
    nodes from each node's own output shape (P x Q x K outputs, R x S x C
    multiply-adds each; an FC has IN x OUT)."""
    total = 0
    for i, nd in enumerate(net.nodes):
        if nd["op"] == "conv":
            P, Q, K = net.shapes[i]
            total += P * Q * K * nd["R"] * nd["S"] * nd["C"]
        elif nd["op"] == "fc":
            total += nd["IN"] * nd["OUT"]
    return total


def test_forward_multiply_adds_per_image_pin_the_graphs():
    """The forward multiply-adds per 224x224 image are fixed by the
    architectures: VGG-19 19.63 G (the commonly quoted 19.6 G), ResNet-152 with
    its stride on the 3x3 convolution 11.51 G (the original placement on the
    first 1x1, quoted as 11.3 G, gives 11.28 G), the VGG-19 stage 1 and the
    ResNet-152 middle stage their shares of those.  The parameter counts cannot
    tell the two ResNet placements apart; the multiply-adds can."""
    want = {"tiny": 360_448, "vgg19_s1": 11_184_832_512, "vgg19": 19_632_062_464,
            "resnet152_mid": 9_916_383_232, "resnet152": 11_513_626_624}
    for name, macs in want.items():
        assert _forward_macs_per_image(nets.by_name(name)) == macs, name
    # the stage shares add up: stage 1 is conv1_1 .. conv3_4 of VGG-19
    v = nets.vgg19()
    s1 = nets.vgg19_s1()
    assert [n for n in v.nodes[:len(s1.nodes)]] == s1.nodes
    # a ResNet-152 with the stride on the first 1x1 of each downsampling block
    # has the same parameters but fewer multiply-adds
    n = nets.Net("r152_v1", 224, 224, 3)
    a = n.relu(n.bn(n.conv(-1, 3, 64, 7, 2, 3), 64))
    a = n.maxpool(a, 3, 2, 1)
    c = 64
    for mid, blocks, stride in nets._RESNET152_GROUPS:
        for bi in range(blocks):
            s = stride if bi == 0 else 1
            out = 4 * mid
            b = n.relu(n.bn(n.conv(a, c, mid, 1, s), mid))
            b = n.relu(n.bn(n.conv(b, mid, mid, 3, 1, 1), mid))
            b = n.bn(n.conv(b, mid, out, 1), out)
            sc = n.bn(n.conv(a, c, out, 1, s), out) if bi == 0 else a
            a, c = n.relu(n.addn(b, sc)), out
    n.fc(n.gap(a), c, 1000)
    assert n.param_count() == nets.resnet152().param_count()
    assert _forward_macs_per_image(n) == 11_282_415_616
    assert _forward_macs_per_image(n) != _forward_macs_per_image(nets.resnet152())


def test_stage_boundaries_of_the_middle_and_first_stages():
    """VGG-19 stage 1 ends at conv3_4's ReLU (pool3 belongs to the next stage);
    the ResNet-152 middle stage is conv3_x + conv4_x: 8 + 36 bottlenecks, two
    of them with projection shortcuts, 56x56x256 in, 14x14x1024 out."""
    s1 = nets.vgg19_s1()
    assert sum(nd["op"] == "conv" for nd in s1.nodes) == 8
    assert sum(nd["op"] == "maxpool" for nd in s1.nodes) == 2
    assert s1.nodes[-1]["op"] == "relu" and s1.out_shape == (56, 56, 256)
    m = nets.resnet152_mid()
    adds = [nd for nd in m.nodes if nd["op"] == "add"]
    assert len(adds) == 44
    convs = [nd for nd in m.nodes if nd["op"] == "conv"]
    assert len(convs) == 3 * 44 + 2
    strided = [nd for nd in convs if nd["stride"] == 2]
    # one 3x3 and one projection per downsampling block
    assert sorted((nd["R"], nd["C"]) for nd in strided) == [(1, 256), (1, 512), (3, 128), (3, 256)]

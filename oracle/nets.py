"""Layer graphs of the oracle's workloads and their flat parameter layout.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A network is a list of nodes in topological order.  Node i's output is value i;
input index -1 is the stage input.  Node kinds:

  conv    C, K, R, S, stride, pad, bias   (weights [K][R][S][C], then bias[K])
  fc      IN, OUT, bias                   (weights [OUT][IN], then bias[OUT]);
          a 4-D input is flattened in (h, w, c) order
  relu, maxpool (R, stride, pad), bn (C, eps; gamma[C] then beta[C]),
  add (two inputs), gap (global average pool), ce (softmax cross-entropy head)

The flat parameter vector concatenates the parameters of the nodes in node
order.  The paper trains VGG-19 and ResNet-152 on ImageNet at batch 32 (Sec. 6,
methodology) and splits them into pipeline stages (Sec. 3); the stages used here
are the standard architectures cut at block boundaries:

  * tiny:       conv3x3 3->8 + ReLU, conv3x3 8->16 + ReLU, max-pool 2x2,
                FC 1024->10, softmax cross-entropy (16x16x3 input).
  * vgg19:      16 conv3x3 (pad 1, bias) + ReLU in blocks of 2, 2, 4, 4, 4 with
                64/128/256/512/512 channels, max-pool 2x2 after each block,
                FC 25088->4096->4096->1000 with ReLU between, softmax CE.
  * vgg19_s1:   conv1_1 .. conv3_4 + ReLU with the first two max-pools inside;
                the stage ends at conv3_4's ReLU (56x56x256 output).
  * resnet152:  stem conv7x7/2 pad 3 + BN + ReLU + max-pool 3x3/2 pad 1, then
                bottleneck blocks [3, 8, 36, 3] (1x1 -> 3x3 with the stride ->
                1x1 with 4x expansion, BN after each conv, ReLU after the first
                two and after the residual add, 1x1 projection + BN on the first
                block of each group), global average pool, FC 2048->1000, CE.
                Convolutions have no bias; BN eps = 1e-5.
  * resnet152_mid: groups conv3_x and conv4_x only (56x56x256 input,
                14x14x1024 output).
"""
from __future__ import annotations

BN_EPS = 1e-5


class Net:
    def __init__(self, name, H, W, C):
        self.name = name
        self.H, self.W, self.C = H, W, C
        self.nodes = []
        self.shapes = []          # per-node output shape (without batch)

    def _shape(self, i):
        return (self.H, self.W, self.C) if i < 0 else self.shapes[i]

    def add(self, node) -> int:
        kind = node["op"]
        s = self._shape(node["in"])
        if kind == "conv":
            H, W, C = s
            assert C == node["C"], (self.name, len(self.nodes), s, node)
            P = (H + 2 * node["pad"] - node["R"]) // node["stride"] + 1
            Q = (W + 2 * node["pad"] - node["S"]) // node["stride"] + 1
            out = (P, Q, node["K"])
        elif kind == "maxpool":
            H, W, C = s
            P = (H + 2 * node["pad"] - node["R"]) // node["stride"] + 1
            Q = (W + 2 * node["pad"] - node["R"]) // node["stride"] + 1
            out = (P, Q, C)
        elif kind == "fc":
            n = 1
            for d in s:
                n *= d
            assert n == node["IN"], (self.name, s, node)
            out = (node["OUT"],)
        elif kind == "gap":
            out = (s[-1],)
        elif kind == "add":
            assert self._shape(node["in2"]) == s
            out = s
        elif kind in ("relu", "bn"):
            out = s
        elif kind == "ce":
            out = ()
        else:
            raise ValueError(kind)
        self.nodes.append(node)
        self.shapes.append(out)
        return len(self.nodes) - 1

    # helpers -----------------------------------------------------------
    def conv(self, i, C, K, R, stride=1, pad=0, bias=False):
        return self.add(dict(op="conv", **{"in": i}, C=C, K=K, R=R, S=R,
                             stride=stride, pad=pad, bias=bias))

    def relu(self, i):
        return self.add(dict(op="relu", **{"in": i}))

    def bn(self, i, C):
        return self.add(dict(op="bn", **{"in": i}, C=C, eps=BN_EPS))

    def maxpool(self, i, R, stride, pad=0):
        return self.add(dict(op="maxpool", **{"in": i}, R=R, stride=stride, pad=pad))

    def fc(self, i, IN, OUT, bias=True):
        return self.add(dict(op="fc", **{"in": i}, IN=IN, OUT=OUT, bias=bias))

    def gap(self, i):
        return self.add(dict(op="gap", **{"in": i}))

    def addn(self, i, j):
        return self.add(dict(op="add", **{"in": i}, in2=j))

    def ce(self, i, classes):
        return self.add(dict(op="ce", **{"in": i}, classes=classes))

    # parameter layout --------------------------------------------------
    def param_segments(self):
        """List of (node index, name, shape, fan_in) in flat-vector order."""
        segs = []
        for i, n in enumerate(self.nodes):
            if n["op"] == "conv":
                segs.append((i, "w", (n["K"], n["R"], n["S"], n["C"]), n["R"] * n["S"] * n["C"]))
                if n["bias"]:
                    segs.append((i, "b", (n["K"],), None))
            elif n["op"] == "fc":
                segs.append((i, "w", (n["OUT"], n["IN"]), n["IN"]))
                if n["bias"]:
                    segs.append((i, "b", (n["OUT"],), None))
            elif n["op"] == "bn":
                segs.append((i, "gamma", (n["C"],), None))
                segs.append((i, "beta", (n["C"],), None))
        return segs

    def param_count(self) -> int:
        total = 0
        for _, _, shape, _ in self.param_segments():
            n = 1
            for d in shape:
                n *= d
            total += n
        return total

    @property
    def has_loss(self) -> bool:
        return bool(self.nodes) and self.nodes[-1]["op"] == "ce"

    @property
    def out_shape(self):
        return self.shapes[-1] if not self.has_loss else self.shapes[-2]


def tiny(H=16, W=16):
    n = Net("tiny", H, W, 3)
    a = n.relu(n.conv(-1, 3, 8, 3, 1, 1, bias=True))
    a = n.relu(n.conv(a, 8, 16, 3, 1, 1, bias=True))
    a = n.maxpool(a, 2, 2)
    a = n.fc(a, (H // 2) * (W // 2) * 16, 10)
    n.ce(a, 10)
    return n


_VGG19_CFG = [(64, 2), (128, 2), (256, 4), (512, 4), (512, 4)]


def vgg19(H=224, W=224, classes=1000, fc_width=4096):
    n = Net("vgg19", H, W, 3)
    a, c = -1, 3
    for k, reps in _VGG19_CFG:
        for _ in range(reps):
            a = n.relu(n.conv(a, c, k, 3, 1, 1, bias=True))
            c = k
        a = n.maxpool(a, 2, 2)
    flat = (H // 32) * (W // 32) * 512
    a = n.relu(n.fc(a, flat, fc_width))
    a = n.relu(n.fc(a, fc_width, fc_width))
    a = n.fc(a, fc_width, classes)
    n.ce(a, classes)
    return n


def vgg19_s1(H=224, W=224):
    n = Net("vgg19_s1", H, W, 3)
    a, c = -1, 3
    for bi, (k, reps) in enumerate(_VGG19_CFG[:3]):
        for _ in range(reps):
            a = n.relu(n.conv(a, c, k, 3, 1, 1, bias=True))
            c = k
        if bi < 2:
            a = n.maxpool(a, 2, 2)
    return n


def _bottleneck(n, a, cin, mid, stride, project):
    out = 4 * mid
    b = n.relu(n.bn(n.conv(a, cin, mid, 1), mid))
    b = n.relu(n.bn(n.conv(b, mid, mid, 3, stride, 1), mid))
    b = n.bn(n.conv(b, mid, out, 1), out)
    sc = a
    if project:
        sc = n.bn(n.conv(a, cin, out, 1, stride), out)
    return n.relu(n.addn(b, sc)), out


_RESNET152_GROUPS = [(64, 3, 1), (128, 8, 2), (256, 36, 2), (512, 3, 2)]


def _resnet_groups(n, a, cin, groups):
    for mid, blocks, stride in groups:
        for bi in range(blocks):
            a, cin = _bottleneck(n, a, cin, mid, stride if bi == 0 else 1, bi == 0)
    return a, cin


def resnet152(H=224, W=224, classes=1000, groups=None):
    n = Net("resnet152", H, W, 3)
    a = n.relu(n.bn(n.conv(-1, 3, 64, 7, 2, 3), 64))
    a = n.maxpool(a, 3, 2, 1)
    a, c = _resnet_groups(n, a, 64, groups or _RESNET152_GROUPS)
    a = n.gap(a)
    a = n.fc(a, c, classes)
    n.ce(a, classes)
    return n


def resnet152_mid(H=56, W=56, groups=None):
    n = Net("resnet152_mid", H, W, 256)
    _resnet_groups(n, -1, 256, groups or _RESNET152_GROUPS[1:3])
    return n


def by_name(name, **kw):
    return {"tiny": tiny, "vgg19": vgg19, "vgg19_s1": vgg19_s1,
            "resnet152": resnet152, "resnet152_mid": resnet152_mid}[name](**kw)

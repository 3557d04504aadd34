"""Layer lists of the stages this library runs (hp_layer dictionaries).

HetPipe trains VGG-19 and ResNet-152 with ImageNet-sized inputs at batch 32
(Sec. 6, methodology) and splits them into pipeline stages (Sec. 3).  The
lists below describe the standard architectures; each entry becomes one
``hp_layer`` (include/hetpipe.h):

  tiny           conv3x3 3->8 + ReLU, conv3x3 8->16 + ReLU, max-pool 2x2, FC -> 10, CE
  vgg19          16 conv3x3 (pad 1, bias) + ReLU in blocks 2/2/4/4/4 of 64/128/256/512/512
                 channels, max-pool 2x2 after each block, FC 25088->4096->4096->1000, CE
  vgg19_s1       conv1_1 .. conv3_4 (+ReLU) with pool1 and pool2: the first of four stages
  resnet152      stem 7x7/2 + BN + ReLU + max-pool 3x3/2, bottlenecks [3, 8, 36, 3]
                 (stride on the 3x3, projection shortcut on each group's first block),
                 global average pool, FC 2048->1000, CE; convolutions without bias
  resnet152_mid  groups conv3_x and conv4_x (56x56x256 in, 14x14x1024 out)
"""
from __future__ import annotations

from .hetpipe import (HP_ADD, HP_BN, HP_CONV, HP_FC, HP_GAP, HP_MAXPOOL, HP_RELU,
                      HP_SOFTMAX_CE)

BN_EPS = 1e-5


class Builder:
    def __init__(self, H, W, C):
        self.layers = []
        self.shape = {-1: (H, W, C)}
        self.input_shape = (H, W, C)

    def _push(self, d, out_shape):
        self.layers.append(d)
        i = len(self.layers) - 1
        self.shape[i] = out_shape
        return i

    def conv(self, x, K, R, stride=1, pad=0, bias=False):
        H, W, C = self.shape[x]
        P = (H + 2 * pad - R) // stride + 1
        Q = (W + 2 * pad - R) // stride + 1
        return self._push(dict(kind=HP_CONV, in0=x, C=C, K=K, R=R, S=R, stride=stride, pad=pad,
                               bias=bias), (P, Q, K))

    def relu(self, x):
        return self._push(dict(kind=HP_RELU, in0=x), self.shape[x])

    def bn(self, x):
        return self._push(dict(kind=HP_BN, in0=x, C=self.shape[x][2], eps=BN_EPS), self.shape[x])

    def maxpool(self, x, R, stride, pad=0):
        H, W, C = self.shape[x]
        P = (H + 2 * pad - R) // stride + 1
        Q = (W + 2 * pad - R) // stride + 1
        return self._push(dict(kind=HP_MAXPOOL, in0=x, R=R, S=R, stride=stride, pad=pad),
                          (P, Q, C))

    def fc(self, x, K, bias=True):
        H, W, C = self.shape[x]
        return self._push(dict(kind=HP_FC, in0=x, C=H * W * C, K=K, bias=bias), (1, 1, K))

    def add(self, a, b):
        assert self.shape[a] == self.shape[b]
        return self._push(dict(kind=HP_ADD, in0=a, in1=b), self.shape[a])

    def gap(self, x):
        return self._push(dict(kind=HP_GAP, in0=x), (1, 1, self.shape[x][2]))

    def ce(self, x):
        return self._push(dict(kind=HP_SOFTMAX_CE, in0=x, K=self.shape[x][2]), (1, 1, 0))

    def param_count(self):
        n = 0
        for d in self.layers:
            if d["kind"] in (HP_CONV, HP_FC):
                n += d["K"] * d.get("R", 1) * d.get("S", 1) * d["C"] if d["kind"] == HP_CONV \
                    else d["K"] * d["C"]
                n += d["K"] if d.get("bias") else 0
            elif d["kind"] == HP_BN:
                n += 2 * d["C"]
        return n


def tiny(H=16, W=16):
    b = Builder(H, W, 3)
    x = b.relu(b.conv(-1, 8, 3, 1, 1, bias=True))
    x = b.relu(b.conv(x, 16, 3, 1, 1, bias=True))
    x = b.maxpool(x, 2, 2)
    x = b.fc(x, 10)
    b.ce(x)
    return b


VGG19_BLOCKS = [(64, 2), (128, 2), (256, 4), (512, 4), (512, 4)]


def vgg19(H=224, W=224, classes=1000, width=4096):
    b = Builder(H, W, 3)
    x = -1
    for k, n in VGG19_BLOCKS:
        for _ in range(n):
            x = b.relu(b.conv(x, k, 3, 1, 1, bias=True))
        x = b.maxpool(x, 2, 2)
    x = b.relu(b.fc(x, width))
    x = b.relu(b.fc(x, width))
    x = b.fc(x, classes)
    b.ce(x)
    return b


def vgg19_s1(H=224, W=224):
    b = Builder(H, W, 3)
    x = -1
    for i, (k, n) in enumerate(VGG19_BLOCKS[:3]):
        for _ in range(n):
            x = b.relu(b.conv(x, k, 3, 1, 1, bias=True))
        if i < 2:
            x = b.maxpool(x, 2, 2)
    return b


def bottleneck(b, x, mid, stride, project):
    y = b.relu(b.bn(b.conv(x, mid, 1)))
    y = b.relu(b.bn(b.conv(y, mid, 3, stride, 1)))
    y = b.bn(b.conv(y, 4 * mid, 1))
    sc = b.bn(b.conv(x, 4 * mid, 1, stride)) if project else x
    return b.relu(b.add(y, sc))


RESNET152_GROUPS = [(64, 3, 1), (128, 8, 2), (256, 36, 2), (512, 3, 2)]


def resnet_groups(b, x, groups):
    for mid, blocks, stride in groups:
        for i in range(blocks):
            x = bottleneck(b, x, mid, stride if i == 0 else 1, i == 0)
    return x


def resnet152(H=224, W=224, classes=1000, groups=None):
    b = Builder(H, W, 3)
    x = b.relu(b.bn(b.conv(-1, 64, 7, 2, 3)))
    x = b.maxpool(x, 3, 2, 1)
    x = resnet_groups(b, x, groups or RESNET152_GROUPS)
    x = b.gap(x)
    x = b.fc(x, classes)
    b.ce(x)
    return b


def resnet152_mid(H=56, W=56, groups=None):
    b = Builder(H, W, 256)
    resnet_groups(b, -1, groups or RESNET152_GROUPS[1:3])
    return b


def by_name(name, **kw):
    return {"tiny": tiny, "vgg19": vgg19, "vgg19_s1": vgg19_s1, "resnet152": resnet152,
            "resnet152_mid": resnet152_mid}[name](**kw)

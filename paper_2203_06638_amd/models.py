"""Model descriptions for lpp_init: layer lists of the workloads' CNNs.

A model is a list of layer records (op, in0, in1, cin, cout, k, stride, pad,
bias, block) in execution order; layers that own parameters are numbered
into blocks 1..P, each block a run of successive parameter tensors (the
paper's partition of the model vector into blocks, Sec. 3).  Residual units
are the granularity of the cuts.

Also produced: the list of parameter tensor specs (kind, numel, fan_in) in
parameter order, for seeding initial parameters, and the output shape of
every layer.
"""
from __future__ import annotations

from .lpp import ADD, BN, CONCAT, CONV, GAP, LINEAR, MAXPOOL, RELU


class Model:
    def __init__(self, name, in_shape, n_classes):
        self.name = name
        self.in_shape = tuple(in_shape)
        self.n_classes = n_classes
        self.layers = []      # tuples for lpp.Layer, block filled by assign_blocks
        self.unit_of = []     # residual unit of each layer
        self.shapes = []      # (c, h, w) output of each layer
        self.specs = []       # (kind, numel, fan_in) in parameter order
        self._unit = 0
        self.P = 0

    # -- graph construction --------------------------------------------------
    def _shape(self, x):
        return self.in_shape if x < 0 else self.shapes[x]

    def _emit(self, rec, shape):
        self.layers.append(list(rec))
        self.unit_of.append(self._unit)
        self.shapes.append(shape)
        return len(self.layers) - 1

    def new_unit(self):
        self._unit += 1

    def conv(self, x, cout, k, stride=1, pad=None, bias=False):
        cin, h, w = self._shape(x)
        pad = k // 2 if pad is None else pad
        ho, wo = (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1
        self.specs.append(("conv_w", cout * cin * k * k, cin * k * k))
        if bias:
            self.specs.append(("bias", cout, cin * k * k))
        return self._emit((CONV, x, -1, cin, cout, k, stride, pad, int(bias), 0), (cout, ho, wo))

    def bn(self, x):
        c = self._shape(x)[0]
        self.specs += [("bn_gamma", c, 0), ("bn_beta", c, 0)]
        return self._emit((BN, x, -1, c, c, 0, 1, 0, 0, 0), self._shape(x))

    def relu(self, x):
        return self._emit((RELU, x, -1, 0, 0, 0, 1, 0, 0, 0), self._shape(x))

    def add(self, x, y):
        assert self._shape(x) == self._shape(y)
        return self._emit((ADD, x, y, 0, 0, 0, 1, 0, 0, 0), self._shape(x))

    def maxpool(self, x, k=3, stride=2, pad=1):
        c, h, w = self._shape(x)
        return self._emit((MAXPOOL, x, -1, 0, 0, k, stride, pad, 0, 0),
                          (c, (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1))

    def gap(self, x):
        return self._emit((GAP, x, -1, 0, 0, 0, 1, 0, 0, 0), (self._shape(x)[0], 1, 1))

    def concat(self, x, y):
        (cx, h, w), (cy, hy, wy) = self._shape(x), self._shape(y)
        assert (h, w) == (hy, wy)
        return self._emit((CONCAT, x, y, 0, 0, 0, 1, 0, 0, 0), (cx + cy, h, w))

    def linear(self, x, cout):
        cin = self._shape(x)[0]
        self.specs += [("linear_w", cout * cin, cin), ("bias", cout, cin)]
        return self._emit((LINEAR, x, -1, cin, cout, 0, 1, 0, 1, 0), (cout, 1, 1))

    # -- partitions ----------------------------------------------------------
    @property
    def n_units(self):
        return self._unit + 1

    def assign_blocks(self, unit_to_block):
        """Block of every residual unit; must be non-decreasing."""
        assert len(unit_to_block) == self.n_units
        assert list(unit_to_block) == sorted(unit_to_block)
        for rec, u in zip(self.layers, self.unit_of):
            rec[9] = unit_to_block[u] if rec[0] in (CONV, BN, LINEAR) else 0
        self.P = max(unit_to_block)
        return self

    @property
    def d(self):
        return sum(n for _, n, _ in self.specs)


# ---------------------------------------------------------------------------
# residual units

def post_act_unit(m, x, cout, stride, act=True):
    """conv3x3-BN-ReLU-conv3x3-BN (+ identity or 1x1/BN projection), ReLU.
    act=False leaves the ReLUs out."""
    m.new_unit()
    relu = m.relu if act else (lambda t: t)
    cin = m.shapes[x][0] if x >= 0 else m.in_shape[0]
    y = relu(m.bn(m.conv(x, cout, 3, stride)))
    y = m.bn(m.conv(y, cout, 3, 1))
    sc = m.bn(m.conv(x, cout, 1, stride, 0)) if (stride != 1 or cin != cout) else x
    return relu(m.add(y, sc))


def pre_act_unit(m, x, cout, stride, act=True):
    """BN-ReLU-conv3x3-BN-ReLU-conv3x3 (+ identity, or 1x1 conv of the
    pre-activated input when the shape changes).  act=False leaves the ReLUs
    out."""
    m.new_unit()
    relu = m.relu if act else (lambda t: t)
    cin = m.shapes[x][0]
    a = relu(m.bn(x))
    y = m.conv(a, cout, 3, stride)
    y = m.conv(relu(m.bn(y)), cout, 3, 1)
    sc = m.conv(a, cout, 1, stride, 0) if (stride != 1 or cin != cout) else x
    return m.add(y, sc)


def bottleneck_unit(m, x, mid, stride, act=True):
    """conv1x1 (mid) - BN - ReLU - conv3x3 (mid, stride) - BN - ReLU - conv1x1
    (4 mid) - BN (+ identity, or 1x1/stride conv + BN projection when the
    shape changes), ReLU.  act=False leaves the ReLUs out."""
    m.new_unit()
    relu = m.relu if act else (lambda t: t)
    cin = m.shapes[x][0]
    cout = 4 * mid
    y = relu(m.bn(m.conv(x, mid, 1, 1, 0)))
    y = relu(m.bn(m.conv(y, mid, 3, stride)))
    y = m.bn(m.conv(y, cout, 1, 1, 0))
    sc = m.bn(m.conv(x, cout, 1, stride, 0)) if (stride != 1 or cin != cout) else x
    return relu(m.add(y, sc))


# ---------------------------------------------------------------------------
# the workloads

def tiny_cnn(n_classes=10, hw=32):
    """conv3x3 3->8 + bias, ReLU, conv3x3 8->16 + bias, ReLU, pool, linear;
    P = 2: convs | linear."""
    m = Model("tiny_cnn", (3, hw, hw), n_classes)
    x = m.relu(m.conv(-1, 8, 3, bias=True))
    x = m.gap(m.relu(m.conv(x, 16, 3, bias=True)))
    m.new_unit()
    m.linear(x, n_classes)
    return m.assign_blocks([1, 2])


def resnet_cifar(depth=20, widths=(16, 32, 64), n_classes=10, hw=32, blocks=None, act=True):
    n = (depth - 2) // 6
    m = Model("resnet%d" % depth, (3, hw, hw), n_classes)
    x = m.bn(m.conv(-1, widths[0], 3))
    x = m.relu(x) if act else x
    for si, wdt in enumerate(widths):
        for u in range(n):
            x = post_act_unit(m, x, wdt, 2 if (si and not u) else 1, act)
    m.new_unit()
    m.linear(m.gap(x), n_classes)
    return m.assign_blocks(blocks or [1] * m.n_units)


def resnet20(n_classes=10, act=True):
    """ResNet-20, P = 4 blocks of residual units balanced by forward work:
    {stem, s1u1, s1u2} {s1u3, s2u1} {s2u2, s2u3, s3u1} {s3u2, s3u3, head}."""
    return resnet_cifar(20, (16, 32, 64), n_classes, blocks=[1, 1, 1, 2, 2, 3, 3, 3, 4, 4, 4], act=act)


def wide_resnet(depth=16, k=8, n_classes=100, hw=32, blocks=None, act=True):
    n = (depth - 4) // 6
    m = Model("wrn%d_%d" % (depth, k), (3, hw, hw), n_classes)
    x = m.conv(-1, 16, 3)
    for si, wdt in enumerate((16 * k, 32 * k, 64 * k)):
        for u in range(n):
            x = pre_act_unit(m, x, wdt, 2 if (si and not u) else 1, act)
    m.new_unit()
    x = m.bn(x)
    m.linear(m.gap(m.relu(x) if act else x), n_classes)
    return m.assign_blocks(blocks or [1] * m.n_units)


def wrn16_8(n_classes=100):
    """WRN-16-8, P = 4: {stem, s1u1, s1u2} {s2u1} {s2u2, s3u1} {s3u2, head}."""
    return wide_resnet(16, 8, n_classes, blocks=[1, 1, 1, 2, 3, 3, 4, 4])


def resnet_imagenet(units=(2, 2, 2, 2), widths=(64, 128, 256, 512), n_classes=1000, hw=224, blocks=None, act=True):
    m = Model("resnet%d" % (2 + 2 * sum(units)), (3, hw, hw), n_classes)
    x = m.bn(m.conv(-1, widths[0], 7, 2, 3))
    x = m.maxpool(m.relu(x) if act else x, 3, 2, 1)
    for si, (wdt, nu) in enumerate(zip(widths, units)):
        for u in range(nu):
            x = post_act_unit(m, x, wdt, 2 if (si and not u) else 1, act)
    m.new_unit()
    m.linear(m.gap(x), n_classes)
    return m.assign_blocks(blocks or [1] * m.n_units)


def resnet18(n_classes=1000):
    """ResNet-18, P = 4: {stem, s1u1} {s1u2, s2u1, s2u2} {s3u1, s3u2}
    {s4u1, s4u2, head}."""
    return resnet_imagenet(n_classes=n_classes, blocks=[1, 1, 2, 2, 2, 3, 3, 4, 4, 4])


def resnet_bottleneck(units=(3, 4, 6, 3), widths=(64, 128, 256, 512), n_classes=1000, hw=224, blocks=None,
                      act=True):
    """ImageNet ResNet with bottleneck units (ResNet-50 by default): 7x7/2
    stem, BN, ReLU, 3x3/2 max pool, four stages whose first unit strides on
    its 3x3 conv (stages 2-4), global pool, linear."""
    m = Model("resnet%d" % (2 + 3 * sum(units)), (3, hw, hw), n_classes)
    x = m.bn(m.conv(-1, widths[0], 7, 2, 3))
    x = m.maxpool(m.relu(x) if act else x, 3, 2, 1)
    for si, (wdt, nu) in enumerate(zip(widths, units)):
        for u in range(nu):
            x = bottleneck_unit(m, x, wdt, 2 if (si and not u) else 1, act)
    m.new_unit()
    m.linear(m.gap(x), n_classes)
    return m.assign_blocks(blocks or [1] * m.n_units)


def resnet50(n_classes=1000, act=True):
    """ResNet-50, P = 4 blocks of units cut nearest to the quartiles of the
    forward work: {stem, s1u1..s1u3, s2u1} {s2u2..s2u4, s3u1}
    {s3u2..s3u5} {s3u6, s4u1..s4u3, head}."""
    return resnet_bottleneck(n_classes=n_classes, act=act,
                             blocks=[1, 1, 1, 1, 1, 2, 2, 2, 2, 3, 3, 3, 3, 4, 4, 4, 4, 4])


# SqueezeNet v1.0's Fire modules: (squeeze, expand 1x1, expand 3x3) channels
SQUEEZENET_FIRES = ((16, 64, 64), (16, 64, 64), (32, 128, 128), (32, 128, 128),
                    (48, 192, 192), (48, 192, 192), (64, 256, 256), (64, 256, 256))


def fire_unit(m, x, s, e1, e3, act=True):
    """Fire module: squeeze 1x1 conv + ReLU, expand 1x1 and expand 3x3
    (padding 1) convs of the squeezed map, each + ReLU, concatenated (1x1
    channels first); every conv has a bias.  act=False leaves the ReLUs out."""
    m.new_unit()
    relu = m.relu if act else (lambda t: t)
    sq = relu(m.conv(x, s, 1, 1, 0, bias=True))
    a = relu(m.conv(sq, e1, 1, 1, 0, bias=True))
    b = relu(m.conv(sq, e3, 3, 1, 1, bias=True))
    return m.concat(a, b)


def squeezenet(n_classes=10, hw=32, stem=96, fires=SQUEEZENET_FIRES, pools_after=(2, 6), blocks=None, act=True):
    """SqueezeNet v1.0 on hw x hw inputs: 3x3 stem conv + ReLU, 3x3/2 max
    pool, the Fire modules (a 3x3/2 max pool after those listed in
    pools_after: fire4 and fire8), a 1x1 conv classifier + ReLU and a global
    average pool whose output are the logits."""
    m = Model("squeezenet", (3, hw, hw), n_classes)
    relu = m.relu if act else (lambda t: t)
    x = m.maxpool(relu(m.conv(-1, stem, 3, 1, 1, bias=True)), 3, 2, 1)
    for i, (s, e1, e3) in enumerate(fires):
        x = fire_unit(m, x, s, e1, e3, act)
        if i in pools_after:
            x = m.maxpool(x, 3, 2, 1)
    m.new_unit()
    m.gap(relu(m.conv(x, n_classes, 1, 1, 0, bias=True)))
    return m.assign_blocks(blocks or [1] * m.n_units)


def squeezenet_p4(n_classes=10, act=True):
    """SqueezeNet, P = 4 blocks of units cut nearest to the quartiles of the
    forward work: {stem, fire2, fire3} {fire4, fire5} {fire6, fire7}
    {fire8, fire9, classifier}."""
    return squeezenet(n_classes, act=act, blocks=[1, 1, 1, 2, 2, 3, 3, 4, 4, 4])

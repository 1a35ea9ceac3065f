"""Layer lists of the CNNs the oracle evaluates (test infrastructure).

Each model is an ordered list of layer records; a layer that owns parameters
holds the offset of its first parameter in the flat model vector x, so x is
the concatenation of the parameter tensors in model order (Sec. 3, "Block
partitions": a block is a run of successive tensors of that list).  Tensors
are flattened in their natural layout: conv W[cout][cin][k][k] then bias,
batch-norm gamma then beta, linear W[out][in] then bias.

Each layer also carries the index of the residual unit it belongs to and the
block (partition) that unit is assigned to.

Architectures (readings where the paper is silent are listed in the design
notes):
  tiny      conv3x3 3->8 +bias, ReLU, conv3x3 8->16 +bias, ReLU, global
            average pool, linear 16->10; blocks = convs | linear
  resnet    CIFAR ResNet-(6n+2): conv3x3 stem + BN + ReLU, three stages of n
            post-activation basic units, the first unit of stages 2 and 3
            with stride 2 and a 1x1 stride-2 conv + BN projection shortcut;
            global average pool, linear
  wrn       pre-activation Wide ResNet: conv3x3 stem, units BN-ReLU-conv
            (stride on the first conv) BN-ReLU-conv; 1x1 conv shortcut on the
            pre-activated input where the shape changes; final BN-ReLU, pool,
            linear
  resnet18  ImageNet ResNet-18: 7x7 stride-2 stem + BN + ReLU + 3x3 stride-2
            max pool, four stages of two basic units, projection shortcuts
  resnet50  ImageNet ResNet-50: the same stem, bottleneck units (3, 4, 6, 3)
  squeezenet  SqueezeNet v1.0's Fire modules (squeeze 1x1, expand 1x1 and
            3x3, outputs concatenated along channels) on 32x32 inputs: 3x3
            stem, max pools after the stem, fire4 and fire8, a 1x1 conv
            classifier with ReLU, global average pool (the logits); every
            conv has a bias, no batch norm
"""
from __future__ import annotations

CONV, BN, RELU, ADD, MAXPOOL, GAP, LINEAR, CONCAT = range(8)


class Net:
    def __init__(self, name, in_c, in_h, in_w, n_classes):
        self.name = name
        self.in_shape = (in_c, in_h, in_w)
        self.n_classes = n_classes
        self.layers = []        # dicts: op in0 in1 cin cout k stride pad bias poff unit block
        self.d = 0
        self.unit = 0
        self.specs = []         # (kind, numel, fan_in) for synth.init_params
        self.tensors = []       # (name, offset, numel)

    def _push(self, rec):
        self.layers.append(rec)
        return len(self.layers) - 1

    def conv(self, x, cin, cout, k, stride, pad, bias=False):
        n = cout * cin * k * k
        rec = dict(op=CONV, in0=x, in1=-1, cin=cin, cout=cout, k=k, stride=stride, pad=pad,
                   bias=int(bias), poff=self.d, unit=self.unit)
        idx = len(self.layers)
        self.tensors.append(("L%d.conv_w" % idx, self.d, n))
        self.specs.append(("conv_w", n, cin * k * k))
        self.d += n
        if bias:
            self.tensors.append(("L%d.conv_b" % idx, self.d, cout))
            self.specs.append(("bias", cout, cin * k * k))
            self.d += cout
        return self._push(rec)

    def bn(self, x, c):
        rec = dict(op=BN, in0=x, in1=-1, cin=c, cout=c, k=0, stride=1, pad=0, bias=0, poff=self.d, unit=self.unit)
        idx = len(self.layers)
        self.tensors.append(("L%d.bn_gamma" % idx, self.d, c))
        self.tensors.append(("L%d.bn_beta" % idx, self.d + c, c))
        self.specs += [("bn_gamma", c, 0), ("bn_beta", c, 0)]
        self.d += 2 * c
        return self._push(rec)

    def _plain(self, op, x, y=-1, k=0, stride=1, pad=0):
        return self._push(dict(op=op, in0=x, in1=y, cin=0, cout=0, k=k, stride=stride, pad=pad, bias=0,
                               poff=-1, unit=self.unit))

    def relu(self, x):
        return self._plain(RELU, x)

    def add(self, x, y):
        return self._plain(ADD, x, y)

    def maxpool(self, x, k=3, stride=2, pad=1):
        return self._plain(MAXPOOL, x, k=k, stride=stride, pad=pad)

    def gap(self, x):
        return self._plain(GAP, x)

    def concat(self, x, y):
        """Channels of x followed by channels of y (same spatial size)."""
        return self._plain(CONCAT, x, y)

    def linear(self, x, cin, cout):
        rec = dict(op=LINEAR, in0=x, in1=-1, cin=cin, cout=cout, k=0, stride=1, pad=0, bias=1,
                   poff=self.d, unit=self.unit)
        idx = len(self.layers)
        self.tensors.append(("L%d.linear_w" % idx, self.d, cout * cin))
        self.tensors.append(("L%d.linear_b" % idx, self.d + cout * cin, cout))
        self.specs += [("linear_w", cout * cin, cin), ("bias", cout, cin)]
        self.d += cout * cin + cout
        return self._push(rec)

    def next_unit(self):
        self.unit += 1

    @property
    def n_units(self):
        return self.unit + 1

    def set_blocks(self, unit_block):
        """unit_block[u] = block (1..P) of residual unit u; blocks must be
        non-decreasing along the model so every block is a contiguous run of
        tensors (Sec. 3, eq. (partition))."""
        assert len(unit_block) == self.n_units
        assert all(unit_block[i] <= unit_block[i + 1] for i in range(len(unit_block) - 1))
        for rec in self.layers:
            rec["block"] = unit_block[rec["unit"]] if rec["poff"] >= 0 else 0
        self.P = max(unit_block)
        return self

    def block_range(self, i):
        """Half-open [lo, hi) of block i in x; block 0 is the whole vector
        (Sec. 3, eq. (partition): x_0 = x[1..d], x_i = x[b_{i-1}+1 .. b_i])."""
        if i == 0:
            return 0, self.d
        offs = []
        for idx, rec in enumerate(self.layers):
            if rec["poff"] >= 0 and rec["block"] == i:
                offs.append((rec["poff"], rec["poff"] + layer_params(rec)))
        if not offs:
            return 0, 0
        return min(o[0] for o in offs), max(o[1] for o in offs)


def layer_params(rec):
    if rec["op"] == CONV:
        return rec["cout"] * rec["cin"] * rec["k"] ** 2 + (rec["cout"] if rec["bias"] else 0)
    if rec["op"] == BN:
        return 2 * rec["cout"]
    if rec["op"] == LINEAR:
        return rec["cout"] * rec["cin"] + rec["cout"]
    return 0


def tiny(n_classes=10, hw=32):
    """Two 3x3 convs with bias and ReLU, global average pool, linear.  Unit 0
    holds the convs, unit 1 the linear head."""
    net = Net("tiny", 3, hw, hw, n_classes)
    a = net.conv(-1, 3, 8, 3, 1, 1, bias=True)
    a = net.relu(a)
    a = net.conv(a, 8, 16, 3, 1, 1, bias=True)
    a = net.relu(a)
    a = net.gap(a)
    net.next_unit()
    net.linear(a, 16, n_classes)
    return net.set_blocks([1, 2])


def _basic_unit(net, x, cin, cout, stride, relu=True):
    net.next_unit()
    h = net.conv(x, cin, cout, 3, stride, 1)
    h = net.bn(h, cout)
    if relu:
        h = net.relu(h)
    h = net.conv(h, cout, cout, 3, 1, 1)
    h = net.bn(h, cout)
    if stride != 1 or cin != cout:
        s = net.conv(x, cin, cout, 1, stride, 0)
        s = net.bn(s, cout)
    else:
        s = x
    h = net.add(h, s)
    return net.relu(h) if relu else h


def resnet_cifar(n_per_stage=3, widths=(16, 32, 64), n_classes=10, hw=32, relu=True):
    """CIFAR ResNet with post-activation basic units and projection (1x1
    conv + BN) shortcuts.  Units: 0 = stem, 1..3n = residual units,
    3n+1 = head.  relu=False drops every ReLU (a piecewise-smooth-free twin
    with the same convolutions, used to compare gradients across
    precisions)."""
    net = Net("resnet%d" % (6 * n_per_stage + 2), 3, hw, hw, n_classes)
    x = net.conv(-1, 3, widths[0], 3, 1, 1)
    x = net.bn(x, widths[0])
    if relu:
        x = net.relu(x)
    cin = widths[0]
    for si, w in enumerate(widths):
        for b in range(n_per_stage):
            stride = 2 if (si > 0 and b == 0) else 1
            x = _basic_unit(net, x, cin, w, stride, relu)
            cin = w
    net.next_unit()
    x = net.gap(x)
    net.linear(x, cin, n_classes)
    return net


def _preact_unit(net, x, cin, cout, stride, relu=True):
    net.next_unit()
    act = net.relu if relu else (lambda t: t)
    o1 = act(net.bn(x, cin))
    h = net.conv(o1, cin, cout, 3, stride, 1)
    h = act(net.bn(h, cout))
    h = net.conv(h, cout, cout, 3, 1, 1)
    if stride != 1 or cin != cout:
        s = net.conv(o1, cin, cout, 1, stride, 0)
    else:
        s = x
    return net.add(h, s)


def wrn(depth=16, widen=8, n_classes=100, hw=32, relu=True):
    """Pre-activation Wide ResNet-depth-widen.  Units: 0 = stem, then
    3*(depth-4)/6 residual units, then the head (final BN-ReLU, pool,
    linear).  relu=False drops every ReLU (the decision-free twin)."""
    n = (depth - 4) // 6
    widths = (16 * widen, 32 * widen, 64 * widen)
    net = Net("wrn%d_%d" % (depth, widen), 3, hw, hw, n_classes)
    x = net.conv(-1, 3, 16, 3, 1, 1)
    cin = 16
    for si, w in enumerate(widths):
        for b in range(n):
            stride = 2 if (si > 0 and b == 0) else 1
            x = _preact_unit(net, x, cin, w, stride, relu)
            cin = w
    net.next_unit()
    x = net.bn(x, cin)
    if relu:
        x = net.relu(x)
    x = net.gap(x)
    net.linear(x, cin, n_classes)
    return net


def resnet_imagenet(units_per_stage=(2, 2, 2, 2), widths=(64, 128, 256, 512), n_classes=1000, hw=224, relu=True):
    """ImageNet ResNet with basic units (ResNet-18 by default): 7x7/2 stem,
    BN, ReLU, 3x3/2 max pool, four stages, projection shortcuts.
    relu=False drops every ReLU (the max pool stays)."""
    net = Net("resnet%d" % (2 + 2 * sum(units_per_stage)), 3, hw, hw, n_classes)
    x = net.conv(-1, 3, widths[0], 7, 2, 3)
    x = net.bn(x, widths[0])
    if relu:
        x = net.relu(x)
    x = net.maxpool(x, 3, 2, 1)
    cin = widths[0]
    for si, (w, nu) in enumerate(zip(widths, units_per_stage)):
        for b in range(nu):
            stride = 2 if (si > 0 and b == 0) else 1
            x = _basic_unit(net, x, cin, w, stride, relu)
            cin = w
    net.next_unit()
    x = net.gap(x)
    net.linear(x, cin, n_classes)
    return net


def _bottleneck(net, x, cin, width, stride, relu=True):
    """Bottleneck residual unit: 1x1 conv to `width`, 3x3 conv (carrying the
    stride), 1x1 conv to 4*width, each followed by BN (and ReLU but the
    last); the shortcut is the input or a 1x1 strided conv + BN; ReLU after
    the sum."""
    net.next_unit()
    out = 4 * width
    h = net.bn(net.conv(x, cin, width, 1, 1, 0), width)
    if relu:
        h = net.relu(h)
    h = net.bn(net.conv(h, width, width, 3, stride, 1), width)
    if relu:
        h = net.relu(h)
    h = net.bn(net.conv(h, width, out, 1, 1, 0), out)
    s = x if (stride == 1 and cin == out) else net.bn(net.conv(x, cin, out, 1, stride, 0), out)
    h = net.add(h, s)
    return net.relu(h) if relu else h


def resnet_bottleneck(units_per_stage=(3, 4, 6, 3), widths=(64, 128, 256, 512), n_classes=1000, hw=224, relu=True):
    """ImageNet ResNet with bottleneck units (ResNet-50 by default): 7x7/2
    stem, BN, ReLU, 3x3/2 max pool, four stages (the first unit of stages
    2-4 strides in its 3x3 conv), global pool, linear."""
    net = Net("resnet%d" % (2 + 3 * sum(units_per_stage)), 3, hw, hw, n_classes)
    x = net.bn(net.conv(-1, 3, widths[0], 7, 2, 3), widths[0])
    if relu:
        x = net.relu(x)
    x = net.maxpool(x, 3, 2, 1)
    cin = widths[0]
    for si, (w, nu) in enumerate(zip(widths, units_per_stage)):
        for b in range(nu):
            x = _bottleneck(net, x, cin, w, 2 if (si > 0 and b == 0) else 1, relu)
            cin = 4 * w
    net.next_unit()
    x = net.gap(x)
    net.linear(x, cin, n_classes)
    return net


# SqueezeNet v1.0's Fire modules (squeeze, expand 1x1, expand 3x3)
SQUEEZENET_FIRES = ((16, 64, 64), (16, 64, 64), (32, 128, 128), (32, 128, 128),
                    (48, 192, 192), (48, 192, 192), (64, 256, 256), (64, 256, 256))


def _fire(net, x, cin, s, e1, e3, relu=True):
    """Fire module: squeeze 1x1 conv (s) + ReLU, then expand 1x1 (e1) and
    expand 3x3 (e3, padding 1) convs on the squeezed map, each + ReLU, their
    outputs concatenated (e1 channels first).  One unit."""
    net.next_unit()
    act = net.relu if relu else (lambda t: t)
    sq = act(net.conv(x, cin, s, 1, 1, 0, bias=True))
    a = act(net.conv(sq, s, e1, 1, 1, 0, bias=True))
    b = act(net.conv(sq, s, e3, 3, 1, 1, bias=True))
    return net.concat(a, b)


def squeezenet(n_classes=10, hw=32, stem=96, fires=SQUEEZENET_FIRES, pools_after=(2, 6), relu=True):
    """SqueezeNet v1.0 for 32x32 inputs.  Units: 0 = stem (3x3 conv + ReLU,
    3x3/2 max pool), one per Fire module (a 3x3/2 max pool follows the
    modules listed in pools_after: fire4 and fire8), last = the classifier
    (1x1 conv to the classes + ReLU, global average pool).  relu=False drops
    every ReLU."""
    net = Net("squeezenet", 3, hw, hw, n_classes)
    act = net.relu if relu else (lambda t: t)
    x = act(net.conv(-1, 3, stem, 3, 1, 1, bias=True))
    x = net.maxpool(x, 3, 2, 1)
    cin = stem
    for i, (s, e1, e3) in enumerate(fires):
        x = _fire(net, x, cin, s, e1, e3, relu)
        cin = e1 + e3
        if i in pools_after:
            x = net.maxpool(x, 3, 2, 1)
    net.next_unit()
    x = act(net.conv(x, cin, n_classes, 1, 1, 0, bias=True))
    net.gap(x)
    return net


# ---- the workloads' models with their partitions (units -> blocks) ----

def tiny_p2():
    return tiny()


def resnet20_p4(n_classes=10, relu=True):
    # units: stem, s1u1..s1u3, s2u1..s2u3, s3u1..s3u3, head
    # blocks: {stem,s1u1,s1u2} {s1u3,s2u1} {s2u2,s2u3,s3u1} {s3u2,s3u3,head}
    return resnet_cifar(3, (16, 32, 64), n_classes, relu=relu).set_blocks([1, 1, 1, 2, 2, 3, 3, 3, 4, 4, 4])


def wrn16_8_p4(n_classes=100):
    # units: stem, s1u1, s1u2, s2u1, s2u2, s3u1, s3u2, head
    return wrn(16, 8, n_classes).set_blocks([1, 1, 1, 2, 3, 3, 4, 4])


def resnet18_p4(n_classes=1000):
    # units: stem, s1u1, s1u2, s2u1, s2u2, s3u1, s3u2, s4u1, s4u2, head
    return resnet_imagenet().set_blocks([1, 1, 2, 2, 2, 3, 3, 4, 4, 4])


def resnet50_p4(n_classes=1000, relu=True):
    # units: stem, s1u1..s1u3, s2u1..s2u4, s3u1..s3u6, s4u1..s4u3, head
    # blocks: {stem,s1u1-3,s2u1} {s2u2-4,s3u1} {s3u2-5} {s3u6,s4u1-3,head}
    return resnet_bottleneck(n_classes=n_classes, relu=relu).set_blocks(
        [1, 1, 1, 1, 1, 2, 2, 2, 2, 3, 3, 3, 3, 4, 4, 4, 4, 4])


def squeezenet_p4(n_classes=10, relu=True):
    # units: stem, fire2..fire9, classifier; cuts nearest to the quartiles of
    # the forward work: {stem, fire2, fire3} {fire4, fire5} {fire6, fire7}
    # {fire8, fire9, classifier}
    return squeezenet(n_classes, relu=relu).set_blocks([1, 1, 1, 2, 2, 3, 3, 4, 4, 4])

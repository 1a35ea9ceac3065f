"""Helpers shared by the GPU parity tests: seeded inputs on both sides, the
per-tensor relative error measure, and twin model builders (oracle list +
library list) for small test networks."""
from __future__ import annotations

import numpy as np

import synth
from oracle import models as OM
from paper_2203_06638_amd import models as PM

# Tolerances (max relative error, per tensor): forward logits and
# activations 1e-4, gradients and updated parameters 1e-3 in fp32.  The
# denominator of an entry is max(|r_e|, tau * max|r|): entries near zero are
# judged against the tensor's largest entry.  tau is chosen per bar so the
# absolute floor is the same, 1e-6 * max|r| (about 8 fp32 ulps of the largest
# entry) -- below that, fp32 sums of hundreds to hundreds of thousands of
# terms cannot resolve a value.
TOL_LOGITS = 1e-4
TOL_GRAD = 1e-3
TOL_PARAM = 1e-3
TAU_LOGITS = 1e-2
TAU = 1e-3
# A gradient entry is a sum of products; when the products cancel, fp32 can
# only resolve it to about the terms' own accuracy times the sum of their
# magnitudes C_e (the oracle's grad_scale).  Activation gradients carry
# errors up to ~1e-6 of their largest entry, i.e. ~5e-6 of their mean
# magnitude, so the denominator also includes KAPPA * C_e: with the 1e-3 bar
# that is an absolute floor of 1e-5 * C_e.
KAPPA = 1e-2

# bf16 workloads (bf16 activations, activation gradients and conv weights;
# fp32 accumulation, fp32 master parameters): max relative error 5e-2 per
# tensor in the max norm, max_e |g_e - r_e| / max_e |r_e| (tau = 1).  Every
# stored tensor and every conv weight is rounded to 8 significant bits
# (relative error up to 2^-8), and the error this leaves in a sum is
# proportional to the magnitudes of its terms, not to the sum: near-zero
# entries of a tensor carry errors of the size of the tensor's typical
# entries (measured: ~2e-3 of max|r| per layer), which an elementwise
# measure with a small floor would report as O(1).  Cancelling gradient sums
# keep the floor KAPPA_BF16 * C_e = 5e-3 * C_e at the 5e-2 bar.
TOL_BF16 = 5e-2
TAU_BF16 = 1.0
KAPPA_BF16 = 0.1


def relerr(gpu, ref, tau=TAU):
    """max_e |g_e - r_e| / max(|r_e|, tau * max|r|)."""
    g = np.asarray(gpu, np.float64).ravel()
    r = np.asarray(ref, np.float64).ravel()
    if r.size == 0:
        return 0.0
    big = np.max(np.abs(r))
    if big == 0.0:
        return float(np.max(np.abs(g)))
    den = np.maximum(np.abs(r), tau * big)
    return float(np.max(np.abs(g - r) / den))


def relerr_scaled(gpu, ref, scale, tau=TAU, kappa=KAPPA):
    """max_e |g_e - r_e| / max(|r_e|, tau * max|r|, kappa * C_e)."""
    g = np.asarray(gpu, np.float64).ravel()
    r = np.asarray(ref, np.float64).ravel()
    c = np.asarray(scale, np.float64).ravel()
    if r.size == 0:
        return 0.0
    den = np.maximum(np.maximum(np.abs(r), tau * np.max(np.abs(r))), kappa * c)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(g - r) / den))


def tensor_errors(net, gpu_vec, ref_vec, lo=0, hi=None, tau=TAU, scale=None, kappa=KAPPA):
    """{tensor name: error} over the oracle net's tensors inside [lo, hi);
    with `scale` (the oracle's condition scales) the measure is
    relerr_scaled, else relerr."""
    hi = net.d if hi is None else hi
    out = {}
    for name, off, n in net.tensors:
        if off >= lo and off + n <= hi:
            if scale is None:
                out[name] = relerr(gpu_vec[off:off + n], ref_vec[off:off + n], tau)
            else:
                out[name] = relerr_scaled(gpu_vec[off:off + n], ref_vec[off:off + n], scale[off:off + n], tau,
                                          kappa)
    return out


def worst(errs):
    if not errs:
        return ("-", 0.0)
    k = max(errs, key=errs.get)
    return (k, errs[k])


# Kink margin required before a gradient comparison between the fp64 oracle
# and the fp32 kernels is called well posed: the smallest ReLU input (or
# max-pool runner-up gap) relative to its layer's largest input must exceed
# twice the largest pre-activation disagreement measured between the two
# (about 1e-6 of the layer's largest input).  Below it, both mask / argmax
# decisions are valid answers and the gradients legitimately differ.
KINK_BAND = 2e-6


def well_posed_seed(net, make, seeds=range(1000, 1200), band=KINK_BAND):
    """First seed whose inputs (x, images) = make(seed) keep every ReLU /
    max-pool decision farther than `band` from its kink, judged by the
    oracle alone.  Returns (seed, margin)."""
    from oracle import lppref as R
    for s in seeds:
        x, img = make(s)
        m = R.kink_margin(net, x, img)
        if m > band:
            return s, m
    raise AssertionError("no well-posed seed found")


def assert_decisions_match(o, ctx, worker, x, img, band=KINK_BAND):
    """The other half of the well-posedness argument: the GPU's values at
    every ReLU / max-pool input deviate from the oracle's by less than
    band/2 of the layer's largest input, so with an oracle margin above
    `band` both sides take every decision the same way.  A ReLU whose input
    the GPU never stores (applied by the producing conv's epilogue) is
    checked through its output: exactly zero wherever the oracle's input is
    negative (the same decision), and within band/2 of the oracle's input
    elsewhere."""
    from oracle import lppref as R
    from oracle import models as OM
    from paper_2203_06638_amd import lpp
    shapes = R.shapes(o)
    worst = 0.0
    for li, rec in enumerate(o.layers):
        if rec["op"] not in (OM.RELU, OM.MAXPOOL) or rec["in0"] < 0:
            continue
        src = rec["in0"]
        ref = R.activation(o, x, img, src)
        big = np.max(np.abs(ref))
        try:
            got = ctx.get_activation(worker, src, shapes[src])
        except lpp.LppError as e:
            assert e.code == lpp.ESTATE and rec["op"] == OM.RELU, (li, e)
            got = ctx.get_activation(worker, li, shapes[li])
            assert not np.any(got[ref < 0]), ("ReLU input of layer %d: a clipped input kept" % li)
            assert np.all(got[ref > 0] > 0), ("ReLU input of layer %d: a passed input clipped" % li)
            ref = np.maximum(ref, 0.0)
        if big > 0:
            worst = max(worst, float(np.max(np.abs(got - ref)) / big))
    assert worst < band / 2, ("decision inputs deviate by %.2e of their scale" % worst)
    return worst


def inputs(seed, n, shape, n_classes):
    return synth.images(seed, n, *shape), synth.labels(seed, n, n_classes)


def init_x(specs, seed, perturb=0.05):
    """He/uniform init, then BN affine and biases moved off 1/0 so their
    gradients are exercised."""
    x = synth.init_params(specs, seed)
    return synth.perturb(x, seed, perturb)


def twin_conv_net(cin, c1, k, stride, pad, c2, hw, n_classes=6):
    """image -> conv(k, stride, pad) -> ReLU -> conv3x3 -> GAP -> linear.
    Block 1: the convs; block 2: the linear head."""
    o = OM.Net("convnet", cin, hw, hw, n_classes)
    a = o.conv(-1, cin, c1, k, stride, pad)
    a = o.relu(a)
    a = o.conv(a, c1, c2, 3, 1, 1)
    a = o.gap(a)
    o.next_unit()
    o.linear(a, c2, n_classes)
    o.set_blocks([1, 2])
    p = PM.Model("convnet", (cin, hw, hw), n_classes)
    x = p.conv(-1, c1, k, stride, pad)
    x = p.relu(x)
    x = p.conv(x, c2, 3, 1, 1)
    x = p.gap(x)
    p.new_unit()
    p.linear(x, n_classes)
    p.assign_blocks([1, 2])
    return o, p


def twin_conv2_net(cin, c0, c1, k, stride, pad, hw, n_classes=6):
    """image -> conv3x3 -> ReLU -> conv(k, stride, pad) -> GAP -> linear: the
    second conv has a data gradient of its own stride.  Block 1: the convs;
    block 2: the linear head."""
    o = OM.Net("conv2net", cin, hw, hw, n_classes)
    a = o.relu(o.conv(-1, cin, c0, 3, 1, 1))
    a = o.gap(o.conv(a, c0, c1, k, stride, pad))
    o.next_unit()
    o.linear(a, c1, n_classes)
    o.set_blocks([1, 2])
    p = PM.Model("conv2net", (cin, hw, hw), n_classes)
    x = p.relu(p.conv(-1, c0, 3, 1, 1))
    x = p.gap(p.conv(x, c1, k, stride, pad))
    p.new_unit()
    p.linear(x, n_classes)
    p.assign_blocks([1, 2])
    return o, p


def twin_bn_net(cin, c, hw, n_classes=5):
    """conv3x3 -> BN -> ReLU -> conv3x3 -> BN -> add(skip) -> ReLU -> GAP ->
    linear, two blocks."""
    o = OM.Net("bnnet", cin, hw, hw, n_classes)
    a = o.relu(o.bn(o.conv(-1, cin, c, 3, 1, 1), c))
    b = o.bn(o.conv(a, c, c, 3, 1, 1), c)
    a = o.relu(o.add(b, a))
    o.next_unit()
    a = o.gap(a)
    o.linear(a, c, n_classes)
    o.set_blocks([1, 2])
    p = PM.Model("bnnet", (cin, hw, hw), n_classes)
    x = p.relu(p.bn(p.conv(-1, c, 3)))
    y = p.bn(p.conv(x, c, 3))
    x = p.relu(p.add(y, x))
    p.new_unit()
    p.linear(p.gap(x), n_classes)
    p.assign_blocks([1, 2])
    return o, p


def routing_lo(o):
    """First parameter index above every max pool: gradients of the
    parameters below a max pool pass through its argmax decisions, which a
    lower-precision forward may take differently (near-ties) from the fp64
    oracle."""
    pools = [i for i, r in enumerate(o.layers) if r["op"] == OM.MAXPOOL]
    if not pools:
        return 0
    lo = 0
    for name, off, n in o.tensors:
        if int(name[1:name.index(".")]) < max(pools):
            lo = max(lo, off + n)
    return lo

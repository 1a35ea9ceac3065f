"""Parity of the bf16 workloads' HIP path (bf16 activations, activation
gradients and conv weights on bf16 matrix cores, fp32 accumulation, fp32
master parameters) with the fp64 CPU oracle, in sequential mode.

Bar: max relative error 5e-2 per tensor on logits, gradients, momenta and
the block update (tests/parity.py: TOL_BF16, TAU_BF16, KAPPA_BF16).  The
images are rounded to bf16 before both sides see them, so input
quantisation is not counted as error; the oracle computes in fp64 without
any bf16 emulation.  Comparisons of gradients are made where both sides
take the same decisions: exact-grid convolution inputs (a ReLU keeps the
sign of a rounded value, so its mask is identical), or ReLU-free twins of
the architectures.  At the workloads' full sizes (batch 128, WRN-16-8 at
32x32 and ResNet-18 at 224x224) every convolution is checked teacher-forced
on sampled outputs: the oracle recomputes sampled output entries and weight-
gradient entries from the GPU's own stored inputs in fp64.
"""
import sys

import numpy as np
import pytest

import synth
from oracle import lppref as R
from oracle import models as OM
from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM
from tests import parity as T

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.init()


def dev(img, lab):
    return (torch.from_numpy(np.ascontiguousarray(img)).cuda(),
            torch.from_numpy(np.ascontiguousarray(lab, np.int32)).cuda())


def bf(a):
    return synth.round_to_bf16(np.asarray(a, np.float32))


def check(o, got, ref, lo, hi, what, scale):
    errs = T.tensor_errors(o, got, ref, lo, hi, tau=T.TAU_BF16, scale=scale, kappa=T.KAPPA_BF16)
    w = T.worst(errs)
    say("  worst %s error %s %.3e" % (what, w[0], w[1]))
    assert w[1] < T.TOL_BF16, (what, w)


# ---------------------------------------------------------------------------
# single convolution passes on exact-grid inputs
# ---------------------------------------------------------------------------

CONV2_CASES = [
    # cin, c0, c1, k, stride, pad, hw, batch
    (3, 8, 16, 3, 1, 1, 8, 3),        # 3-channel image padded to 8, ragged pixel tiles
    (3, 16, 32, 3, 2, 1, 9, 2),       # stride-2 data gradient, odd size: four unequal parity classes
    (8, 32, 64, 1, 2, 0, 8, 5),       # 1x1 stride 2: three parity classes receive nothing
    (3, 16, 64, 7, 2, 3, 20, 2),      # 7x7 stride 2: 16/12/12/9 taps per class
    (16, 64, 128, 3, 1, 1, 6, 3),     # 128-wide output tiles
    (8, 128, 256, 3, 1, 1, 8, 8),     # K-steps within one tap, two output tiles
]


def grid_inputs(o, seed, n):
    """Images and first-conv weights on grids that bf16 holds exactly (so
    the first conv's output is exact in fp32 accumulation, and rounding it
    keeps every sign: the ReLU takes the same decisions on both sides)."""
    x = T.init_x(o.specs, seed)
    rec = o.layers[0]
    nw = rec["cout"] * rec["cin"] * rec["k"] ** 2
    x[:nw] = synth.grid_values(seed, nw, 2.0 ** -5, 0.5)
    img = synth.grid_values(seed + 1, (n,) + o.in_shape, 2.0 ** -6, 4.0)
    assert np.array_equal(bf(img), img) and np.array_equal(bf(x[:nw]), x[:nw])
    lab = synth.labels(seed, n, o.n_classes)
    return x, img, lab


@pytest.mark.parametrize("case", CONV2_CASES, ids=lambda c: "x".join(map(str, c)))
def test_bf16_conv_passes(case):
    cin, c0, c1, k, st, pad, hw, n = case
    say("bf16 conv case", case)
    o, p = T.twin_conv2_net(cin, c0, c1, k, st, pad, hw)
    x, img, lab = grid_inputs(o, 13, n)
    loss, logits, _ = R.forward_backward(o, x, img, lab)
    g, sc = R.grad_scale(o, x, img, lab)
    with lpp.Context(p, K=1, batch=n, dtype=lpp.BF16) as ctx:
        ctx.set_params(x)
        ctx.step(0, *dev(img, lab), 0, 0.0)
        ref0 = R.activation(o, x, img, 0)
        # exact sums, rounded once to bf16
        assert np.array_equal(ctx.get_activation(0, 0, ref0.shape[1:]), bf(ref0))
        ref2 = R.activation(o, x, img, 2)
        e2 = T.relerr(ctx.get_activation(0, 2, ref2.shape[1:]), ref2, T.TAU_BF16)
        el = T.relerr(ctx.get_logits(0), logits, T.TAU_BF16)
        say("  second conv output error %.3e, logits error %.3e" % (e2, el))
        assert e2 < T.TOL_BF16 and el < T.TOL_BF16
        assert abs(ctx.get_loss(0) - loss) < 1e-2 * max(1.0, abs(loss))
        check(o, ctx.get_grad(0), g, 0, o.d, "grad", sc)
        # the data gradient into the ReLU output, against the oracle's
        dref = R.activation_grad(o, x, img, lab, 1)
        assert T.relerr(ctx.get_activation_grad(0, 1, dref.shape[1:]), dref, T.TAU_BF16) < T.TOL_BF16
        assert np.array_equal(ctx.get_params(0), x)


# ---------------------------------------------------------------------------
# the architectures' small instances, every partition (ReLU-free twins for
# the gradients, the real networks for the forward pass)
# ---------------------------------------------------------------------------

def _wrn_mini(relu):
    return (OM.wrn(10, 2, 10, 16, relu=relu).set_blocks([1, 1, 2, 3, 4]),
            PM.wide_resnet(10, 2, 10, 16, blocks=[1, 1, 2, 3, 4], act=relu))


def _rn_mini(relu):
    return (OM.resnet_imagenet((1, 1, 1, 1), (16, 32, 64, 128), 10, 128, relu=relu).set_blocks([1, 1, 2, 3, 4, 4]),
            PM.resnet_imagenet((1, 1, 1, 1), (16, 32, 64, 128), 10, 128, blocks=[1, 1, 2, 3, 4, 4], act=relu))


def _bottleneck_mini(relu):
    return (OM.resnet_bottleneck((1, 2, 1, 1), (8, 16, 16, 32), 10, 64, relu=relu).set_blocks([1, 1, 2, 2, 3, 4, 4]),
            PM.resnet_bottleneck((1, 2, 1, 1), (8, 16, 16, 32), 10, 64, blocks=[1, 1, 2, 2, 3, 4, 4], act=relu))


# batch sizes: the bottleneck mini's last stage is 2x2 at 64x64 input, so its
# batch norm sees 4 values per image and channel; batch 8 keeps the
# normalisation from amplifying bf16 rounding (at batch 2, 8 values)
MINIS = {"wrn10_2": (_wrn_mini, 4), "resnet_imagenet_mini": (_rn_mini, 2), "resnet_bottleneck_mini": (_bottleneck_mini, 8)}


def _bf16_partition_step(o, p, x, m0, img, lab, partition, lr=0.1, mu=0.9):
    xr = x.astype(np.float64)
    mr = m0.astype(np.float64)
    _, sc = R.grad_scale(o, xr, img, lab)
    g, loss, logits = R.step(o, xr, mr, img, lab, partition, lr, mu)
    n = img.shape[0]
    with lpp.Context(p, K=1, batch=n, dtype=lpp.BF16, momentum=mu) as ctx:
        ctx.set_params(x)
        w = max(partition - 1, 0)
        ctx.set_momentum(w, m0)
        ctx.step(w, *dev(img, lab), partition, lr)
        el = T.relerr(ctx.get_logits(w), logits, T.TAU_BF16)
        say("  logits error %.3e" % el)
        assert el < T.TOL_BF16
        lo, hi = o.block_range(partition)
        clo = max(lo, T.routing_lo(o))
        check(o, ctx.get_grad(w), g, clo, hi, "grad", sc)
        check(o, ctx.get_momentum(w), mr, clo, hi, "momentum", sc)
        # the block's update x_new - x against the oracle's
        got = ctx.get_params(0)
        check(o, got.astype(np.float64) - x, xr - x.astype(np.float64), clo, hi, "update", lr * sc)
        assert np.array_equal(got[:lo], x[:lo]) and np.array_equal(got[hi:], x[hi:])


@pytest.mark.parametrize("name", sorted(MINIS))
def test_bf16_minis_all_partitions(name):
    mk, n = MINIS[name]
    o, p = mk(False)
    x = T.init_x(o.specs, 3001)
    img, lab = T.inputs(3002, n, o.in_shape, 10)
    img = bf(img)
    m0 = (np.random.default_rng(7).standard_normal(o.d) * 1e-2).astype(np.float32)
    for part in range(0, 5):
        say(name, "partition", part)
        _bf16_partition_step(o, p, x, m0, img, lab, part)


@pytest.mark.parametrize("name", sorted(MINIS))
def test_bf16_minis_forward_with_relu(name):
    mk, n = MINIS[name]
    o, p = mk(True)
    x = T.init_x(o.specs, 3011)
    img, lab = T.inputs(3012, n, o.in_shape, 10)
    img = bf(img)
    loss, logits, _ = R.forward_backward(o, x, img, lab, grad=False)
    with lpp.Context(p, K=1, batch=n, dtype=lpp.BF16) as ctx:
        ctx.set_params(x)
        ctx.step(0, *dev(img, lab), 0, 0.0)
        el = T.relerr(ctx.get_logits(0), logits, T.TAU_BF16)
        say(name, "logits error %.3e, loss %.5f vs %.5f" % (el, ctx.get_loss(0), loss))
        assert el < T.TOL_BF16
        assert abs(ctx.get_loss(0) - loss) < 2e-2 * abs(loss)


def test_bf16_full_width_small_batch_forward():
    """WRN-16-8 (widths 128/256/512) at batch 16 and ResNet-18 at 224x224,
    batch 2, with ReLUs: logits and loss against the oracle."""
    for o, p, n, seed in ((OM.wrn16_8_p4(), PM.wrn16_8(), 16, 3021), (OM.resnet18_p4(), PM.resnet18(), 2, 3031)):
        x = T.init_x(o.specs, seed)
        img, lab = T.inputs(seed + 1, n, o.in_shape, o.n_classes)
        img = bf(img)
        loss, logits, _ = R.forward_backward(o, x, img, lab, grad=False)
        with lpp.Context(p, K=1, batch=n, dtype=lpp.BF16) as ctx:
            ctx.set_params(x)
            ctx.step(0, *dev(img, lab), 0, 0.0)
            err = T.relerr(ctx.get_logits(0), logits, T.TAU_BF16)
            say(o.name, "logits error %.3e" % err)
            assert err < T.TOL_BF16
            assert abs(ctx.get_loss(0) - loss) < 2e-2 * abs(loss)


# ---------------------------------------------------------------------------
# full size, in the benchmark's launch configuration: teacher-forced checks
# of every convolution on sampled outputs, and properties of the gradient
# ---------------------------------------------------------------------------

def _teacher_forced_convs(o, ctx, x, img, rng, samples=96, fused=None):
    """For each conv: sampled output entries recomputed in fp64 from the
    GPU's stored input and the bf16-rounded weights; sampled weight-gradient
    entries recomputed from the GPU's stored input and output gradient.
    Returns the worst normalised errors (forward, weight gradient); fused[0]
    counts the convs checked through their fused residual add."""
    shapes = R.shapes(o)
    fused = [0] if fused is None else fused
    n = img.shape[0]
    xw = bf(x).astype(np.float64)
    gvec = ctx.get_grad(0).astype(np.float64)
    worst_f = worst_w = 0.0
    for li, rec in enumerate(o.layers):
        if rec["op"] != OM.CONV:
            continue
        src = img.astype(np.float64) if rec["in0"] < 0 else ctx.get_activation(0, rec["in0"], shapes[rec["in0"]]).astype(np.float64)
        resid = None
        try:
            out = ctx.get_activation(0, li, shapes[li]).astype(np.float64)
            dout = ctx.get_activation_grad(0, li, shapes[li]).astype(np.float64)
        except lpp.LppError as e:
            # a conv whose epilogue adds the residual (its only consumer, a
            # residual add): check the stored sum round(round(conv) + res)
            # against the conv recomputed plus the GPU's stored residual; the
            # gradient at the conv output is the add's
            assert e.code == lpp.ESTATE
            add = next(c for c, r in enumerate(o.layers) if r["in0"] == li or r["in1"] == li)
            assert o.layers[add]["op"] == OM.ADD
            other = o.layers[add]["in1"] if o.layers[add]["in0"] == li else o.layers[add]["in0"]
            out = ctx.get_activation(0, add, shapes[add]).astype(np.float64)
            resid = ctx.get_activation(0, other, shapes[other]).astype(np.float64)
            dout = ctx.get_activation_grad(0, add, shapes[add]).astype(np.float64)
            fused[0] += 1
        k, s, pd, cin, cout = rec["k"], rec["stride"], rec["pad"], rec["cin"], rec["cout"]
        W = xw[rec["poff"]:rec["poff"] + cout * cin * k * k].reshape(cout, cin, k, k)
        xp = np.pad(src, ((0, 0), (0, 0), (pd, pd), (pd, pd)))
        ho, wo = shapes[li][1], shapes[li][2]
        for _ in range(samples):
            b, co, i, j = rng.integers(n), rng.integers(cout), rng.integers(ho), rng.integers(wo)
            patch = xp[b, :, i * s:i * s + k, j * s:j * s + k]
            ref = float((patch * W[co]).sum())
            scale = float(np.abs(patch * W[co]).sum()) + 1e-30
            # one rounding to bf16 (at most 2^-8 relative: half a unit in the
            # last of 8 significant bits) of an fp32 sum of the exact bf16
            # products (a few fp32 units of the terms' magnitude sum); with a
            # fused residual, a second rounding of the sum
            bound = 2.0 ** -8 * abs(ref) + 5e-5 * scale
            if resid is not None:
                ref += resid[b, co, i, j]
                bound += 2.0 ** -8 * abs(ref)
            worst_f = max(worst_f, abs(out[b, co, i, j] - ref) / bound)
        gW = gvec[rec["poff"]:rec["poff"] + cout * cin * k * k].reshape(cout, cin, k, k)
        for _ in range(samples // 4):
            co, ci, r, q = rng.integers(cout), rng.integers(cin), rng.integers(k), rng.integers(k)
            xs = xp[:, ci, r:r + (ho - 1) * s + 1:s, q:q + (wo - 1) * s + 1:s]
            prod = dout[:, co] * xs
            ref = float(prod.sum())
            scale = float(np.abs(prod).sum()) + 1e-30
            worst_w = max(worst_w, abs(gW[co, ci, r, q] - ref) / (1e-4 * abs(ref) + 1e-5 * scale))
    return worst_f, worst_w


@pytest.mark.parametrize("which", ["wrn16_8", "resnet18", "resnet50"])
def test_bf16_full_size_teacher_forced(which):
    n = 128
    if which == "wrn16_8":
        o, p = OM.wrn16_8_p4(), PM.wrn16_8()
    elif which == "resnet18":
        o, p = OM.resnet18_p4(), PM.resnet18()
    else:
        o, p = OM.resnet50_p4(), PM.resnet50()
        n = 32                                # the paper's local batch for ResNet-50
    x = T.init_x(o.specs, 3041)
    img, lab = T.inputs(3042, n, o.in_shape, o.n_classes)
    img = bf(img)
    with lpp.Context(p, K=1, batch=n, dtype=lpp.BF16, momentum=0.9) as ctx:
        ctx.set_params(x)
        ti, tl = dev(img, lab)
        ctx.step(0, ti, tl, 0, 0.0)
        loss = ctx.get_loss(0)
        say(which, "loss %.4f (ln C = %.4f)" % (loss, np.log(o.n_classes)))
        assert np.isfinite(loss)
        fused = [0]
        wf, ww = _teacher_forced_convs(o, ctx, x, img, np.random.default_rng(5), fused=fused)
        say(which, "teacher-forced: forward %.3f, weight gradient %.3f (bar 1); %d convs with a fused residual add"
            % (wf, ww, fused[0]))
        if which == "wrn16_8":
            assert fused[0] == 6                 # every unit's last conv adds the shortcut in its epilogue
        assert wf < 1.0 and ww < 1.0
        g = ctx.get_grad(0)
        for part in range(1, 5):
            ctx.step(part - 1, ti, tl, part, 0.0)
            gp = ctx.get_grad(part - 1)
            lo, hi = o.block_range(part)
            assert np.array_equal(gp[lo:hi], g[lo:hi]), part

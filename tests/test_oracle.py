"""Pins of the fp64 CPU oracle against facts fixed outside the oracle itself:
the paper's worked example, closed forms, invariants, an independent library
implementation (PyTorch CPU fp64 functional ops + autograd) and finite
differences.  CPU only.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import lppref as R
from oracle import models as M

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# independent reference: PyTorch CPU fp64 interpreter of a layer list
# --------------------------------------------------------------------------

def torch_loss(net, x, images, labels):
    """Loss and logits of the layer list computed with torch.nn.functional
    (fp64, CPU); x is a torch leaf so autograd gives the gradient."""
    loss, logits, _ = torch_forward(net, x, images, labels)
    return loss, logits


def torch_forward(net, x, images, labels):
    """As torch_loss, also returning every layer's output tensor."""
    acts = []
    img = torch.as_tensor(np.asarray(images, np.float64))
    for rec in net.layers:
        a = img if rec["in0"] < 0 else acts[rec["in0"]]
        op = rec["op"]
        if op == M.CONV:
            n = rec["cout"] * rec["cin"] * rec["k"] ** 2
            w = x[rec["poff"]:rec["poff"] + n].view(rec["cout"], rec["cin"], rec["k"], rec["k"])
            b = x[rec["poff"] + n:rec["poff"] + n + rec["cout"]] if rec["bias"] else None
            y = F.conv2d(a, w, b, stride=rec["stride"], padding=rec["pad"])
        elif op == M.BN:
            c = rec["cout"]
            y = F.batch_norm(a, None, None, x[rec["poff"]:rec["poff"] + c], x[rec["poff"] + c:rec["poff"] + 2 * c],
                             training=True, eps=R.BN_EPS)
        elif op == M.RELU:
            y = F.relu(a)
        elif op == M.ADD:
            y = a + (img if rec["in1"] < 0 else acts[rec["in1"]])
        elif op == M.MAXPOOL:
            y = F.max_pool2d(a, rec["k"], rec["stride"], rec["pad"])
        elif op == M.GAP:
            y = a.mean(dim=(2, 3), keepdim=True)
        elif op == M.CONCAT:
            y = torch.cat([a, img if rec["in1"] < 0 else acts[rec["in1"]]], dim=1)
        elif op == M.LINEAR:
            n = rec["cout"] * rec["cin"]
            w = x[rec["poff"]:rec["poff"] + n].view(rec["cout"], rec["cin"])
            b = x[rec["poff"] + n:rec["poff"] + n + rec["cout"]]
            y = F.linear(a.reshape(a.shape[0], -1), w, b).view(a.shape[0], -1, 1, 1)
        acts.append(y)
    logits = acts[-1].reshape(img.shape[0], -1)
    loss = F.cross_entropy(logits, torch.as_tensor(np.asarray(labels, np.int64)))
    return loss, logits, acts


def torch_grad(net, x0, images, labels):
    x = torch.tensor(np.asarray(x0, np.float64), requires_grad=True)
    loss, logits = torch_loss(net, x, images, labels)
    loss.backward()
    return float(loss.detach()), logits.detach().numpy(), x.grad.numpy()


def _inputs(net, n, seed, perturb=0.1):
    x = synth.init_params(net.specs, seed).astype(np.float64)
    x = synth.perturb(x.astype(np.float32), seed, perturb).astype(np.float64)
    img = synth.images(seed, n, *net.in_shape)
    lab = synth.labels(seed, n, net.n_classes)
    return x, img, lab


MINI_NETS = {
    "tiny": lambda: M.tiny(hw=8),
    "resnet_mini": lambda: M.resnet_cifar(1, (4, 8, 16), n_classes=10, hw=8).set_blocks([1, 1, 2, 3, 4]),
    "wrn_mini": lambda: M.wrn(10, 1, n_classes=7, hw=8).set_blocks([1, 1, 2, 3, 3]),
    "resnet18_mini": lambda: M.resnet_imagenet((1, 1, 1, 1), (4, 8, 8, 16), n_classes=12, hw=32)
    .set_blocks([1, 1, 2, 3, 4, 4]),
    "resnet50_mini": lambda: M.resnet_bottleneck((1, 2, 1, 1), (2, 4, 4, 8), n_classes=9, hw=32)
    .set_blocks([1, 1, 2, 2, 3, 4, 4]),
    "squeezenet_mini": lambda: M.squeezenet(7, 16, 8, ((4, 4, 8), (4, 8, 4), (8, 8, 8)), (1,))
    .set_blocks([1, 1, 2, 3, 4]),
}


# --------------------------------------------------------------------------
# the paper's worked example and the partition definition
# --------------------------------------------------------------------------

def test_block_subtraction_worked_example():
    """Sec. 5: a -|_[2,3] b with a=(1,2,3,4), b=(-10,-20) is (1,12,23,4).
    ref_block_update with lr=1 over the 1-indexed block [2,3] is that
    operator; it pins the inclusive 1-indexed range and the sign."""
    g = json.load(open(os.path.join(GOLDEN, "block_subtraction.json")))
    a = np.array(g["a"], np.float64)
    lo, hi = g["block_first_1indexed"] - 1, g["block_last_1indexed"]
    full_b = np.zeros_like(a)
    full_b[lo:hi] = g["b"]
    R.block_update(a, None, full_b, lo, hi, 1.0)
    assert a.tolist() == g["expected"]


@pytest.mark.parametrize("builder", [M.tiny_p2, M.resnet20_p4, M.wrn16_8_p4, M.resnet18_p4, M.resnet50_p4,
                                     M.squeezenet_p4])
def test_partition_definition(builder):
    """Sec. 3 eq. (partition): b_0 = 0 < b_1 < ... < b_P = d, block 0 is the
    whole vector, blocks 1..P are disjoint and cover it."""
    net = builder()
    assert net.block_range(0) == (0, net.d)
    prev = 0
    for i in range(1, net.P + 1):
        lo, hi = net.block_range(i)
        assert lo == prev and hi > lo
        prev = hi
    assert prev == net.d


# --------------------------------------------------------------------------
# model sizes and shapes
# --------------------------------------------------------------------------

def test_param_counts():
    """d of each model: ResNet-18 (ImageNet, 1000 classes) has the widely
    published 11,689,512 parameters; WRN-16-8 has the ~11.0M of the Wide
    ResNet paper; the tiny CNN's count follows from its layer list."""
    assert M.tiny_p2().d == 3 * 8 * 9 + 8 + 8 * 16 * 9 + 16 + 16 * 10 + 10 == 1562
    assert M.resnet18_p4().d == 11_689_512
    assert round(M.wrn16_8_p4(100).d / 1e6, 1) == 11.0
    assert M.resnet20_p4(10).d == 272_474
    assert M.resnet20_p4(100).d == 278_324
    # ResNet-50 (bottleneck units): the widely published 25,557,032
    assert M.resnet50_p4().d == 25_557_032
    # SqueezeNet v1.0 has the published 1,248,424 parameters at 1000 classes
    # with its 7x7 stem (7*7*3*96 + 96 = 14,208); the 32x32 variant's 3x3
    # stem has 3*3*3*96 + 96 = 2,688 and its classifier 512*C + C
    assert M.squeezenet_p4(10).d == 1_248_424 - 14_208 + 2_688 - (512 * 1000 + 1000) + (512 * 10 + 10) == 729_034
    assert M.squeezenet_p4(100).d == 729_034 + 90 * 513
    for b in (M.tiny_p2, M.resnet20_p4, M.wrn16_8_p4, M.resnet18_p4, M.resnet50_p4, M.squeezenet_p4):
        net = b()
        assert R.num_params(net) == net.d


def _fwd_macs(net):
    S = R.shapes(net)
    macs = 0
    for l, rec in enumerate(net.layers):
        if rec["op"] == M.CONV:
            c, h, w = (int(v) for v in S[l])
            macs += c * h * w * rec["cin"] * rec["k"] ** 2
        elif rec["op"] == M.LINEAR:
            macs += rec["cin"] * rec["cout"]
    return macs


def test_forward_macs():
    """Per-image multiply-adds: ResNet-18 at 224x224 is the widely published
    ~1.82 GMAC; CIFAR ResNet-20 ~41 MMAC; the 10-class ResNet-20 at batch 128
    gives 10.45 GFLOP forward."""
    assert abs(_fwd_macs(M.resnet18_p4()) / 1e9 - 1.82) < 0.01
    # ResNet-50 at 224x224: the widely published ~4.09 GMAC
    assert abs(_fwd_macs(M.resnet50_p4()) / 1e9 - 4.09) < 0.01
    r20 = _fwd_macs(M.resnet20_p4())
    assert abs(r20 * 2 * 128 / 1e9 - 10.45) < 0.02
    S = R.shapes(M.resnet18_p4())
    assert tuple(S[-2]) == (512, 1, 1) and tuple(S[3]) == (64, 56, 56)


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------

@pytest.mark.parametrize("ncls", [10, 100, 1000])
def test_cross_entropy_at_zero_logits(ncls):
    """With all logits 0 the mean CE is ln C, and each row of dlogits
    (softmax - onehot)/N sums to 0, so the bias gradient sums to 0."""
    net = M.tiny(n_classes=ncls, hw=8)
    x, img, lab = _inputs(net, 5, 3)
    lin = net.layers[-1]
    x[lin["poff"]:] = 0.0
    loss, logits, g = R.forward_backward(net, x, img, lab)
    assert np.all(logits == 0.0)
    assert abs(loss - math.log(ncls)) < 1e-14
    db = g[lin["poff"] + lin["cout"] * lin["cin"]:]
    assert abs(db.sum()) < 1e-15
    onehot = np.zeros(ncls)
    for y in lab:
        onehot[y] += 1
    np.testing.assert_allclose(db, (5 / ncls - onehot) / 5, atol=1e-15)


def test_delta_kernel_conv_is_identity():
    """A 3x3 conv whose kernel is 1 at the centre on the diagonal (c -> c)
    and 0 elsewhere reproduces its input."""
    net = M.Net("delta", 3, 9, 7, 3)
    net.conv(-1, 3, 3, 3, 1, 1)
    x = np.zeros(net.d)
    for c in range(3):
        x[((c * 3 + c) * 3 + 1) * 3 + 1] = 1.0
    img = synth.images(5, 2, 3, 9, 7)
    out = R.activation(net, x, img, 0)
    np.testing.assert_array_equal(out, img.astype(np.float64))


def test_1x1_conv_is_matmul_and_strided_conv_vs_numpy():
    """A 1x1 stride-2 conv is a channel matmul of the even-indexed pixels."""
    net = M.Net("pw", 5, 6, 6, 1)
    net.conv(-1, 5, 4, 1, 2, 0, bias=True)
    rng = np.random.default_rng(1)
    x = rng.standard_normal(net.d)
    img = synth.images(6, 3, 5, 6, 6)
    out = R.activation(net, x, img, 0)
    W = x[:20].reshape(4, 5)
    b = x[20:24]
    ref = np.einsum("kc,nchw->nkhw", W, img[:, :, ::2, ::2].astype(np.float64)) + b[None, :, None, None]
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)


def test_maxpool_and_gap_definitions():
    net = M.Net("pool", 2, 7, 7, 2)
    a = net.maxpool(-1, 3, 2, 1)
    net.gap(a)
    img = synth.images(8, 2, 2, 7, 7).astype(np.float64)
    mp = R.activation(net, np.zeros(0), img, 0)
    padded = np.pad(img, ((0, 0), (0, 0), (1, 1), (1, 1)), constant_values=-np.inf)
    ref = np.zeros((2, 2, 4, 4))
    for p in range(4):
        for q in range(4):
            ref[:, :, p, q] = padded[:, :, 2 * p:2 * p + 3, 2 * q:2 * q + 3].max(axis=(2, 3))
    np.testing.assert_array_equal(mp, ref)
    gap = R.activation(net, np.zeros(0), img, 1)
    np.testing.assert_allclose(gap[:, :, 0, 0], ref.mean(axis=(2, 3)), atol=1e-15)


# --------------------------------------------------------------------------
# batch-norm invariants
# --------------------------------------------------------------------------

def _conv_bn_net():
    net = M.Net("cbn", 3, 6, 6, 4)
    a = net.conv(-1, 3, 5, 3, 1, 1, bias=True)
    a = net.bn(a, 5)
    a = net.relu(a)
    a = net.gap(a)
    net.linear(a, 5, 4)
    return net


def test_bn_output_is_normalised():
    """gamma=1, beta=0: per-channel batch mean 0 and biased variance
    var/(var+eps) (i.e. 1 up to eps)."""
    net = _conv_bn_net()
    x, img, lab = _inputs(net, 6, 11)
    bn = net.layers[1]
    x[bn["poff"]:bn["poff"] + 5] = 1.0
    x[bn["poff"] + 5:bn["poff"] + 10] = 0.0
    pre = R.activation(net, x, img, 0)
    y = R.activation(net, x, img, 1)
    var = pre.var(axis=(0, 2, 3))
    np.testing.assert_allclose(y.mean(axis=(0, 2, 3)), 0.0, atol=1e-14)
    np.testing.assert_allclose(y.var(axis=(0, 2, 3)), var / (var + R.BN_EPS), rtol=1e-12)


def test_bn_backward_invariants():
    """Training-mode BN removes the per-channel mean and scale of its input:
    (1) the gradient of a conv bias feeding BN is 0 (sum of dx = 0);
    (2) the loss is invariant to scaling one filter with its bias, so
    sum over that filter of theta * dL/dtheta is 0 (sum of dx*xhat = 0) up to
    the eps term of the variance."""
    net = _conv_bn_net()
    x, img, lab = _inputs(net, 6, 12)
    _, _, g = R.forward_backward(net, x, img, lab)
    conv = net.layers[0]
    nw = 5 * 3 * 9
    assert np.max(np.abs(g[nw:nw + 5])) < 1e-15
    w = x[:nw].reshape(5, 27)
    gw = g[:nw].reshape(5, 27)
    dirderiv = (w * gw).sum(axis=1)
    assert np.max(np.abs(dirderiv)) < 1e-4 * np.max(np.abs(gw))


# --------------------------------------------------------------------------
# whole-model forward and gradient against an independent implementation
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", sorted(MINI_NETS))
def test_against_torch_fp64(name):
    net = MINI_NETS[name]()
    x, img, lab = _inputs(net, 6, 21)
    loss, logits, g = R.forward_backward(net, x, img, lab)
    tl, tlog, tg = torch_grad(net, x, img, lab)
    assert abs(loss - tl) < 1e-12
    np.testing.assert_allclose(logits, tlog, rtol=0, atol=1e-12)
    np.testing.assert_allclose(g, tg, rtol=1e-9, atol=1e-13)


def test_resnet20_against_torch_fp64():
    """The full ResNet-20 layer list (100 classes) at batch 4."""
    net = M.resnet20_p4(100)
    x, img, lab = _inputs(net, 4, 22)
    loss, logits, g = R.forward_backward(net, x, img, lab)
    tl, tlog, tg = torch_grad(net, x, img, lab)
    assert abs(loss - tl) < 1e-11
    np.testing.assert_allclose(logits, tlog, rtol=0, atol=1e-11)
    np.testing.assert_allclose(g, tg, rtol=1e-8, atol=1e-12)


# --------------------------------------------------------------------------
# finite differences
# --------------------------------------------------------------------------

def _fd_check(net, x, img, lab, idx, tol=1e-6):
    _, _, g = R.forward_backward(net, x, img, lab)
    errs = []
    for e in idx:
        h = 1e-6 * max(1.0, abs(x[e]))
        xp = x.copy(); xp[e] += h
        xm = x.copy(); xm[e] -= h
        lp, _, _ = R.forward_backward(net, xp, img, lab, grad=False)
        lm, _, _ = R.forward_backward(net, xm, img, lab, grad=False)
        fd = (lp - lm) / (2 * h)
        errs.append(abs(fd - g[e]) / max(abs(g[e]), 1e-3 * np.max(np.abs(g))))
    return max(errs)


def test_finite_differences_tiny_all_params():
    net = M.tiny(hw=6)
    x, img, lab = _inputs(net, 4, 31)
    assert _fd_check(net, x, img, lab, range(net.d)) < 1e-5


@pytest.mark.parametrize("name", ["resnet_mini", "wrn_mini", "resnet18_mini", "resnet50_mini", "squeezenet_mini"])
def test_finite_differences_sampled(name):
    net = MINI_NETS[name]()
    x, img, lab = _inputs(net, 3, 32)
    rng = np.random.default_rng(5)
    idx = sorted(set(rng.choice(net.d, size=min(net.d, 120), replace=False).tolist()))
    assert _fd_check(net, x, img, lab, idx) < 1e-5


# --------------------------------------------------------------------------
# optimiser steps
# --------------------------------------------------------------------------

def test_momentum_update_matches_torch_sgd():
    """The coupled-weight-decay heavy-ball form (dampening 0, no Nesterov)
    over several steps equals torch.optim.SGD on the restricted block."""
    rng = np.random.default_rng(3)
    d, lo, hi = 40, 7, 29
    x = rng.standard_normal(d)
    m = np.zeros(d)
    xt = torch.tensor(x[lo:hi].copy(), requires_grad=True)
    opt = torch.optim.SGD([xt], lr=0.1, momentum=0.9, weight_decay=5e-4)
    x0 = x.copy()
    for _ in range(5):
        g = rng.standard_normal(d)
        R.block_update(x, m, g, lo, hi, 0.1, 0.9, 5e-4)
        xt.grad = torch.tensor(g[lo:hi].copy())
        opt.step()
    np.testing.assert_allclose(x[lo:hi], xt.detach().numpy(), rtol=1e-14, atol=1e-14)
    assert np.array_equal(x[:lo], x0[:lo]) and np.array_equal(x[hi:], x0[hi:])
    assert np.all(m[:lo] == 0) and np.all(m[hi:] == 0)


@pytest.mark.parametrize("K", [1, 2, 3, 4])
def test_averaging_invariants(K):
    rng = np.random.default_rng(K)
    reps = [rng.standard_normal(257) for _ in range(K)]
    before = [r.copy() for r in reps]
    mean0 = np.mean(before, axis=0)
    R.average(reps)
    for r in reps:
        np.testing.assert_allclose(r, mean0, rtol=0, atol=4e-15)
        np.testing.assert_allclose(r, reps[0], rtol=0, atol=4e-15)
    again = [r.copy() for r in reps]
    R.average(again)
    for a, r in zip(again, reps):
        np.testing.assert_allclose(a, r, rtol=0, atol=4e-15)
    if K == 1:
        assert np.array_equal(reps[0], before[0])


def test_step_is_restricted_full_gradient():
    """A block step moves only its block, by -lr times the restriction of the
    full gradient at the snapshot (Alg. 1 updater; Sec. 2 block gradient)."""
    net = M.resnet_cifar(1, (4, 8, 16), n_classes=10, hw=8).set_blocks([1, 1, 2, 3, 4])
    x, img, lab = _inputs(net, 4, 41)
    _, _, gfull = R.forward_backward(net, x, img, lab)
    for part in range(net.P + 1):
        lo, hi = net.block_range(part)
        xs = x.copy()
        g, _, _ = R.step(net, xs, None, img, lab, part, 0.05)
        assert np.array_equal(g[lo:hi], gfull[lo:hi])
        assert np.all(g[:lo] == 0) and np.all(g[hi:] == 0)
        np.testing.assert_array_equal(xs[:lo], x[:lo])
        np.testing.assert_array_equal(xs[hi:], x[hi:])
        np.testing.assert_allclose(xs[lo:hi], x[lo:hi] - 0.05 * gfull[lo:hi], rtol=0, atol=1e-15)


def test_sequential_schedule_composes_to_averaged_update():
    """Zero-delay eq. (update) of Sec. 5: after one averaging round the
    common iterate is xbar_0 - (lr/K) * sum over replicas and steps of the
    block gradients (plain SGD)."""
    net = M.resnet_cifar(1, (4, 8, 16), n_classes=10, hw=8).set_blocks([1, 1, 2, 3, 4])
    K, P, H, lr = 2, 4, 2, 0.05
    x0 = _inputs(net, 4, 51)[0]
    batches = {b: (synth.images(100 + b, 4, 3, 8, 8), synth.labels(100 + b, 4, 10)) for b in range(8)}
    sched = []
    for rnd in range(H):
        for q in range(K):
            w = q * P + rnd
            sched.append((w, rnd + 1, len(sched)))
    reps, _, _ = R.run_sequential(net, x0, sched, batches, K, P, H, lr)
    # replay each replica alone, collecting its gradients
    total = np.zeros(net.d)
    for q in range(K):
        xq = x0.copy()
        for (w, part, key) in sched:
            if w // P != q:
                continue
            g, _, _ = R.step(net, xq, None, *batches[key], part, lr)
            total += g
    np.testing.assert_allclose(reps[0], x0 - lr / K * total, rtol=0, atol=1e-14)
    # x_k + (vbar - x_k) equals vbar only up to one rounding per replica
    np.testing.assert_allclose(reps[0], reps[1], rtol=0, atol=1e-15)


def test_concat_forward_and_backward_closed_form():
    """Concatenation along channels: the output holds x's channels then y's,
    and the gradient reaching each input is its slice of the output's.  A
    two-branch net (1x1 convs a, b of the image, concatenated, pooled) has
    logits = [mean(a), mean(b)] and the loss gradient of each branch's bias
    is the matching slice of dlogits summed over the batch."""
    net = M.Net("cat", 3, 4, 4, 5)
    a = net.conv(-1, 3, 2, 1, 1, 0, bias=True)
    b = net.conv(-1, 3, 3, 1, 1, 0, bias=True)
    net.gap(net.concat(a, b))
    net.set_blocks([1])
    x, img, lab = _inputs(net, 4, 41)
    loss, logits, g = R.forward_backward(net, x, img, lab)
    wa, ba = x[0:6].reshape(2, 3), x[6:8]
    wb, bb = x[8:17].reshape(3, 3), x[17:20]
    m = img.astype(np.float64).mean(axis=(2, 3))    # [N, 3]
    want = np.concatenate([m @ wa.T + ba, m @ wb.T + bb], axis=1)
    np.testing.assert_allclose(logits, want, rtol=0, atol=1e-13)
    z = want - want.max(axis=1, keepdims=True)
    p = np.exp(z) / np.exp(z).sum(axis=1, keepdims=True)
    dz = (p - np.eye(5)[lab]) / len(lab)
    np.testing.assert_allclose(g[6:8], dz[:, :2].sum(axis=0), rtol=0, atol=1e-14)
    np.testing.assert_allclose(g[17:20], dz[:, 2:].sum(axis=0), rtol=0, atol=1e-14)


# --------------------------------------------------------------------------
# the oracle's helper outputs: activation gradients, condition scales and
# kink margins, each against a definition computed outside the oracle
# --------------------------------------------------------------------------

def _torch_layer_grads(net, x0, images, labels):
    """PyTorch fp64 autograd with retain_grad on every layer output: returns
    (layer outputs, their loss gradients, parameter gradient)."""
    x = torch.tensor(np.asarray(x0, np.float64), requires_grad=True)
    loss, _, acts = torch_forward(net, x, images, labels)
    for a in acts:
        a.retain_grad()
    loss.backward()
    outs = [a.detach().numpy() for a in acts]
    grads = [np.zeros(a.shape) if a.grad is None else a.grad.numpy() for a in acts]
    return outs, grads, x.grad.numpy()


@pytest.mark.parametrize("name", sorted(MINI_NETS))
def test_activation_grad_matches_autograd_every_layer(name):
    """ref_activation_grad(layer) is dL/d(output of layer) of the full
    backward (Sec. 2: the chain rule through every layer).  Against PyTorch
    fp64 autograd with retain_grad, for every layer of every mini net."""
    net = MINI_NETS[name]()
    x, img, lab = _inputs(net, 4, 61)
    _, tgrads, _ = _torch_layer_grads(net, x, img, lab)
    for l in range(len(net.layers)):
        got = R.activation_grad(net, x, img, lab, l)
        want = tgrads[l].reshape(got.shape)
        scale = max(np.max(np.abs(want)), 1e-300)
        assert np.max(np.abs(got - want)) <= 1e-12 * scale, (name, l)


def _windows(xp, k, st, oh, ow):
    """xp[N, C, H, W] (already padded) -> [N, C, oh, ow, k, k] windows."""
    n, c = xp.shape[:2]
    out = np.empty((n, c, oh, ow, k, k))
    for r in range(k):
        for s in range(k):
            out[..., r, s] = xp[:, :, r:r + st * oh:st, s:s + st * ow:st]
    return out


def _scale_net():
    """conv(+bias) -> BN -> ReLU -> conv 3x3/2 -> BN -> ReLU -> GAP ->
    linear: every kind of parameter gradient the oracle scales."""
    net = M.Net("scale", 3, 8, 8, 5)
    a = net.conv(-1, 3, 4, 3, 1, 1, bias=True)
    a = net.relu(net.bn(a, 4))
    a = net.conv(a, 4, 6, 3, 2, 1)
    a = net.relu(net.bn(a, 6))
    net.linear(net.gap(a), 6, 5)
    net.set_blocks([1])
    return net


def test_grad_scale_definition_from_autograd():
    """ref_grad_scale's C_e is, for each parameter gradient entry (a sum of
    products), the sum of the magnitudes of those products.  Written out
    from autograd's layer inputs X and output gradients dY (fp64):
    conv weight C[k,c,r,s] = sum_{n,p,q} |dY[n,k,p,q]| |X_pad[n,c,p*st+r,q*st+s]|,
    conv bias sum |dY|; BN gamma sum |dY * xhat|, beta sum |dY|; linear
    weight |dz|^T |F|, bias sum |dz|."""
    net = _scale_net()
    x, img, lab = _inputs(net, 5, 62, perturb=0.3)
    outs, grads, gt = _torch_layer_grads(net, x, img, lab)
    g, sc = R.grad_scale(net, x, img, lab)
    np.testing.assert_allclose(g, gt, rtol=1e-10, atol=1e-14)
    img64 = np.asarray(img, np.float64)
    want = np.zeros(net.d)
    for l, rec in enumerate(net.layers):
        X = img64 if rec["in0"] < 0 else outs[rec["in0"]]
        dY = grads[l]
        po = rec["poff"]
        if rec["op"] == M.CONV:
            k, st, pad = rec["k"], rec["stride"], rec["pad"]
            xp = np.pad(np.abs(X), ((0, 0), (0, 0), (pad, pad), (pad, pad)))
            oh, ow = dY.shape[2:]
            win = _windows(xp, k, st, oh, ow)                  # [N, C, oh, ow, k, k]
            cw = np.einsum("nkpq,ncpqrs->kcrs", np.abs(dY), win)
            n = cw.size
            want[po:po + n] = cw.ravel()
            if rec["bias"]:
                want[po + n:po + n + rec["cout"]] = np.abs(dY).sum(axis=(0, 2, 3))
        elif rec["op"] == M.BN:
            c = rec["cout"]
            mu = X.mean(axis=(0, 2, 3), keepdims=True)
            var = X.var(axis=(0, 2, 3), keepdims=True)
            xhat = (X - mu) / np.sqrt(var + R.BN_EPS)
            want[po:po + c] = np.abs(dY * xhat).sum(axis=(0, 2, 3))
            want[po + c:po + 2 * c] = np.abs(dY).sum(axis=(0, 2, 3))
        elif rec["op"] == M.LINEAR:
            Fm = np.abs(X.reshape(X.shape[0], -1))
            dz = np.abs(dY.reshape(dY.shape[0], -1))
            n = rec["cout"] * rec["cin"]
            want[po:po + n] = (dz.T @ Fm).ravel()
            want[po + n:po + n + rec["cout"]] = dz.sum(axis=0)
    np.testing.assert_allclose(sc, want, rtol=1e-10, atol=0)
    # a scale that dropped a term or took |sum| instead of sum|.| would be
    # at most |g|; the definition gives strictly more wherever terms cancel
    assert np.all(sc >= np.abs(gt) * (1 - 1e-12))
    assert np.mean(sc > 1.5 * np.abs(gt)) > 0.5


@pytest.mark.parametrize("name", sorted(MINI_NETS))
def test_grad_scale_bounds_gradient_on_minis(name):
    """|g_e| = |sum of terms| <= sum |terms| = C_e for every entry (triangle
    inequality), with equality only where no terms cancel; the gradient the
    function returns is the oracle's full gradient."""
    net = MINI_NETS[name]()
    x, img, lab = _inputs(net, 4, 63)
    g, sc = R.grad_scale(net, x, img, lab)
    _, _, gref = R.forward_backward(net, x, img, lab)
    assert np.array_equal(g, gref)
    assert np.all(sc >= np.abs(g) * (1 - 1e-12) - 1e-300)
    assert np.all(np.isfinite(sc)) and np.max(sc) > 0


def _relu_probe_net(c, h, w):
    net = M.Net("relu_probe", c, h, w, 3)
    a = net.relu(-1)
    net.linear(net.gap(a), c, 3)
    net.set_blocks([1])
    return net


def _pool_probe_net(c, h, w, k, st, pad):
    net = M.Net("pool_probe", c, h, w, 3)
    a = net.maxpool(-1, k, st, pad)
    net.linear(net.gap(a), c, 3)
    net.set_blocks([1])
    return net


def test_kink_margin_relu_closed_form():
    """For a ReLU reading the images directly, the margin is
    min|v| / max|v| over the images: built with every value of magnitude
    in [0.5, 4] except one of magnitude 0.02 (and one of 4), it is 0.005."""
    rng = np.random.default_rng(7)
    img = rng.uniform(0.5, 3.5, size=(2, 3, 4, 4)) * rng.choice([-1.0, 1.0], size=(2, 3, 4, 4))
    img[1, 2, 3, 0] = -0.02
    img[0, 1, 0, 2] = 4.0
    net = _relu_probe_net(3, 4, 4)
    x = synth.init_params(net.specs, 1).astype(np.float64)
    assert R.kink_margin(net, x, img) == pytest.approx(0.02 / 4.0, rel=1e-15)
    img[1, 2, 3, 0] = 0.0
    assert R.kink_margin(net, x, img) == 0.0


def test_kink_margin_maxpool_closed_form():
    """For a max pool reading the images, the margin is the smallest gap
    between a window's largest and second largest value, over max|v|.
    2x2/2 windows without padding: each window holds {t, t - gap_w, lower
    values}; the smallest gap is 0.03 and max|v| is 6, so 0.005.  A window
    with a repeated maximum gives 0 (both argmax choices are valid)."""
    rng = np.random.default_rng(8)
    n, c, h, w = 2, 2, 4, 4
    img = np.zeros((n, c, h, w))
    gaps = rng.uniform(0.2, 1.0, size=(n, c, 2, 2))
    gaps[1, 0, 1, 1] = 0.03
    for b in range(n):
        for ch in range(c):
            for i in range(2):
                for j in range(2):
                    t = rng.uniform(1.0, 5.0)
                    vals = [t, t - gaps[b, ch, i, j], t - 2.0 - rng.uniform(), t - 3.5]
                    perm = rng.permutation(4)
                    for m, v in zip(perm, vals):
                        img[b, ch, 2 * i + m // 2, 2 * j + m % 2] = v
    img[0, 0, 0, 0] = 6.0
    img[0, 0, 0, 1] = 5.0
    img[0, 0, 1, 0] = 0.0
    img[0, 0, 1, 1] = -1.0
    net = _pool_probe_net(c, h, w, 2, 2, 0)
    x = synth.init_params(net.specs, 1).astype(np.float64)
    want = min(0.03, 1.0) / 6.0
    assert R.kink_margin(net, x, img) == pytest.approx(want, rel=1e-12)
    img[1, 1, 2, 2] = img[1, 1, 2:4, 2:4].max()
    img[1, 1, 3, 3] = img[1, 1, 2, 2]
    assert R.kink_margin(net, x, img) == 0.0


def test_kink_margin_padded_pool_and_min_over_layers():
    """3x3/2 pad-1 windows ignore the padding (it never counts as a
    runner-up): a 1x1 image has one-element windows only, so no pool
    margin exists; with a ReLU after the pool the margin is the ReLU's.
    The result is the minimum over every ReLU and pool layer, each
    relative to its own input's largest magnitude."""
    net = M.Net("mix", 1, 3, 3, 2)
    a = net.maxpool(-1, 3, 2, 1)          # 3x3 -> 2x2
    a = net.relu(a)
    net.linear(net.gap(a), 1, 2)
    net.set_blocks([1])
    x = synth.init_params(net.specs, 2).astype(np.float64)
    img = np.array([[[[1.0, -2.0, 0.5],
                      [3.0, 8.0, -0.25],
                      [-4.0, 0.75, -0.1]]]])
    # windows (rows/cols clipped to the image): (0,0): {1,-2,3,8} -> 8 vs 3;
    # (0,1): {-2,0.5,8,-0.25} -> 8 vs 0.5; (1,0): {3,8,-4,0.75} -> 8 vs 3;
    # (1,1): {8,-0.25,0.75,-0.1} -> 8 vs 0.75.  Pool margin 5 / 8.
    # pool output is all 8: ReLU margin 8 / 8 = 1.
    assert R.kink_margin(net, x, img) == pytest.approx(5.0 / 8.0, rel=1e-15)
    img[0, 0, 2, 1] = 7.96       # window (1,1): 8 vs 7.96; (1,0): 8 vs 7.96
    assert R.kink_margin(net, x, img) == pytest.approx(0.04 / 8.0, rel=1e-12)
    one = M.Net("one", 1, 1, 1, 2)
    a = one.maxpool(-1, 3, 2, 1)
    a = one.relu(a)
    one.linear(one.gap(a), 1, 2)
    one.set_blocks([1])
    x1 = synth.init_params(one.specs, 2).astype(np.float64)
    # no window has a runner-up, so only the ReLU counts: |-0.5| / 0.5 = 1
    assert R.kink_margin(one, x1, np.array([[[[-0.5]]]])) == 1.0

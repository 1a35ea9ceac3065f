"""The headline workload's gradient at full size with its ReLUs, and the
folded BN + ReLU path with real clipping.

ResNet-20 (batch 128, fused kernels, folds active) has about 1e5 ReLU inputs
per image, so some input always lies closer to zero than the fp32 / fp64
disagreement and both mask decisions are correct there: the fp64 oracle's
own forward is not a valid reference for the whole backward.  Instead every
layer's backward is checked teacher-forced: the reference for a layer's
gradient is computed in fp64 from the GPU's own stored tensors one level
downstream (its consumers' output gradients, its own forward input, the
ReLU decisions the GPU took, read from its stored or rebuilt outputs), by
the definitions of Sec. 2's chain rule through conv, batch norm, ReLU,
residual add, pooling and the linear head.  Bar: 1e-3 in the C_e measure
(tests/parity.py), C_e being the sum of the magnitudes of the terms each
entry sums.

The folded path against the oracle itself: ResNet-20 at batch 32 with
batch-norm shifts of +4 and -4 on alternate channels, so that the folded
ReLUs clip half of their inputs while every decision keeps a margin
(chosen by the oracle), every partition."""
import sys

import numpy as np
import pytest

from oracle import lppref as R
from oracle import models as OM
from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM
from tests import parity as T
from tests.test_gpu_parity import _partition_step, check_grads, dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.init()


# ---------------------------------------------------------------------------
# fp64 local backward operators (definitions), each returning the value and
# the sum of the magnitudes of the terms it adds
# ---------------------------------------------------------------------------

def conv_data_grad(dY, W, stride, pad, hw):
    """dX of Y = conv(X, W): dX[n,c,i,j] = sum_{k,r,s} dY[n,k,p,q] W[k,c,r,s]
    over i = p*stride - pad + r, j = q*stride - pad + s."""
    n, k, ho, wo = dY.shape
    _, c, rr, ss = W.shape
    h, w = hw
    out = np.zeros((n, c, h + 2 * pad + rr, w + 2 * pad + ss))
    mag = np.zeros_like(out)
    for r in range(rr):
        for s in range(ss):
            sl = (slice(None), slice(None), slice(r, r + stride * ho, stride), slice(s, s + stride * wo, stride))
            out[sl] += np.einsum("nkhw,kc->nchw", dY, W[:, :, r, s], optimize=True)
            mag[sl] += np.einsum("nkhw,kc->nchw", np.abs(dY), np.abs(W[:, :, r, s]), optimize=True)
    return out[:, :, pad:pad + h, pad:pad + w], mag[:, :, pad:pad + h, pad:pad + w]


def conv_weight_grad(X, dY, stride, pad, k):
    """dW[k,c,r,s] = sum_{n,p,q} dY[n,k,p,q] X[n,c,p*stride-pad+r,q*stride-pad+s]."""
    ho, wo = dY.shape[2:]
    xp = np.pad(X, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    g = np.zeros((dY.shape[1], X.shape[1], k, k))
    m = np.zeros_like(g)
    for r in range(k):
        for s in range(k):
            xs = xp[:, :, r:r + stride * (ho - 1) + 1:stride, s:s + stride * (wo - 1) + 1:stride]
            g[:, :, r, s] = np.tensordot(dY, xs, axes=([0, 2, 3], [0, 2, 3]))
            m[:, :, r, s] = np.tensordot(np.abs(dY), np.abs(xs), axes=([0, 2, 3], [0, 2, 3]))
    return g, m


def bn_backward(x, gamma, g, eps=R.BN_EPS):
    """Training-mode BN with batch statistics of x: (dx, dgamma, dbeta) and
    their term-magnitude sums."""
    mcount = x.shape[0] * x.shape[2] * x.shape[3]
    mu = x.mean(axis=(0, 2, 3), keepdims=True)
    rstd = 1.0 / np.sqrt(x.var(axis=(0, 2, 3), keepdims=True) + eps)
    xh = (x - mu) * rstd
    dgam = (g * xh).sum(axis=(0, 2, 3))
    dbet = g.sum(axis=(0, 2, 3))
    sg = np.abs(g * xh).sum(axis=(0, 2, 3))
    sb = np.abs(g).sum(axis=(0, 2, 3))
    f = gamma.reshape(1, -1, 1, 1) * rstd / mcount
    dx = f * (mcount * g - dbet.reshape(1, -1, 1, 1) - xh * dgam.reshape(1, -1, 1, 1))
    sdx = np.abs(f) * (mcount * np.abs(g) + sb.reshape(1, -1, 1, 1) + np.abs(xh) * sg.reshape(1, -1, 1, 1))
    return (dx, sdx), (dgam, sg), (dbet, sb)


class Teacher:
    """The GPU's stored tensors of worker 0's last step and the fp64
    reference gradients built from them."""

    def __init__(self, o, ctx, x, labels):
        self.o, self.x = o, x.astype(np.float64)
        self.shapes = R.shapes(o)
        self.cons = [[c for c, r in enumerate(o.layers) if r["in0"] == l or r["in1"] == l]
                     for l in range(len(o.layers))]
        self.A, self.D = {}, {}
        for l in range(len(o.layers)):
            try:
                self.A[l] = ctx.get_activation(0, l, self.shapes[l]).astype(np.float64)
            except lpp.LppError as e:
                assert e.code == lpp.ESTATE
            try:
                self.D[l] = ctx.get_activation_grad(0, l, self.shapes[l]).astype(np.float64)
            except lpp.LppError as e:
                assert e.code == lpp.ESTATE
        z = ctx.get_logits(0).astype(np.float64)
        p = np.exp(z - z.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        self.dz = (p - np.eye(z.shape[1])[labels]) / z.shape[0]
        self._memo = {}

    def params(self, rec, n, off=0):
        return self.x[rec["poff"] + off:rec["poff"] + off + n]

    def out_grad(self, l):
        """dL/d(output of l): the GPU's stored gradient if it is kept, else
        the reference from l's consumers (through fused-away layers)."""
        if l in self.D:
            return self.D[l], None
        return self.ref_grad(l)

    def ref_grad(self, l):
        """Reference dL/d(output of l) and its term-magnitude sum, from the
        stored gradients of l's consumers (one level, or through fused-away
        layers until stored ones)."""
        if l in self._memo:
            return self._memo[l]
        o, n_cls = self.o, self.o.n_classes
        tot = np.zeros((self.dz.shape[0],) + tuple(self.shapes[l]))
        mag = np.zeros_like(tot)
        if l == len(o.layers) - 1:
            tot[:] = self.dz.reshape(tot.shape)
            mag[:] = np.abs(tot)
        for c in self.cons[l]:
            rec = o.layers[c]
            op = rec["op"]
            if op == OM.CONV:
                k = rec["k"]
                W = self.params(rec, rec["cout"] * rec["cin"] * k * k).reshape(rec["cout"], rec["cin"], k, k)
                g, m = conv_data_grad(self.D[c], W, rec["stride"], rec["pad"], self.shapes[l][1:])
            elif op == OM.BN:
                gc, _ = self.out_grad(c)
                gam = self.params(rec, rec["cout"])
                (g, m), _, _ = bn_backward(self.A[l], gam, gc)
            elif op == OM.ADD:
                g, _ = self.out_grad(c)
                m = np.abs(g)
            elif op == OM.RELU:
                gc, _ = self.out_grad(c)
                g = np.where(self.A[c] > 0, gc, 0.0)
                m = np.abs(g)
            elif op == OM.GAP:
                gc, _ = self.out_grad(c)
                hw = self.shapes[l][1] * self.shapes[l][2]
                g = np.broadcast_to(gc / hw, tot.shape)
                m = np.abs(g)
            elif op == OM.LINEAR:
                W = self.params(rec, rec["cout"] * rec["cin"]).reshape(rec["cout"], rec["cin"])
                g = (self.dz @ W).reshape(tot.shape)
                m = (np.abs(self.dz) @ np.abs(W)).reshape(tot.shape)
            else:
                raise AssertionError("unexpected consumer %d" % op)
            tot += g
            mag += m
        self._memo[l] = (tot, mag)
        return tot, mag


def test_full_size_resnet20_backward_teacher_forced():
    """ResNet-20 with its ReLUs at batch 128, fused kernels (BN + ReLU folds
    active), sequential mode, partition 0.  For every layer whose gradient
    the GPU keeps, that gradient against the reference from its consumers'
    stored gradients; every conv's weight gradient from its stored input and
    output gradient; every BN's gamma and beta gradients from its stored
    input and the gradient reaching its output (through the group's ReLU
    with the GPU's own decisions and the residual add); the head's weight
    and bias gradients from the stored pooled features and logits."""
    o, p = OM.resnet20_p4(), PM.resnet20()
    x = T.init_x(o.specs, 87)
    img, lab = T.inputs(88, 128, o.in_shape, 10)
    with lpp.Context(p, K=1, batch=128) as ctx:
        ctx.set_params(x)
        ctx.timer_enable("bn_act")
        ctx.step(0, *dev(img, lab), 0, 0.0)
        _, launches, _ = ctx.timer_read()
        ctx.timer_enable(None)
        say("bn_act launches", launches, "of", sum(1 for r in o.layers if r["op"] == OM.BN), "BNs")
        assert launches <= 10                      # the folds are active
        tf = Teacher(o, ctx, x, lab)
        gpu_g = ctx.get_grad(0).astype(np.float64)
    checked = {"act": 0, "conv_w": 0, "bn": 0, "head": 0}
    worst = ("-", 0.0)

    def note(what, e):
        nonlocal worst
        if e > worst[1]:
            worst = (what, e)
        assert e < T.TOL_GRAD, (what, e)

    for l, rec in enumerate(o.layers):
        if l in tf.D and l != len(o.layers) - 1:
            ref, mag = tf.ref_grad(l)
            note("activation grad L%d" % l, T.relerr_scaled(tf.D[l], ref, mag))
            checked["act"] += 1
        op = rec["op"]
        if op == OM.CONV:
            k = rec["k"]
            X = img.astype(np.float64) if rec["in0"] < 0 else tf.A[rec["in0"]]
            g, m = conv_weight_grad(X, tf.D[l], rec["stride"], rec["pad"], k)
            n = g.size
            note("conv weight grad L%d" % l,
                 T.relerr_scaled(gpu_g[rec["poff"]:rec["poff"] + n], g.ravel(), m.ravel()))
            checked["conv_w"] += 1
        elif op == OM.BN:
            c = rec["cout"]
            gout, _ = tf.out_grad(l)
            _, (dg, sg), (db, sb) = bn_backward(tf.A[rec["in0"]], tf.params(rec, c), gout)
            note("bn gamma grad L%d" % l, T.relerr_scaled(gpu_g[rec["poff"]:rec["poff"] + c], dg, sg))
            note("bn beta grad L%d" % l, T.relerr_scaled(gpu_g[rec["poff"] + c:rec["poff"] + 2 * c], db, sb))
            checked["bn"] += 1
        elif op == OM.LINEAR:
            F = tf.A[rec["in0"]].reshape(128, -1)
            n = rec["cout"] * rec["cin"]
            note("linear weight grad", T.relerr_scaled(gpu_g[rec["poff"]:rec["poff"] + n], (tf.dz.T @ F).ravel(),
                                                       (np.abs(tf.dz).T @ np.abs(F)).ravel()))
            note("linear bias grad", T.relerr_scaled(gpu_g[rec["poff"] + n:rec["poff"] + n + rec["cout"]],
                                                     tf.dz.sum(axis=0), np.abs(tf.dz).sum(axis=0)))
            checked["head"] += 1
    say("teacher-forced checks", checked, "worst", worst)
    n_conv = sum(1 for r in o.layers if r["op"] == OM.CONV)
    n_bn = sum(1 for r in o.layers if r["op"] == OM.BN)
    assert checked["conv_w"] == n_conv and checked["bn"] == n_bn and checked["head"] == 1
    assert checked["act"] >= n_conv          # at least every conv output's gradient


def test_folded_bn_relu_with_clipping_all_partitions():
    """The folded BN + ReLU path (forward staging, weight-gradient staging,
    the data-gradient epilogue's BN sums with the ReLU mask) against the
    oracle where the ReLUs clip: ResNet-20 at batch 32 (the smallest batch
    at which its 32x32 and 16x16 stages take the spatial kernels that fold),
    BN shifts +4 on even and -4 on odd channels, so that the folded ReLUs
    zero about half of their inputs (all but a few of the odd channels')
    while every decision keeps a margin above the fp32 / fp64 disagreement
    (a ReLU input near 0 needs a normalised value near 4).  Every partition
    in sequential mode, two in async mode."""
    o, p = OM.resnet20_p4(), PM.resnet20()
    n = 32
    band = 1e-5

    def make(seed):
        x = T.init_x(o.specs, seed)
        for name, off, cnt in o.tensors:
            if name.endswith("bn_beta"):
                x[off:off + cnt] = np.where(np.arange(cnt) % 2 == 0, 4.0, -4.0)
        return x.astype(np.float64), T.inputs(seed + 7, n, o.in_shape, 10)[0]

    seed, margin = T.well_posed_seed(o, make, seeds=range(2600, 2640), band=band)
    x = make(seed)[0].astype(np.float32)
    img, lab = T.inputs(seed + 7, n, o.in_shape, 10)
    # clipping is real at every folded ReLU (one whose only consumer is a conv)
    fr = []
    for li, rec in enumerate(o.layers):
        cons = [r for r in o.layers if r["in0"] == li or r["in1"] == li]
        if rec["op"] == OM.RELU and len(cons) == 1 and cons[0]["op"] == OM.CONV:
            fr.append(float(np.mean(R.activation(o, x, img, rec["in0"]) < 0)))
    say("clipped folds seed", seed, "margin %.2e" % margin, "clipped fractions at the folded ReLUs",
        np.round(fr, 3))
    assert len(fr) == 9 and min(fr) > 0.4
    with lpp.Context(p, K=1, batch=n) as ctx:
        ctx.set_params(x)
        ctx.timer_enable("bn_act")
        ctx.step(0, *dev(img, lab), 1, 0.0)
        _, launches, _ = ctx.timer_read()
        ctx.timer_enable(None)
    say("bn_act launches per step", launches, "(19 BN + ReLU groups without folding)")
    assert launches <= 10
    m0 = (np.random.default_rng(9).standard_normal(o.d) * 1e-2).astype(np.float32)
    for part in range(0, 5):
        say("clipped folds, partition", part)
        _partition_step(o, p, x, m0, img, lab, part, band=band)
    for part in (0, 3):
        say("clipped folds, async partition", part)
        _partition_step(o, p, x, m0, img, lab, part, band=band, mode=lpp.ASYNC)


def _schedule_with_scales(o, x0, sched, batches, K, P, H, lr, mu):
    """The oracle's sequential schedule (as run_sequential: replica q's counter
    advances with each of its updates; an averaging round when every counter
    has advanced by H), also accumulating, per replica and parameter, the
    error scale of a trajectory: an fp32 gradient carries errors up to the
    gradient bar's floor, a fraction of C_e (the sum of the magnitudes of the
    products it sums, grad_scale), and a gradient error d at one step moves
    the parameter by at most lr * d / (1 - mu) over the momentum's later
    steps, so S_e = lr / (1 - mu) * (sum over the updates of e of C_e); an
    averaging round averages the replicas' errors, so their S as well.  The
    momentum's scale is (sum of C_e) / (1 - mu)."""
    reps = [x0.copy() for _ in range(K)]
    moms = [np.zeros(o.d) for _ in range(K * P)]
    S = [np.zeros(o.d) for _ in range(K)]
    SM = [np.zeros(o.d) for _ in range(K * P)]
    counters, s_pre = [0] * K, 0
    for (w, part, key) in sched:
        q = w // P
        counters[q] += 1
        img, lab = batches[key]
        g, sc = R.grad_scale(o, reps[q], img, lab)
        lo, hi = o.block_range(part)
        gb = np.zeros(o.d)
        gb[lo:hi] = g[lo:hi]
        R.block_update(reps[q], moms[w], gb, lo, hi, lr, mu)
        S[q][lo:hi] += lr / (1.0 - mu) * sc[lo:hi]
        SM[w][lo:hi] += sc[lo:hi] / (1.0 - mu)
        if min(counters) - s_pre >= H:
            s_pre = min(counters)
            R.average(reps)
            sbar = np.mean(S, axis=0)
            S = [sbar.copy() for _ in range(K)]
    return reps, moms, S, SM


def test_resnet20_100_k4_h8_cadence():
    """The ResNet-20-100 workload's schedule: K = 4 replicas x P = 4 workers,
    momentum 0.9, an averaging round whenever every replica's counter has
    advanced by H = 8; 80 updates issued round-robin over the 16 workers
    (two averaging rounds, at 32 and 64 updates), batch 8, against the
    oracle's sequential schedule (run_sequential, reproduced bit for bit by
    the scale-tracking replay below).  ReLU-free twin, so the trajectory is
    well posed.  Parameters and momenta are compared in the C_e measure with
    the trajectory's accumulated scale: gradients of cancelling sums (the
    stem BN's shift, whose every path meets a later BN) are fp32 noise of
    order 1e-6 C_e at every step, and that noise accumulates over the run."""
    o, p = OM.resnet20_p4(100, relu=False), PM.resnet20(100, act=False)
    K, P, H, n_upd, n = 4, 4, 8, 80, 8
    x0 = T.init_x(o.specs, 77)
    sched, batches = [], {}
    for s in range(n_upd):
        w = s % (K * P)
        batches[s] = T.inputs(400 + s, n, o.in_shape, 100)
        sched.append((w, w % P + 1, s))
    reps, moms, _ = R.run_sequential(o, x0.astype(np.float64), sched, batches, K, P, H, 0.05, 0.9)
    reps2, moms2, S, SM = _schedule_with_scales(o, x0.astype(np.float64), sched, batches, K, P, H, 0.05, 0.9)
    for q in range(K):
        assert np.array_equal(reps[q], reps2[q])
    rounds = 0
    with lpp.Context(p, K=K, batch=n, momentum=0.9) as ctx:
        ctx.set_params(x0)
        s_pre = 0
        for (w, part, key) in sched:
            ctx.step(w, *dev(*batches[key]), part, 0.05)
            c = min(ctx.counter(q) for q in range(K))
            if c - s_pre >= H:
                s_pre = c
                ctx.average()
                rounds += 1
        assert rounds == 2
        assert [ctx.counter(q) for q in range(K)] == [n_upd // K] * K
        worst = ("-", 0.0)
        for q in range(K):
            errs = T.tensor_errors(o, ctx.get_params(q), reps[q], scale=S[q])
            worst = max(worst, T.worst(errs), key=lambda t: t[1])
            assert max(errs.values()) < T.TOL_PARAM, (q, T.worst(errs))
        for w in range(K * P):
            lo, hi = o.block_range(w % P + 1)
            errs = T.tensor_errors(o, ctx.get_momentum(w), moms[w], lo, hi, scale=SM[w])
            assert max(errs.values()) < T.TOL_PARAM, (w, T.worst(errs))
        say("K=4 H=8 cadence: worst parameter error", worst)

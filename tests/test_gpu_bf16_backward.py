"""The bf16 workloads' batch-norm backward at full size, teacher-forced.

With ReLUs, the bf16 path and the fp64 oracle take different decisions on
inputs near zero, so the oracle's own backward is no reference for the
whole network (the same holds for fp32 at the headline size; see
test_gpu_parity_headline).  Here every batch norm's backward is checked from
the GPU's own stored tensors: its input x, the gradient reaching its output
(through the group's ReLU with the GPU's stored decisions and through the
residual add), and gamma; the references are Sec. 2's chain rule through
training-mode batch norm in fp64 (tests/test_gpu_parity_headline:
bn_backward).  Checked per BN: dgamma and dbeta (fp32 results of sums over
the stored bf16 gradient: bar 1e-3 in the C_e measure of tests/parity.py),
and the stored bf16 gradient at the BN input against the sum over its
consumers (bar 2^-7 in the same measure: the one rounding of the stored
value to 8 significant bits is up to 2^-8 relative, and the fp32 arithmetic
before it stays below 1e-3 of the measure's floor 1e-2 C_e).  Sequential mode merges
the sums from fixed-order partials, async mode through fp64 atomics."""
import sys
import time

import numpy as np
import pytest

import synth
from oracle import lppref as R
from oracle import models as OM
from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM
from tests import parity as T
from tests.test_gpu_parity_headline import Teacher, bn_backward

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL_STORED = 2.0 ** -7


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.init()


def dev(img, lab):
    return (torch.from_numpy(np.ascontiguousarray(img)).cuda(),
            torch.from_numpy(np.ascontiguousarray(lab, np.int32)).cuda())


class _Lazy(dict):
    """The GPU's stored tensors, read on first use and kept until drop();
    a tensor that is fused away (ESTATE) is absent."""

    def __init__(self, get, shapes):
        super().__init__()
        self._get, self._shapes, self._missing = get, shapes, set()

    def _load(self, l):
        if l in self._missing:
            return False
        if dict.__contains__(self, l):
            return True
        try:
            v = self._get(l, self._shapes[l]).astype(np.float64)
        except lpp.LppError as e:
            assert e.code == lpp.ESTATE
            self._missing.add(l)
            return False
        dict.__setitem__(self, l, v)
        return True

    def __contains__(self, l):
        return self._load(l)

    def __getitem__(self, l):
        if not self._load(l):
            raise KeyError(l)
        return dict.__getitem__(self, l)

    def drop(self):
        dict.clear(self)


class LazyTeacher(Teacher):
    """Teacher over tensors fetched per use (the full-size bf16 networks do
    not fit in host memory as fp64 all at once)."""

    def __init__(self, o, ctx, x, labels):
        self.o, self.x = o, x.astype(np.float64)
        self.shapes = R.shapes(o)
        self.cons = [[c for c, r in enumerate(o.layers) if r["in0"] == l or r["in1"] == l]
                     for l in range(len(o.layers))]
        self.A = _Lazy(lambda l, s: ctx.get_activation(0, l, s), self.shapes)
        self.D = _Lazy(lambda l, s: ctx.get_activation_grad(0, l, s), self.shapes)
        z = ctx.get_logits(0).astype(np.float64)
        p = np.exp(z - z.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        self.dz = (p - np.eye(z.shape[1])[labels]) / z.shape[0]
        self._memo = {}

    def drop(self):
        self.A.drop()
        self.D.drop()
        self._memo.clear()


CASES = {
    # name: (oracle model, library model, batch) -- the workloads' own batches
    "wrn16_8": (OM.wrn16_8_p4, PM.wrn16_8, 128),
    "resnet18": (OM.resnet18_p4, PM.resnet18, 128),
    "resnet50": (OM.resnet50_p4, PM.resnet50, 32),
}


@pytest.mark.parametrize("which,mode", [("wrn16_8", lpp.SEQUENTIAL), ("resnet18", lpp.SEQUENTIAL),
                                        ("resnet50", lpp.SEQUENTIAL), ("wrn16_8", lpp.ASYNC)],
                         ids=["wrn16_8", "resnet18", "resnet50", "wrn16_8-async"])
def test_bf16_bn_backward_teacher_forced(which, mode):
    mo, mp, n = CASES[which]
    o, p = mo(), mp()
    x = T.init_x(o.specs, 3051)
    img, lab = T.inputs(3052, n, o.in_shape, o.n_classes)
    img = synth.round_to_bf16(np.asarray(img, np.float32))
    say(which, "batch", n, "mode", mode)
    with lpp.Context(p, K=1, batch=n, dtype=lpp.BF16, mode=mode, momentum=0.9) as ctx:
        ctx.set_params(x)
        ctx.step(0, *dev(img, lab), 0, 0.0)
        tf = LazyTeacher(o, ctx, x, lab)
        gpu_g = ctx.get_grad(0).astype(np.float64)
        worst = {"gamma/beta": ("-", 0.0), "dx": ("-", 0.0)}
        checked = {"bn": 0, "dx": 0}
        t0 = time.time()
        for l, rec in enumerate(o.layers):
            if rec["op"] != OM.BN:
                continue
            c = rec["cout"]
            gout, _ = tf.out_grad(l)
            _, (dg, sg), (db, sb) = bn_backward(tf.A[rec["in0"]], tf.params(rec, c), gout)
            for what, got, ref, mag in (("gamma", gpu_g[rec["poff"]:rec["poff"] + c], dg, sg),
                                        ("beta", gpu_g[rec["poff"] + c:rec["poff"] + 2 * c], db, sb)):
                e = T.relerr_scaled(got, ref, mag)
                if e > worst["gamma/beta"][1]:
                    worst["gamma/beta"] = ("%s L%d" % (what, l), e)
                assert e < T.TOL_GRAD, (what, l, e)
            checked["bn"] += 1
            src = rec["in0"]
            if src >= 0 and src in tf.D:
                ref, mag = tf.ref_grad(src)
                e = T.relerr_scaled(tf.D[src], ref, mag)
                if e > worst["dx"][1]:
                    worst["dx"] = ("L%d" % src, e)
                assert e < TOL_STORED, ("dx", src, e)
                checked["dx"] += 1
            tf.drop()
        say("  checked", checked, "worst", worst, "(%.0f s)" % (time.time() - t0))
        assert checked["bn"] == sum(1 for r in o.layers if r["op"] == OM.BN)
        assert checked["dx"] > 0

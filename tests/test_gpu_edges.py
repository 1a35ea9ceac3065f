"""Degenerate configurations of the method on the HIP path, against the fp64
oracle: a batch of one image (every tile ragged, batch-norm-free model), a
single block (P = 1: the partial backward is the full one), averaging a
single replica (the identity, bit for bit), and the step's argument checks
(a rejected call launches nothing and leaves the context usable)."""
import sys

import numpy as np
import pytest

from oracle import lppref as R
from oracle import models as OM
from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM
from tests import parity as T
from tests.test_gpu_parity import _partition_step, dev, grid_conv_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.init()


def _tiny_seed(o, n, band=8e-7):
    """An exact-grid input set of n images whose ReLU decisions all keep the
    margin `band` (chosen by the oracle)."""
    return T.well_posed_seed(o, lambda s: grid_conv_inputs(o, s, n)[:2], seeds=range(300, 400), band=band)


@pytest.mark.parametrize("partition", [0, 1, 2])
def test_batch_of_one(partition):
    """Tiny CNN at batch 1: 32x32 maps, every reduction over a single image."""
    o, p = OM.tiny_p2(), PM.tiny_cnn()
    seed, margin = _tiny_seed(o, 1)
    say("batch 1 seed", seed, "margin %.2e" % margin)
    x, img, lab = grid_conv_inputs(o, seed, 1)
    m0 = (np.random.default_rng(seed).standard_normal(o.d) * 1e-2).astype(np.float32)
    _partition_step(o, p, x.astype(np.float32), m0, img, lab, partition, band=8e-7)


def test_single_block_is_the_full_step():
    """P = 1: the only block is the whole model, so partition 1 must give the
    full gradient bit for bit and match the oracle."""
    o = OM.tiny().set_blocks([1, 1])
    p = PM.tiny_cnn().assign_blocks([1, 1])
    assert o.P == 1 and p.P == 1
    seed, _ = _tiny_seed(o, 4)
    x, img, lab = grid_conv_inputs(o, seed, 4)
    x = x.astype(np.float32)
    m0 = np.zeros(o.d, np.float32)
    _partition_step(o, p, x, m0, img, lab, 1, band=8e-7)
    with lpp.Context(p, K=1, batch=4) as ctx:
        assert ctx.block_range(1) == (0, o.d)
        ctx.set_params(x)
        ti, tl = dev(img, lab)
        ctx.step(0, ti, tl, 0, 0.0)
        g0 = ctx.get_grad(0)
        ctx.step(0, ti, tl, 1, 0.0)
        assert np.array_equal(ctx.get_grad(0), g0)


def test_single_replica_average_is_identity():
    """Averaging one replica (and the averaging kernel on one array) leaves it
    unchanged bit for bit; with two replicas the library's rounds match the
    oracle's average."""
    o, p = OM.tiny_p2(), PM.tiny_cnn()
    rng = np.random.default_rng(5)
    x = rng.standard_normal(o.d).astype(np.float32)
    with lpp.Context(p, K=2, batch=2) as ctx:
        ctx.set_params(x, 0)
        ctx.set_params(-x, 1)
        ctx.average([0])
        ctx.sync()
        assert np.array_equal(ctx.get_params(0), x)
        assert np.array_equal(ctx.get_params(1), -x)
    t = torch.from_numpy(x.copy()).cuda()
    lpp.kernel_average([t])
    torch.cuda.synchronize()
    assert np.array_equal(t.cpu().numpy(), x)


def test_step_argument_checks_leave_the_context_usable():
    """A step with a wrong batch size, worker or partition is rejected with
    LPP_EINVAL before anything is launched; the replica is untouched and the
    next valid step still matches the oracle."""
    o, p = OM.tiny_p2(), PM.tiny_cnn()
    seed, _ = _tiny_seed(o, 4)
    x, img, lab = grid_conv_inputs(o, seed, 4)
    x = x.astype(np.float32)
    g_ref, _, logits = R.step(o, x.astype(np.float64), None, img, lab, 2, 0.1)
    with lpp.Context(p, K=1, batch=4) as ctx:
        ctx.set_params(x)
        ti, tl = dev(img, lab)
        bad = [(lambda: ctx.step(0, ti[:3], tl[:3], 1, 0.1)),   # batch 3 on a batch-4 context
               (lambda: ctx.step(2, ti, tl, 1, 0.1)),           # worker 2 of 2
               (lambda: ctx.step(0, ti, tl, 3, 0.1)),           # partition 3 of P = 2
               (lambda: ctx.step(-1, ti, tl, 1, 0.1))]
        for call in bad:
            with pytest.raises(lpp.LppError) as e:
                call()
            assert e.value.code == lpp.EINVAL, e.value
        ctx.sync()
        assert np.array_equal(ctx.get_params(0), x)
        assert ctx.counter(0) == 0
        ctx.step(1, ti, tl, 2, 0.1)
        assert T.relerr(ctx.get_logits(1), logits, T.TAU_LOGITS) < T.TOL_LOGITS
        lo, hi = o.block_range(2)
        assert T.relerr(ctx.get_grad(1)[lo:hi], g_ref[lo:hi]) < T.TOL_GRAD
        assert ctx.counter(0) == 1

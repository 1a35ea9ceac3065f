"""The host-side LPP-SGD policy driving the HIP library (GPU).

Sequential mode: a policy-driven run over K replicas x P workers (warm-up
phase of full-model steps, then full model / own block alternating, K_j = 1
then H, warm-up + cosine learning rate, momentum) is replayed step by step
by the fp64 oracle (the same plan: worker, partition, learning rate, batch,
averaging rounds); every replica's parameters must agree at the 1e-3 bar.
ReLU-free ResNet-20 twin, so the multi-step trajectory is well posed.
Async mode: the same policy on the real ResNet-20 trains (loss curve falls).
"""
import sys

import numpy as np
import pytest

from oracle import lppref as R
from oracle import models as OM
from paper_2203_06638_amd import lpp
from paper_2203_06638_amd import models as PM
from paper_2203_06638_amd import policy as PL
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


def test_policy_run_matches_oracle_replay():
    o, p = OM.resnet20_p4(10, relu=False), PM.resnet20(10, act=False)
    K, P, mu = 2, 4, 0.9
    sched = PL.Schedule(T=12, T_st=3, H=4, base_lr=0.02, warm_lr=0.05, warmup=4)
    x0 = T.init_x(o.specs, 501)
    host = [T.inputs(510 + b, 4, o.in_shape, 10) for b in range(5)]
    pool = [dev(*b) for b in host]
    # the oracle replays the plan
    pl = PL.plan(sched, K, P)
    reps = [x0.astype(np.float64) for _ in range(K)]
    moms = [np.zeros(o.d) for _ in range(K * P)]
    n = 0
    for e in pl.events:
        if e[0] == "average":
            R.average(reps)
            continue
        _, w, part, lr, _s = e
        img, lab = host[n % len(host)]
        R.step(o, reps[w // P], moms[w], img, lab, part, lr, mu)
        n += 1
    parts = {e[2] for e in pl.steps}
    say("partitions used", sorted(parts), "averaging rounds", sum(1 for e in pl.events if e[0] == "average"))
    assert parts == {0, 1, 2, 3, 4}
    with lpp.Context(p, K=K, batch=4, momentum=mu) as ctx:
        ctx.set_params(x0)
        pl2, curve = PL.run(ctx, pool, sched)
        assert pl2.events == pl.events
        assert [ctx.counter(q) for q in range(K)] == [sched.T] * K
        for q in range(K):
            errs = T.tensor_errors(o, ctx.get_params(q), reps[q])
            say("replica", q, "worst", T.worst(errs))
            assert max(errs.values()) < T.TOL_PARAM, (q, T.worst(errs))


def test_policy_async_training_curve():
    p = PM.resnet20()
    K, P = 1, 4
    sched = PL.Schedule(T=160, T_st=16, H=8, base_lr=0.05, warm_lr=0.125, warmup=16)
    x = T.init_x(p.specs, 601)
    pool = [dev(*T.inputs(602 + b, 32, p.in_shape, 10)) for b in range(4)]
    with lpp.Context(p, K=K, batch=32, mode=lpp.ASYNC, momentum=0.9) as ctx:
        ctx.set_params(x)
        pl, curve = PL.run(ctx, pool, sched, log_every=40)
        say("loss curve", [(n, round(l, 4)) for n, l in curve])
        assert ctx.counter(0) == sched.T
        assert all(np.isfinite(l) for _, l in curve)
        assert curve[-1][1] < curve[0][1]
        xn = ctx.get_params(0)
        for i in range(1, P + 1):
            lo, hi = ctx.block_range(i)
            assert not np.array_equal(xn[lo:hi], x[lo:hi])


# ---------------------------------------------------------------------------
# step tracing: the orders of the delay model observed on the device
# ---------------------------------------------------------------------------

def _traced_run(p, K, P, sched, pool, mode, x, trace):
    with lpp.Context(p, K=K, batch=pool[0][0].shape[0], momentum=0.9, mode=mode) as ctx:
        ctx.set_params(x)
        if trace:
            ctx.trace_enable(4096)
        PL.run(ctx, pool, sched)
        tr = ctx.trace_read() if trace else None
        return [ctx.get_params(q) for q in range(K)], tr


def test_trace_sequential_orders_and_no_effect_on_results():
    from paper_2203_06638_amd import delays as D
    p = PM.resnet20()
    K, P = 2, 4
    sched = PL.Schedule(T=16, T_st=4, H=2, base_lr=0.02, warm_lr=0.05, warmup=4)
    x = T.init_x(p.specs, 701)
    pool = [dev(*T.inputs(702 + b, 8, p.in_shape, 10)) for b in range(3)]
    plain, _ = _traced_run(p, K, P, sched, pool, lpp.SEQUENTIAL, x, False)
    traced, (steps, rounds, khz) = _traced_run(p, K, P, sched, pool, lpp.SEQUENTIAL, x, True)
    for q in range(K):
        assert np.array_equal(plain[q], traced[q])                # tracing changes nothing
    pl = PL.plan(sched, K, P)
    assert len(steps) == len(pl.steps) and len(rounds) == sum(1 for e in pl.events if e[0] == "average")
    assert khz > 0
    for s, e in zip(steps, pl.steps):
        assert (s["worker"], s["partition"]) == (e[1], e[2]) and s["counter"] == e[4]
        assert s["t"][0] <= s["t"][1] <= s["t"][2] <= s["t"][3]
    # sequential: nothing overlaps, in issue order
    evs = sorted([tuple(s["t"][::3]) for s in steps] + [tuple(r["t"]) for r in rounds])
    assert all(evs[i][1] <= evs[i + 1][0] for i in range(len(evs) - 1))
    ann, summ = D.analyze(steps, rounds)
    say("sequential trace", summ)
    assert summ["staleness_max"] == 0 and summ["p_good"] == 1.0 and summ["order_inversions"] == 0


def test_trace_async_delay_statistics():
    from paper_2203_06638_amd import delays as D
    p = PM.resnet20()
    K, P = 2, 4
    x = T.init_x(p.specs, 711)
    pool = [dev(*T.inputs(712 + b, 32, p.in_shape, 10)) for b in range(4)]
    for H in (1, 8):
        sched = PL.Schedule(T=48, T_st=4, H=H, base_lr=0.02, warm_lr=0.05, warmup=4)
        _, (steps, rounds, khz) = _traced_run(p, K, P, sched, pool, lpp.ASYNC, x, True)
        assert len(steps) == K * sched.T
        assert all(s["t"][0] <= s["t"][1] <= s["t"][2] <= s["t"][3] for s in steps)
        assert all(r["t"][0] <= r["t"][1] for r in rounds)
        ann, summ = D.analyze(steps, rounds)
        # Alg. 1: the averager runs concurrently with the updaters.  Rounds
        # whose kernel interval overlaps an updater iteration (snapshot start
        # to update end) of some worker, and overlaps a block update itself.
        ov_iter = sum(1 for r in rounds if any(s["t"][0] < r["t"][1] and r["t"][0] < s["t"][3] for s in steps))
        ov_upd = sum(1 for r in rounds if any(s["t"][2] < r["t"][1] and r["t"][0] < s["t"][3] for s in steps))
        say("async trace H=%d" % H, summ, "rounds overlapping an iteration %d, an update %d of %d"
            % (ov_iter, ov_upd, len(rounds)))
        assert 0.0 <= summ["p_good"] <= 1.0 and summ["staleness_max"] >= 0
        assert ov_iter >= 1, "no averaging round ran concurrently with an updater"

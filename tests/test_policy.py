"""The host-side LPP-SGD policy (paper_2203_06638_amd/policy.py) against the
paper's statements (Sec. 3 "Block Selection Rule", "Discussion on the Rule",
"Synchronization Frequency Scheme"; Sec. 4 hyperparameters).  CPU only."""
import math

import pytest

from paper_2203_06638_amd import policy as PL


def test_warmup_phase_takes_the_full_model():
    s = PL.Schedule(T=100, T_st=10)
    for w in range(8):
        for c in range(0, 11):
            assert PL.partition(s, w, 4, c, 0) == 0


def test_after_warmup_full_model_and_own_block_alternate():
    s = PL.Schedule(T=100, T_st=10)
    for w in range(8):
        got = [PL.partition(s, w, 4, 50, i) for i in range(6)]
        assert got == [0, w % 4 + 1] * 3


def test_lap_sgd_always_takes_the_full_model():
    s = PL.Schedule(T=100, T_st=10, lpp=False)
    assert {PL.partition(s, w, 4, c, i) for w in range(4) for c in range(100) for i in range(3)} == {0}


@pytest.mark.parametrize("T,K,P", [(400, 1, 4), (800, 2, 4), (1000, 4, 4), (300, 1, 6)])
def test_about_nine_twentieths_of_the_iterations_are_partial(T, K, P):
    """With T_st = T/10 the rule performs partial gradient computation in
    about 9T/20 of the iterations (Sec. 3, "Discussion on the Rule")."""
    s = PL.Schedule(T=T, T_st=T // 10)
    steps = PL.plan(s, K, P).steps
    assert len(steps) == K * T                       # exactly T updates per replica
    partial = sum(1 for e in steps if e[2] != 0)
    assert abs(partial - K * 9 * T / 20) <= K * P, (partial, K * 9 * T / 20)
    # every updater steps only on the full model or on its own block
    assert all(e[2] in (0, e[1] % P + 1) for e in steps)


def test_counters_and_replica_membership():
    s = PL.Schedule(T=37, T_st=3)
    steps = PL.plan(s, 3, 4).steps
    for q in range(3):
        cs = [e[4] for e in steps if e[1] // 4 == q]
        assert cs == list(range(37))                 # the replica's counter values, each once


def test_synchronization_frequency_scheme():
    """K_j = 1 until the counter reaches T/2, then H: with P workers per
    replica stepping in turn, a round after every pass of P updates while
    s < T/2, then after every H updates per replica."""
    T, K, P, H = 64, 2, 4, 8
    s = PL.Schedule(T=T, T_st=6, H=H)
    assert PL.sync_interval(s, T // 2 - 1) == 1 and PL.sync_interval(s, T // 2) == H
    ev = PL.plan(s, K, P).events
    counter, last, gaps = 0, 0, []
    for e in ev:
        if e[0] == "step" and e[1] // P == 0:
            counter += 1
        elif e[0] == "average":
            gaps.append((last, counter - last))
            last = counter
    for start, gap in gaps:
        assert gap >= PL.sync_interval(s, start + gap)
    # rounds at counters 4, 8, ..., 28 (K_j = 1); at 32 = T/2 the interval is
    # already H, so the next rounds come at 36, 44, 52, 60
    assert [st + g for st, g in gaps] == [4, 8, 12, 16, 20, 24, 28, 36, 44, 52, 60]


def test_learning_rate_warmup_then_cosine():
    s = PL.Schedule(T=1000, T_st=100, base_lr=0.1, warm_lr=0.25, warmup=50)
    assert PL.learning_rate(s, 0) == pytest.approx(0.1)
    assert PL.learning_rate(s, 25) == pytest.approx(0.175)
    assert PL.learning_rate(s, 50) == pytest.approx(0.25)
    assert PL.learning_rate(s, 50 + 475) == pytest.approx(0.125)       # cosine midpoint
    assert PL.learning_rate(s, 1000) == pytest.approx(0.0, abs=1e-12)
    lrs = [PL.learning_rate(s, c) for c in range(50, 1001)]
    assert all(a >= b for a, b in zip(lrs, lrs[1:]))
    # the cosine shape itself
    for c in (100, 300, 700):
        assert PL.learning_rate(s, c) == pytest.approx(0.125 * (1 + math.cos(math.pi * (c - 50) / 950)))


class _FakeCtx:
    """Records the calls the driver makes (no GPU)."""

    def __init__(self, K, P):
        self.K, self.P = K, P
        self.calls = []
        self.count = [0] * K

    def step(self, w, img, lab, p, lr):
        self.calls.append(("step", w, p, lr, img))
        self.count[w // self.P] += 1

    def average(self):
        self.calls.append(("average",))

    def get_loss(self, w):
        return 1.0

    def sync(self):
        pass


def test_driver_issues_the_plan():
    s = PL.Schedule(T=20, T_st=2, H=4, warmup=3)
    ctx = _FakeCtx(2, 4)
    pl, curve = PL.run(ctx, [("b0", None), ("b1", None)], s, log_every=8)
    assert ctx.count == [20, 20]
    got = [c[:4] if c[0] == "step" else c for c in ctx.calls]
    want = [e[:4] if e[0] == "step" else e for e in pl.events]
    assert got == want
    assert [c[4] for c in ctx.calls if c[0] == "step"][:3] == ["b0", "b1", "b0"]
    assert curve[-1] == (40, 1.0) and len(curve) == 6

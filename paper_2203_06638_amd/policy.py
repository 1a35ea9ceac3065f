"""Host-side LPP-SGD training policy on top of the C ABI (lpp_step,
lpp_average): which block each updater steps on, how often the replicas are
averaged, and the learning rate -- all decided on the host; every step of
the hot path still runs in the library.

From the paper (Sec. 3):
  * Block selection rule: while the iteration counter s read by an updater
    (Alg. 1) is at most T_st, the updater takes the full model (partition 0);
    after that it alternates between the full model and its own block
    rank(u) = worker % P + 1, one iteration each.  With T_st about T/10,
    about 9T/20 of the iterations are partial ("Discussion on the Rule").
  * LAP-SGD is the same loop with the full model in every iteration.
  * Synchronization frequency scheme: K_j = 1 until the counter reaches T/2,
    then K_j = H (post-local-SGD style).
  * Learning rate (Sec. 4, hyperparameters): linear warm-up from the base
    rate to the warmed-up rate over the first epochs, then cosine annealing
    to zero without restarts; for LPP-SGD the warmed-up rate is 1.25x that
    of LAP-SGD.

Readings where the paper leaves room: "alternate iterations" alternate on
the updater's own iteration count after the warm-up phase, starting with the
full model; an averaging round over the K co-resident replicas runs when
every replica's counter has advanced by K_j since the last round; the run
stops after exactly T updates per replica.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field


@dataclass
class Schedule:
    T: int                      # updates per replica (minibatches processed)
    T_st: int                   # warm-up phase of full-model steps
    H: int = 8                  # synchronization period after T/2
    base_lr: float = 0.1        # rate at the start of the warm-up
    warm_lr: float = 0.25       # warmed-up rate (LPP: 1.25x the LAP value)
    warmup: int = 0             # warm-up length in updates
    lpp: bool = True            # False: LAP-SGD (always the full model)


def partition(sched: Schedule, worker: int, P: int, s: int, local_iter: int) -> int:
    """Block for an updater that read counter value s (0-based: the s-th
    update of its replica) on its local_iter-th own iteration."""
    if not sched.lpp or s <= sched.T_st:
        return 0
    return 0 if local_iter % 2 == 0 else worker % P + 1


def sync_interval(sched: Schedule, s: int) -> int:
    """K_j for a replica whose counter reads s."""
    return 1 if s < sched.T // 2 else sched.H


def learning_rate(sched: Schedule, s: int) -> float:
    """Linear warm-up base_lr -> warm_lr over `warmup` updates, then cosine
    annealing from warm_lr to 0 at s = T."""
    if sched.warmup > 0 and s < sched.warmup:
        return sched.base_lr + (sched.warm_lr - sched.base_lr) * s / sched.warmup
    span = max(1, sched.T - sched.warmup)
    x = min(1.0, (s - sched.warmup) / span)
    return 0.5 * sched.warm_lr * (1.0 + math.cos(math.pi * x))


@dataclass
class Plan:
    """The events of a run, in issue order: ("step", worker, partition, lr,
    counter) and ("average",)."""
    events: list = field(default_factory=list)

    @property
    def steps(self):
        return [e for e in self.events if e[0] == "step"]


def plan(sched: Schedule, K: int, P: int) -> Plan:
    """The issue order of a whole run: workers round-robin (replicas in
    turn, workers of a replica in rank order), exactly T updates per
    replica, averaging rounds by the synchronization scheme."""
    out = Plan()
    counters = [0] * K
    local = [0] * (K * P)
    since = [0] * K
    while min(counters) < sched.T:
        for q in range(K):
            for r in range(P):
                if counters[q] >= sched.T:
                    continue
                w = q * P + r
                s = counters[q]                   # s := read&inc(C^q)
                counters[q] += 1
                since[q] += 1
                p = partition(sched, w, P, s, local[w])
                if not sched.lpp or s > sched.T_st:
                    local[w] += 1
                out.events.append(("step", w, p, learning_rate(sched, s), s))
        # Alg. 1 averager: s_cur - s_pre >= K_j, K_j chosen by s_cur
        if K > 1 and all(since[q] >= sync_interval(sched, counters[q]) for q in range(K)):
            out.events.append(("average",))
            since = [0] * K
    return out


def run(ctx, batches, sched: Schedule, log_every: int = 0):
    """Drives an lpp.Context through plan(sched, K, P).  batches is a list of
    (images, labels) device tensors, cycled per step.  Returns the plan and
    the loss curve [(update index, mean loss over workers)] read every
    log_every steps (0: only at the end)."""
    K, P = ctx.K, ctx.P
    pl = plan(sched, K, P)
    curve = []
    n = 0
    for e in pl.events:
        if e[0] == "average":
            ctx.average()
            continue
        _, w, p, lr, _s = e
        img, lab = batches[n % len(batches)]
        ctx.step(w, img, lab, p, lr)
        n += 1
        if log_every and n % log_every == 0:
            curve.append((n, sum(ctx.get_loss(v) for v in range(K * P)) / (K * P)))
    ctx.sync()
    curve.append((n, sum(ctx.get_loss(v) for v in range(K * P)) / (K * P)))
    return pl, curve

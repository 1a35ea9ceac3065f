"""Delay statistics of a traced run (lpp_trace_enable / lpp_trace_read): the
orders and the delay event of the paper's convergence model (Sec. 5 and the
appendix), measured on the device.

Per step i of replica q the trace gives the interval [a_i, b_i] that contains
its snapshot and [c_i, d_i] that contains its block update (device clock);
per averaging round r the interval [e_r, f_r] of its averaging kernel.
  * snapshot order: the counter value C^q the step read (Alg. 1);
  * update order: the rank of c_i among the updates of replica q;
  * iteration order (j, t): j = averaging rounds finished before c_i, t = the
    step's position among replica q's steps with the same j;
  * staleness: the number of other updates of replica q that can have
    written into the model between the start of step i's snapshot and the
    start of its own update (d_j > a_i and c_j < c_i) -- the number of
    minor iterations its snapshot may lag behind;
  * good iterate (Assumption 1): every component of the snapshot was read
    after the latest synchronization round before the update finished
    writing: with r the last round that began before c_i, a_i > f_r (or no
    round yet).  The fraction of good iterates estimates p-bar of
    Assumption 1.
Intervals are bracketed by timestamp kernels on the same stream, so they
contain the kernels they bracket; the conditions above are therefore
conservative (a step is counted good only if it surely was).
"""
from __future__ import annotations

import bisect


def analyze(steps, rounds):
    """steps: dicts with replica, counter, t = [a, b, c, d]; rounds: dicts
    with t = [e, f].  Returns per-step annotations and a summary."""
    rounds = sorted(rounds, key=lambda r: r["t"][0])
    r_start = [r["t"][0] for r in rounds]
    r_end_sorted = sorted(r["t"][1] for r in rounds)
    by_rep = {}
    for i, s in enumerate(steps):
        by_rep.setdefault(s["replica"], []).append(i)
    ann = [dict() for _ in steps]
    for q, idx in by_rep.items():
        order = sorted(idx, key=lambda i: steps[i]["t"][2])
        for rank, i in enumerate(order):
            ann[i]["update_order"] = rank
        for i in idx:
            a, _, c, _ = steps[i]["t"]
            ann[i]["staleness"] = sum(1 for j in idx if j != i and steps[j]["t"][3] > a and steps[j]["t"][2] < c)
            k = bisect.bisect_left(r_start, c) - 1          # last round that began before the update
            ann[i]["good"] = k < 0 or a > rounds[k]["t"][1]
            ann[i]["major"] = bisect.bisect_left(r_end_sorted, c)   # rounds finished before the update
        minor = {}
        for i in order:
            j = ann[i]["major"]
            ann[i]["minor"] = minor.get(j, 0)
            minor[j] = ann[i]["minor"] + 1
    n = len(steps)
    st = [a["staleness"] for a in ann]
    inv = 0
    for q, idx in by_rep.items():
        snap = sorted(idx, key=lambda i: steps[i]["counter"])
        upd = [ann[i]["update_order"] for i in snap]
        inv += sum(1 for x in range(len(upd)) for y in range(x + 1, len(upd)) if upd[x] > upd[y])
    summary = {
        "steps": n,
        "rounds": len(rounds),
        "p_good": (sum(1 for a in ann if a["good"]) / n) if n else None,
        "staleness_mean": (sum(st) / n) if n else None,
        "staleness_max": max(st) if st else None,
        "staleness_hist": {k: st.count(k) for k in sorted(set(st))},
        "order_inversions": inv,
    }
    return ann, summary

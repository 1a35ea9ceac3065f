"""Delay statistics of traced runs (paper_2203_06638_amd/delays.py) on
hand-built timelines whose orders, staleness and good-iterate events are
known (CPU only)."""
from paper_2203_06638_amd import delays as D


def st(rep, counter, a, b, c, d):
    return dict(replica=rep, counter=counter, t=[a, b, c, d])


def test_sequential_timeline():
    steps = [st(0, k, 10 * k, 10 * k + 2, 10 * k + 5, 10 * k + 7) for k in range(5)]
    ann, s = D.analyze(steps, [])
    assert [a["update_order"] for a in ann] == list(range(5))
    assert s["staleness_max"] == 0 and s["p_good"] == 1.0 and s["order_inversions"] == 0
    assert [a["major"] for a in ann] == [0] * 5 and [a["minor"] for a in ann] == list(range(5))


def test_overlapping_updates_are_stale():
    # step 1 snapshots while step 0's update is running; step 2 snapshots
    # after both updates; step 3's update is issued later but runs first
    steps = [st(0, 0, 0, 2, 5, 9), st(0, 1, 6, 8, 10, 12), st(0, 2, 13, 14, 20, 22), st(0, 3, 13, 14, 16, 18)]
    ann, s = D.analyze(steps, [])
    assert [a["staleness"] for a in ann] == [0, 1, 1, 0]
    assert [a["update_order"] for a in ann] == [0, 1, 3, 2]
    assert s["order_inversions"] == 1
    assert s["staleness_hist"] == {0: 2, 1: 2}


def test_good_iterates_against_averaging_rounds():
    rounds = [dict(t=[20, 30]), dict(t=[60, 70])]
    steps = [st(0, 0, 0, 5, 10, 12),      # before any round: good
             st(0, 1, 25, 28, 40, 42),    # snapshot inside round 0: not good
             st(1, 0, 31, 33, 40, 44),    # snapshot after round 0 ended: good
             st(1, 1, 50, 55, 65, 68),    # update while round 1 runs, snapshot before it: not good
             st(0, 2, 71, 72, 80, 81)]    # after round 1: good
    ann, s = D.analyze(steps, rounds)
    assert [a["good"] for a in ann] == [True, False, True, False, True]
    assert s["p_good"] == 3 / 5
    assert [a["major"] for a in ann] == [0, 1, 1, 1, 2]

"""Controller bookkeeping of replication and recovery (CPU)."""
import os

import pytest

from paper_2403_01876_amd import recovery as R


def test_processing_order_is_round_robin():
    M = 3
    seq = [(0, 0)]
    for _ in range(7):
        seq.append(R.successor(seq[-1], M))
    assert seq == [(0, 0), (1, 0), (2, 0), (0, 1), (1, 1), (2, 1), (0, 2), (1, 2)]
    assert [R.order(s, M) for s in seq] == list(range(8))


def test_resume_point_follows_the_failed_workers_replication():
    tab = R.ReplicationTable(workers=4, microbatches=3)
    assert tab.resume_point(1) == (0, 0)  # nothing replicated yet
    # worker 2 holds worker 1's updates up to (1, 4), reported in order
    step = (0, 0)
    while R.order(step, 3) <= R.order((1, 4), 3):
        tab.report(2, *step)
        step = R.successor(step, 3)
    assert tab.replicated_upto(1) == (1, 4)
    assert tab.resume_point(1) == (2, 4)
    tab.report(2, 2, 4)
    assert tab.resume_point(1) == (0, 5)  # wraps to the next step


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "ft_protocol_example.txt")


def read_example(path):
    """The worked example, converted from the paper's 1-based labels (stages,
    microbatches, step letters A, B, C, ...) to 0-based indices."""
    ex = {"transfers": []}
    for line in open(path):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] in ("stages", "microbatches", "failed_stage"):
            ex[f[0]] = int(f[1]) - (1 if f[0] == "failed_stage" else 0)
        elif f[0] in ("first_unreplicated", "resume"):
            ex[f[0]] = (int(f[1]) - 1, ord(f[2]) - ord("A"))
        elif f[0] == "transfer":
            ex["transfers"].append((int(f[1]) - 1, int(f[2]) - 1, f[3], int(f[4]) - 1))
    return ex


def test_paper_example_stage_two_fails():
    """The paper's worked example (fixture in tests/golden): the replication
    status just before the failure, then the two recovery transfers and the
    resume point the controller derives from it."""
    ex = read_example(GOLDEN)
    n, m, failed = ex["stages"], ex["microbatches"], ex["failed_stage"]
    tab = R.ReplicationTable(workers=n, microbatches=m)
    stop = R.order(ex["first_unreplicated"], m)
    for k in range(stop):  # every (j, t) before it was replicated on every stage
        j, t = k % m, k // m
        for x in range(n):
            tab.report(x, j, t)
    plan, resume = tab.recovery_plan(failed)
    assert resume == ex["resume"] == ex["first_unreplicated"]
    expect = [R.Transfer(sender=snd, receiver=rcv, owner=own, into_replica=(what == "replica_of"))
              for snd, rcv, what, own in ex["transfers"]]
    assert plan == expect


def test_recovery_plan_wraps_around_the_ring():
    tab = R.ReplicationTable(workers=3, microbatches=2)
    plan, resume = tab.recovery_plan(0)
    assert plan[0].sender == 1 and plan[1].sender == 2 and plan[1].owner == 2
    plan, resume = tab.recovery_plan(2)
    assert plan[0].sender == 0 and plan[1].sender == 1


def test_reports_keep_the_latest_step():
    tab = R.ReplicationTable(workers=2, microbatches=2)
    tab.report(1, 1, 0)
    tab.report(1, 0, 0)  # a re-executed step does not move the status back
    assert tab.held[1] == (1, 0)
    tab.report(1, 0, 1)
    assert tab.held[1] == (0, 1)
    assert tab.steps_held(1, 0) == 2 and tab.steps_held(1, 1) == 1
    with pytest.raises(ValueError):
        tab.report(2, 0, 1)
    with pytest.raises(ValueError):
        tab.report(0, 2, 0)
    with pytest.raises(ValueError):
        R.ReplicationTable(workers=1, microbatches=1)

"""Controller bookkeeping of replication and recovery (CPU)."""
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


def test_paper_example_stage_two_fails():
    """Four stages; stage 2 (index 1) fails after its update for microbatch 1,
    step C had not reached stage 3: all stages resume from (1, C)."""
    C = 2
    tab = R.ReplicationTable(workers=4, microbatches=4)
    for t in range(C + 1):
        for j in range(4):
            if R.order((j, t), 4) < R.order((1, C), 4):
                for x in range(4):
                    tab.report(x, j, t)
    plan, resume = tab.recovery_plan(1)
    assert resume == (1, C)
    assert plan[0] == R.Transfer(sender=2, receiver=1, owner=1, into_replica=False)
    assert plan[1] == R.Transfer(sender=0, receiver=1, owner=0, into_replica=True)


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

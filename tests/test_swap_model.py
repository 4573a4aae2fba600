"""The swap-benefit model against closed forms (CPU)."""
import math

import pytest

from paper_2403_01876_amd import swap_model as M


def test_transfer_is_linear_in_tokens_and_requests():
    assert M.transfer_time(1000, 8, 589824, 57e9) == pytest.approx(1000 * 8 * 589824 / 57e9)
    assert M.transfer_time(0, 8, 100, 1.0) == 0.0


def test_compute_bound_steps_always_win():
    # every transfer shorter than a step: the swapped phase is N t, and 2 N t >= N t
    N, p, t = 50, 100, 1.0
    assert M.swapped_token_phase(N, p, t, 1, 1.0, 1e9) == pytest.approx(N * t)
    assert M.swapping_wins(N, p, t, 1, 1.0, 1e9)


def test_transfer_bound_sum_is_arithmetic_series():
    # t = 0: the phase is sum_{i=p}^{p+N-1} i * R * C / bw
    N, p, R, C, bw = 7, 10, 3, 5.0, 2.0
    exp = R * C / bw * (N * p + N * (N - 1) / 2)
    assert M.swapped_token_phase(N, p, 0.0, R, C, bw) == pytest.approx(exp)
    assert not M.swapping_wins(N, p, 0.0, R, C, bw)


def test_single_step_breakeven_is_half_the_transfer():
    # N = 1: 2 t >= max(t, T_p)  <=>  t >= T_p / 2
    T = M.transfer_time(300, 4, 10.0, 100.0)
    assert M.breakeven_step_time(1, 300, 4, 10.0, 100.0) == pytest.approx(T / 2, rel=1e-9)


def test_breakeven_solves_the_inequality():
    N, p, R, C, bw = 200, 1000, 8, 589824.0, 57e9
    t = M.breakeven_step_time(N, p, R, C, bw)
    assert M.swapping_wins(N, p, t * (1 + 1e-9), R, C, bw)
    assert not M.swapping_wins(N, p, t * (1 - 1e-6), R, C, bw)
    # when every step is transfer-bound (t below every T_i) the root is the
    # mean transfer time over two: 2 N t = sum T_i
    t_mean = M.swapped_token_phase(N, p, 0.0, R, C, bw) / (2 * N)
    assert t <= M.transfer_time(p, R, C, bw) + 1e-15 or math.isclose(t, t_mean, rel_tol=1e-9)
    if t < M.transfer_time(p, R, C, bw):
        assert t == pytest.approx(t_mean, rel=1e-9)


def test_swap_schedule_matches_the_papers_example():
    """Steady state of swap_schedule against the paper's 4-stage example
    (fixture in tests/golden, 1-based labels)."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                        "swap_schedule_example.txt")
    rows, n = [], None
    for line in open(path):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "microbatches":
            n = int(f[1])
        else:
            rows.append(tuple(int(v) - 1 for v in f))
    sched = list(M.swap_schedule(n, 3))
    steady = sched[n:2 * n]  # the middle round: neither the first nor the last step
    assert steady == rows
    # edges: nothing to swap out before the first step or in after the last
    assert sched[0] == (0, 1, None) and sched[-1] == (n - 1, None, n - 2)
    # every microbatch is swapped in before it is processed (except the first,
    # prefetched before the loop) and swapped out right after
    for k, (x, nxt, prev) in enumerate(sched):
        if k > 0:
            assert sched[k - 1][1] == x and prev == sched[k - 1][0]


def test_swap_schedule_single_microbatch_and_errors():
    assert list(M.swap_schedule(1, 2)) == [(0, 0, None), (0, None, 0)]
    assert list(M.swap_schedule(3, 0)) == []
    with pytest.raises(ValueError):
        list(M.swap_schedule(0, 1))

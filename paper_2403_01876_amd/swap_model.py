"""When microbatch swapping pays off (the paper's App. E model).

Without swapping a stage fits microbatches of size B; with swapping it fits
2B, so one swapped batch of 2B replaces two unswapped batches of B.  With a
constant decode-step time t, prompt time P for B (2P for 2B), N generated
tokens and a prompt of p tokens, swapping wins when

    2 (P + N t)  >=  2 P + sum_i max(t, transf_i),   i.e.
    2 N t        >=  sum_i max(t, transf_i),

where transf_i = i * requests * C / bw is the time to bring the cache of
the swapped microbatch back over the host link at the step where it holds i
tokens per request; C is the single-token, single-request KV size (bytes,
all layers of the stage) and bw the host-link bandwidth (bytes/s).

Readings (the printed sums disagree on their limits and the printed
transfer term writes B): the sum runs over the N decode steps, i = p ..
p+N-1; ``requests`` is the number of requests whose cache is swapped.
"""
from __future__ import annotations


def transfer_time(i: int, requests: int, kv_bytes_per_token: float, bw: float) -> float:
    """Seconds to swap in a microbatch whose requests hold i tokens each."""
    return i * requests * kv_bytes_per_token / bw


def swapped_token_phase(n_tokens: int, prompt: int, t: float, requests: int,
                        kv_bytes_per_token: float, bw: float) -> float:
    """Right-hand side: the token phase of one swapped microbatch, each step
    taking the longer of its compute and its swap-in."""
    return sum(max(t, transfer_time(i, requests, kv_bytes_per_token, bw))
               for i in range(prompt, prompt + n_tokens))


def swapping_wins(n_tokens: int, prompt: int, t: float, requests: int,
                  kv_bytes_per_token: float, bw: float) -> bool:
    return 2 * n_tokens * t >= swapped_token_phase(n_tokens, prompt, t, requests,
                                                   kv_bytes_per_token, bw)


def breakeven_step_time(n_tokens: int, prompt: int, requests: int, kv_bytes_per_token: float,
                        bw: float) -> float:
    """Smallest step time t at which swapping wins.

    f(t) = 2 N t - sum_i max(t, T_i) is continuous, negative at t = 0 and
    increasing (slope 2N minus the number of terms with t > T_i, at least N),
    so the root is unique; it is found by bisection on [0, T_max].
    """
    if n_tokens <= 0:
        return 0.0
    t_max = transfer_time(prompt + n_tokens - 1, requests, kv_bytes_per_token, bw)
    lo, hi = 0.0, t_max
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if swapping_wins(n_tokens, prompt, mid, requests, kv_bytes_per_token, bw):
            hi = mid
        else:
            lo = mid
    return hi


def swap_schedule(microbatches: int, rounds: int):
    """The round-robin order of microbatch swapping (Sec. 4.2.2, Figure
    "swapping"): microbatches are processed 0, 1, ..., M-1, 0, ... and while
    microbatch x is processed, the next one, (x+1) % M, is swapped in and
    the update of the previous one, (x-1) % M, is swapped out.  Yields one
    (process, swap_in, swap_out) triple per step; swap_in is None on the last
    step and swap_out None on the first (nothing precedes or follows them).
    With the scheduler (dv_swapper_*) a caller issues, for each triple, the
    prefetch of swap_in before beginning the step of `process`, and the
    end_step of `process` after it; that end_step is the swap-out the next
    triple lists."""
    if microbatches < 1 or rounds < 0:
        raise ValueError("need at least one microbatch and a non-negative round count")
    steps = microbatches * rounds
    for k in range(steps):
        yield (k % microbatches,
               (k + 1) % microbatches if k + 1 < steps else None,
               (k - 1) % microbatches if k > 0 else None)

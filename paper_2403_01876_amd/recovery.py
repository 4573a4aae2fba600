"""Controller bookkeeping for KV-cache replication and failure recovery
(the paper's failure handling, Sec. 4.2.3, Figure "ft_protocol").

Worker x of an N-stage pipeline streams its KV cache, one token step at a
time, to worker (x+1) % N.  When worker x has received worker (x-1) % N's
update for microbatch j and generation step t it reports (x, j, t), so the
controller knows, for every worker, how far its cache is replicated.  On a
failure of worker f:

  1. worker (f+1) % N sends back the replica of f's cache it holds;
  2. worker (f-1) % N sends its own cache to f (f held its replica);
  3. the controller finds the (microbatch, step) to re-execute: the first
     one whose update of f had not been replicated;
  4. every stage resumes from that (microbatch, step).

Microbatches are processed round-robin, so the order of (j, t) at a stage is
(0, t), (1, t), ..., (M-1, t), (0, t+1), ...  This module holds only that
host-side bookkeeping; the transfers themselves are dv_stream_out_prompt /
dv_stream_in calls (a replica is restored like any received stream).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

Step = Tuple[int, int]  # (microbatch j, generation step t)


def order(step: Step, microbatches: int) -> int:
    """Position of (j, t) in a stage's processing order."""
    j, t = step
    return t * microbatches + j


def successor(step: Step, microbatches: int) -> Step:
    j, t = step
    return (j + 1, t) if j + 1 < microbatches else (0, t + 1)


@dataclasses.dataclass
class Transfer:
    """One recovery transfer: the cache of `owner`, held at `sender`, goes
    to `receiver` (as its own cache, or as the replica it holds)."""
    sender: int
    receiver: int
    owner: int
    into_replica: bool


class ReplicationTable:
    """The controller's replication status of an N-worker ring."""

    def __init__(self, workers: int, microbatches: int):
        if workers < 2 or microbatches < 1:
            raise ValueError("a ring needs at least 2 workers and 1 microbatch")
        self.workers = workers
        self.microbatches = microbatches
        # held[x]: latest (j, t) of worker (x-1)'s cache that worker x holds
        self.held: List[Optional[Step]] = [None] * workers

    def report(self, x: int, j: int, t: int) -> None:
        """Worker x received worker (x-1)'s update for microbatch j, step t.
        The table keeps the latest step per worker: a re-executed step
        reported again after a recovery does not move it back."""
        if not (0 <= x < self.workers and 0 <= j < self.microbatches and t >= 0):
            raise ValueError(f"bad report ({x}, {j}, {t})")
        prev = self.held[x]
        if prev is None or order((j, t), self.microbatches) > order(prev, self.microbatches):
            self.held[x] = (j, t)

    def steps_held(self, x: int, j: int) -> int:
        """Generation steps of microbatch j of worker (x-1)'s cache held at x."""
        done = self.held[x]
        if done is None:
            return 0
        jd, td = done
        return td + 1 if j <= jd else td

    def replicated_upto(self, owner: int) -> Optional[Step]:
        """Latest (j, t) of `owner`'s cache held by its successor."""
        return self.held[(owner + 1) % self.workers]

    def resume_point(self, failed: int) -> Step:
        """Step 3: the first (j, t) whose update of the failed worker was not
        replicated; (0, 0) if none was."""
        done = self.replicated_upto(failed)
        return (0, 0) if done is None else successor(done, self.microbatches)

    def recovery_plan(self, failed: int) -> Tuple[List[Transfer], Step]:
        """Steps 1-3 for a failure of `failed`: the two transfers and the
        resume point (step 4 is re-executing from it on every stage)."""
        n = self.workers
        plan = [Transfer(sender=(failed + 1) % n, receiver=failed, owner=failed,
                         into_replica=False),
                Transfer(sender=(failed - 1) % n, receiver=failed, owner=(failed - 1) % n,
                         into_replica=True)]
        return plan, self.resume_point(failed)

    def after_recovery(self, failed: int, predecessor_done: Optional[Step]) -> None:
        """After step 2 the failed worker holds its predecessor's cache again,
        up to what the predecessor had computed; the failed worker's own
        status is unchanged (its replica at the successor survived)."""
        self.held[failed] = predecessor_done

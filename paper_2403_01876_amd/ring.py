"""Ring KV replication and the four-step recovery on one GPU (the paper's
failure handling, Sec. 4.2.3), built on the C-ABI streaming calls.

N pipeline stages ("workers") each hold their own KV cache for M
microbatches and a replica of their predecessor's.  Generation is emulated:
a worker's step (j, t) writes that step's token for all its layers (the
bytes are a function of (worker, j, t), so re-executing a step rewrites the
same bytes).  After each step the worker streams the increment to its
successor (dv_stream_out_token, then dv_stream_in into the successor's
replica) and the successor reports (x, j, t) to the controller
(recovery.ReplicationTable).  A failure poisons a worker's cache and the
replica it holds; recovery runs the controller's plan with whole-cache
streams (dv_stream_out_prompt / dv_stream_in over each microbatch's valid
tokens) and resumes every stage from the controller's resume point.
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np

from . import dv
from .recovery import ReplicationTable, Step, order, successor


class RingSim:
    def __init__(self, workers: int, microbatches: int, layers: int, heads: int,
                 head_dim: int, batch: int, max_seq: int, prompt_lens, seed: int = 0):
        import torch

        import synth

        self.torch, self.synth = torch, synth
        self.N, self.M, self.L = workers, microbatches, layers
        self.H, self.D, self.B, self.S = heads, head_dim, batch, max_seq
        self.prompt = np.asarray(prompt_lens, np.int32).reshape(microbatches, batch)
        self.seed = seed
        dev = torch.device("cuda:0")
        self.mb_bytes = layers * 2 * batch * heads * max_seq * head_dim * 2
        self.caches = [torch.zeros(microbatches * self.mb_bytes, dtype=torch.uint8, device=dev)
                       for _ in range(workers)]
        self.replicas = [torch.zeros(microbatches * self.mb_bytes, dtype=torch.uint8,
                                     device=dev) for _ in range(workers)]
        self.c = [self._desc(t) for t in self.caches]
        self.r = [self._desc(t) for t in self.replicas]
        full = dv.dv_packed_bytes(self.c[0], 0, layers, None, np.full(batch, max_seq, np.int32))
        self.wire = torch.empty(full, dtype=torch.uint8, device=dev)
        self.tok = torch.empty(dv.dv_packed_bytes(self.c[0], 0, layers, None,
                                                  np.ones(batch, np.int32)),
                               dtype=torch.uint8, device=dev)
        self.table = ReplicationTable(workers, microbatches)
        self.done: List[Optional[Step]] = [None] * workers  # latest step computed
        self.stream = torch.cuda.current_stream()

    def _desc(self, t):
        return dv.Cache(dv.DV_DENSE, self.L, self.H, self.D, self.B,
                        [t.data_ptr() + j * self.mb_bytes for j in range(self.M)],
                        max_seq=self.S)

    PROMPT, TOKEN = 1, 2

    def seed_for(self, kind: int, x: int, j: int, t: int = 0) -> int:
        """Seed of the bytes a worker's prompt pass or step (j, t) writes."""
        return self.synth.derived_seed(self.seed, (kind << 56) ^ (x << 40) ^ (j << 24) ^ t)

    def _fill(self, buf, nbytes, kind, x, j, t=0):
        self.synth.device_fill(buf.data_ptr(), nbytes, self.seed_for(kind, x, j, t),
                               stream=self.stream.cuda_stream)

    # -- generation ---------------------------------------------------------
    def prefill(self) -> None:
        """Prompt pass on every stage, its cache streamed whole to the
        successor's replica (layer ranges could equally go one by one)."""
        zero = np.zeros(self.B, np.int32)
        for x in range(self.N):
            for j in range(self.M):
                lens = self.prompt[j]
                n = dv.dv_packed_bytes(self.c[x], 0, self.L, zero, lens)
                self._fill(self.wire, n, self.PROMPT, x, j)
                dv.dv_stream_in(self.c[x], j, 0, self.L, zero, lens, self.wire, n, self.stream)
                self._send(x, j, zero, lens)

    def _send(self, x, j, t0, t1) -> None:
        n = dv.dv_stream_out_prompt(self.c[x], j, 0, self.L, t0, t1, self.wire,
                                    self.wire.numel(), self.stream)
        dv.dv_stream_in(self.r[(x + 1) % self.N], j, 0, self.L, t0, t1, self.wire, n,
                        self.stream)

    def compute(self, x: int, j: int, t: int) -> None:
        pos = self.prompt[j] + t
        self._fill(self.tok, self.tok.numel(), self.TOKEN, x, j, t)
        dv.dv_stream_in(self.c[x], j, 0, self.L, pos, pos + 1, self.tok, self.tok.numel(),
                        self.stream)
        self.done[x] = (j, t) if self.done[x] is None or \
            order((j, t), self.M) > order(self.done[x], self.M) else self.done[x]

    def replicate(self, x: int, j: int, t: int) -> None:
        pos = self.prompt[j] + t
        n = dv.dv_stream_out_token(self.c[x], j, 0, self.L, pos, self.tok, self.tok.numel(),
                                   self.stream)
        dv.dv_stream_in(self.r[(x + 1) % self.N], j, 0, self.L, pos, pos + 1, self.tok, n,
                        self.stream)
        self.table.report((x + 1) % self.N, j, t)

    def run(self, start: Step, end: Step, fail_at: Optional[Tuple[int, int, int]] = None):
        """Steps in processing order from `start` up to but not including
        `end`, each on every stage in pipeline order.  With fail_at =
        (worker, j, t) the run stops after that worker computed (j, t) and
        before it streamed the update; returns True if it stopped there."""
        step = start
        while order(step, self.M) < order(end, self.M):
            j, t = step
            for x in range(self.N):
                self.compute(x, j, t)
                if fail_at == (x, j, t):
                    return True
                self.replicate(x, j, t)
            step = successor(step, self.M)
        return False

    # -- failure and recovery ------------------------------------------------
    def fail(self, f: int) -> None:
        self.caches[f].fill_(0xA5)
        self.replicas[f].fill_(0xA5)

    def _steps(self, done: Optional[Step], j: int) -> int:
        if done is None:
            return 0
        jd, td = done
        return td + 1 if j <= jd else td

    def recover(self, f: int) -> Step:
        """Steps 1-3 of the recovery; returns the resume point."""
        plan, resume = self.table.recovery_plan(f)
        zero = np.zeros(self.B, np.int32)
        for tr in plan:
            for j in range(self.M):
                if tr.into_replica:   # step 2: the predecessor's own cache
                    src, dst = self.c[tr.sender], self.r[tr.receiver]
                    steps = self._steps(self.done[tr.owner], j)
                else:                 # step 1: the replica held by the successor
                    src, dst = self.r[tr.sender], self.c[tr.receiver]
                    steps = self.table.steps_held(tr.sender, j)
                t1 = (self.prompt[j] + steps).astype(np.int32)
                n = dv.dv_stream_out_prompt(src, j, 0, self.L, zero, t1, self.wire,
                                            self.wire.numel(), self.stream)
                dv.dv_stream_in(dst, j, 0, self.L, zero, t1, self.wire, n, self.stream)
        self.table.after_recovery(f, self.done[(f - 1) % self.N])
        self.done[f] = None if resume == (0, 0) else self._prev(resume)
        return resume

    def _prev(self, step: Step) -> Step:
        j, t = step
        return (j - 1, t) if j > 0 else (self.M - 1, t - 1)

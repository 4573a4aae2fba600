#!/usr/bin/env python3
"""KV-cache streaming benchmark on one MI355X.

A step is one pass of the streaming hot path over the largest workload, the
LLaMA-2-70B-shaped paged pool (20 of 80 layers, 8 KV heads x 128, block 16,
32 sequences of U[128, 4096] tokens from the seed, fp16):

  paged gather of the prompt caches through table A (pack) -> scatter of the
  contiguous buffer into a second pool through the freshly permuted table B
  (unpack, in pool order through an owner-map workspace) -> 128 decode steps,
  each tail-block increment packed out of pool A and streamed into pool B.

Inputs are resident in HBM before timing starts.  The step's 258 calls are
captured once into a HIP graph and the graph is replayed (the increments are
launch-bound, 2.6 MB each); the same step issued call by call is timed too
and reported as ``eager_ms_per_step`` (``--eager`` makes it the headline).
``value`` is algorithmic bytes per step (every payload byte read once and
written once: 2 x payload per call) over the step time, in GB/s.
``roofline`` is the paged gather kernel, its duration from HIP events around
back-to-back launches on its stream, with two ceilings beside it: a plain
contiguous copy of the same bytes, and a copy of the whole pool block by
block in the table's order (the gather's random block placement).
``rooflines`` lists every bulk operation measured, per workload.  Further
objects report the OPT-13B stage step (prompt and increments, with the dense
pack kernel's roofline), the other kernels, the microbatch swap over the
host link and the swap scheduler's protocol (OPT-66B stage), the full-cache
replica and restore (BLOOM-176B shard), multi-token steps, streaming
overlapped with emulated compute, ring recovery, buffered against
per-region copies, and the oracle timed on the host cores (multi- and
single-threaded, and compared over every byte with the GPU's gather and
scatter).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--eager]
                       [--extras all|bulk|calib|swap|none] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# HIP multiplexes streams onto GPU_MAX_HW_QUEUES hardware queues (4 by
# default) and two streams sharing one execute in order.  This process
# creates many streams (torch's pool, graph capture, the swap scheduler's
# two), and with 4 queues the scheduler's input stream can land on the
# compute stream's queue, which serialises every swap-in with the step it
# should hide behind.  8 queues keep them apart.  Set before HIP starts.
if int(os.environ.get("GPU_MAX_HW_QUEUES", "4") or 4) < 8:
    os.environ["GPU_MAX_HW_QUEUES"] = "8"

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
PCIE_PEAK_GBS = 63.0        # PCIe Gen5 x16 per direction after 128b/130b encoding
METRIC = "KV pack/scatter GB/s and % of HBM peak; swap GB/s vs host-link peak (1 GPU)"


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--no-extras", action="store_true")
    p.add_argument("--extras", choices=("all", "bulk", "calib", "swap", "none"), default="all",
                   help="calib: only the known-size copy used to scale counter runs; "
                        "bulk: the bulk workloads and that copy; swap: the OPT-66B swaps and "
                        "the swap protocol only")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--eager", action="store_true",
                   help="report the step issued call by call instead of graph-replayed")
    return p.parse_args()


class Timer:
    """HIP-event pairs on one stream; mean duration in ms."""

    def __init__(self, torch, stream):
        self.torch, self.stream, self.pairs = torch, stream, []

    def __enter__(self):
        a = self.torch.cuda.Event(enable_timing=True)
        a.record(self.stream)
        self.pairs.append([a, None])
        return self

    def __exit__(self, *exc):
        b = self.torch.cuda.Event(enable_timing=True)
        b.record(self.stream)
        self.pairs[-1][1] = b

    def mean_ms(self) -> float:
        ts = [a.elapsed_time(b) for a, b in self.pairs]
        return sum(ts) / len(ts)

    def min_ms(self) -> float:
        return min(a.elapsed_time(b) for a, b in self.pairs)

    def median_ms(self) -> float:
        ts = sorted(a.elapsed_time(b) for a, b in self.pairs)
        n = len(ts)
        return ts[n // 2] if n % 2 else 0.5 * (ts[n // 2 - 1] + ts[n // 2])


def flush_l2(torch, scratch):
    """Overwrite 512 MB so no payload is served from L2 / MALL."""
    scratch.add_(1)


def ranges_match(torch, recv, src, L, B, H, S, D, t0, t1, fill=0):
    """Receiver equals source on the token ranges of every (layer, K|V,
    sequence, head) of two dense fp16 caches, and holds `fill` bytes
    everywhere else (the streaming invariants, checked on the device)."""
    r = recv[: L * 2 * B * H * S * D * 2].view(torch.int16).view(L, 2, B, H, S, D)
    x = src[: L * 2 * B * H * S * D * 2].view(torch.int16).view(L, 2, B, H, S, D)
    outside = torch.ones((L, 2, B, H, S), dtype=torch.bool, device=recv.device)
    for b in range(B):
        a, e = int(t0[b]), int(t1[b])
        if not torch.equal(r[:, :, b, :, a:e], x[:, :, b, :, a:e]):
            return False
        outside[:, :, b, :, a:e] = False
    fv = torch.tensor([fill], dtype=torch.uint8, device=recv.device).repeat(2).view(torch.int16)
    return bool((r[outside] == fv).all())


def main_step_bench(args, torch, dv, synth):
    """The step on the OPT-13B stage: replayed as one captured HIP graph (the
    default; the 258 launches of a step are launch-bound otherwise) or issued
    eagerly call by call (--eager).  Both are timed; ``value`` uses the mode
    asked for."""
    dev = torch.device("cuda:0")
    w = synth.make_workload(1)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    nbytes = w.dense_bytes()
    stream = torch.cuda.current_stream()
    sender = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    synth.device_fill(sender.data_ptr(), nbytes, w.data_seed, stream=stream.cuda_stream)
    recv = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [sender], max_seq=S)
    cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S)
    t0, t1 = w.prompt_ranges()
    P = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = torch.empty(P, dtype=torch.uint8, device=dev)
    pos = [w.step_positions(i) for i in range(w.steps)]
    ends = [p + 1 for p in pos]
    I = dv.dv_packed_bytes(cs, 0, L, pos[0], ends[0])
    incs = torch.empty(I, dtype=torch.uint8, device=dev)

    def pack(st):
        dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, P, st)

    def unpack(st):
        dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, P, st)

    def step(st):
        pack(st)
        unpack(st)
        for i in range(w.steps):
            dv.dv_stream_out_token(cs, 0, 0, L, pos[i], incs, I, st)
            dv.dv_stream_in(cr, 0, 0, L, pos[i], ends[i], incs, I, st)

    def timed(fn, n):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    # eager
    for _ in range(args.warmup):
        step(stream)
    eager_ms = timed(lambda: step(stream), args.steps)
    log(f"eager: {eager_ms:.3f} ms/step")
    # The step's own invariants (no oracle): the receiver, zero before,
    # equals the sender on [0, len + steps) and is zero elsewhere.
    full = t1 + w.steps
    checks = {"eager_receiver_equals_sender_on_ranges":
              ranges_match(torch, recv, sender, L, B, H, S, D, t0, full)}
    eager_wire = wire.clone()
    # graph
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        graph.replay()
    graph_ms = timed(graph.replay, args.steps)
    log(f"graph: {graph_ms:.3f} ms/step")
    recv.zero_()
    wire.zero_()
    graph.replay()
    torch.cuda.synchronize()
    checks["graph_receiver_equals_sender_on_ranges"] = ranges_match(
        torch, recv, sender, L, B, H, S, D, t0, full)
    checks["graph_wire_equals_eager_wire"] = bool(torch.equal(wire, eager_wire))
    del eager_wire
    ms = eager_ms if args.eager else graph_ms

    # Per-kernel durations: one event pair around back-to-back launches that
    # follow a leading untimed one, so the queue never drains and the mean is
    # pure kernel time (an event pair per launch would add its own packets).
    # Single launches vary by about 1 %, so at least 20 are averaged.
    kern = {}
    nk = max(args.steps, 20)
    for name, fn in (("pack", pack), ("unpack", unpack)):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        fn(stream)
        a.record(stream)
        for _ in range(nk):
            fn(stream)
        b.record(stream)
        torch.cuda.synchronize()
        kern[name] = a.elapsed_time(b) / nk
    # The copy ceiling: a plain contiguous copy of the same P bytes, timed the
    # same way, in the pack kernel's launch shape (the layout is the only
    # difference left).
    from paper_2403_01876_amd import baseline

    def plain(s):
        baseline.plain_copy(wire, sender, P, s)

    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    plain(stream)
    a.record(stream)
    for _ in range(nk):
        plain(stream)
    b.record(stream)
    torch.cuda.synchronize()
    kern["plain_copy"] = a.elapsed_time(b) / nk
    checks["plain_copy_equals_source"] = bool(torch.equal(wire[:P], sender[:P]))
    step_bytes = 2 * P * 2 + w.steps * 2 * I * 2
    res = {
        "ms": ms, "eager_ms": eager_ms, "graph_ms": graph_ms, "P": P, "I": I,
        "step_bytes": step_bytes, "value": step_bytes / (ms * 1e-3) / 1e9,
        "pack_ms": kern["pack"], "unpack_ms": kern["unpack"], "copy_ms": kern["plain_copy"],
        "checks": checks,
    }
    del sender, recv, wire, incs, graph
    torch.cuda.empty_cache()
    return w, res


def block_order(w, table):
    """For the paged pool of workload ``w``: the pool blocks of every (layer,
    K|V) slab in the order the block table visits them (sequence by sequence,
    logical block by logical block), as global block indices.  The workload's
    tables use every pool block once, so this is a permutation of all the
    pool's blocks."""
    nb = w.num_blocks
    per_slab = np.asarray(table, np.int64).reshape(-1)
    per_slab = per_slab[(per_slab >= 0) & (per_slab < nb)]
    assert per_slab.size == nb and np.unique(per_slab).size == nb
    slabs = np.arange(2 * w.layers, dtype=np.int64)[:, None] * nb
    return (slabs + per_slab[None, :]).reshape(-1).astype(np.int32)


def back_to_back_ms(torch, stream, fn, n):
    """Mean duration of ``fn`` from one event pair around ``n`` back-to-back
    calls that follow a leading untimed one, so the queue never drains and
    the mean is pure kernel time (an event pair per launch would add its own
    packets)."""
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    fn()
    a.record(stream)
    for _ in range(n):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


def paged_step_bench(args, torch, dv, synth):
    """The step on the LLaMA-2-70B paged pool (20 of 80 layers, 8 KV heads x
    128, block 16, 32 sequences of U[128, 4096] tokens): paged gather of the
    prompt caches through table A into one contiguous buffer, scatter of that
    buffer into a second pool through the freshly permuted table B (pool
    order, through an owner-map workspace), then 128 decode steps whose
    tail-block increments are packed out of pool A and streamed into pool B.
    Replayed as one captured HIP graph (the default) or issued call by call
    (--eager); both are timed.  Then the bulk kernels alone, back to back,
    with the sequential copy ceiling and the block-order ceiling beside
    them."""
    from paper_2403_01876_amd import baseline
    dev = torch.device("cuda:0")
    w = synth.make_workload(4)
    L, H, D, B = w.layers, w.heads, w.head_dim, w.batch
    nb, bs, mbk = w.num_blocks, w.block_size, w.max_blocks
    stream = torch.cuda.current_stream()
    pool_bytes = w.pool_bytes()
    pool_a = torch.empty(pool_bytes, dtype=torch.uint8, device=dev)
    synth.device_fill(pool_a.data_ptr(), pool_bytes, w.data_seed, stream=stream.cuda_stream)
    pool_b = torch.zeros(pool_bytes, dtype=torch.uint8, device=dev)
    bta = torch.from_numpy(w.block_table_a).to(dev)
    btb = torch.from_numpy(w.block_table_b).to(dev)
    owners = torch.empty(nb * 4, dtype=torch.uint8, device=dev)
    kw = dict(block_size=bs, num_blocks=nb, max_blocks=mbk)
    ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_a], block_tables=[bta], **kw)
    cb = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_b], block_tables=[btb], block_owners=[owners],
                  **kw)
    cb_table = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_b], block_tables=[btb], **kw)
    t0, t1 = w.prompt_ranges()
    P = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = torch.empty(P, dtype=torch.uint8, device=dev)
    pos = [w.step_positions(i) for i in range(w.steps)]
    ends = [p + 1 for p in pos]
    I = dv.dv_packed_bytes(ca, 0, L, pos[0], ends[0])
    inc = torch.empty(I, dtype=torch.uint8, device=dev)

    def gather(st):
        dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, P, st)

    def scatter(st):
        dv.dv_stream_in(cb, 0, 0, L, t0, t1, wire, P, st)

    def step(st):
        gather(st)
        scatter(st)
        for i in range(w.steps):
            dv.dv_stream_out_token(ca, 0, 0, L, pos[i], inc, I, st)
            dv.dv_stream_in(cb, 0, 0, L, pos[i], ends[i], inc, I, st)

    def timed(fn, n):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    full = (t1 + w.steps).astype(np.int32)
    M = dv.dv_packed_bytes(ca, 0, L, t0, full)

    def pools_agree():
        """The step's invariant, on the device: pool B gathers through table
        B to the same bytes as pool A through table A over [0, len + 128)."""
        ga = torch.empty(M, dtype=torch.uint8, device=dev)
        gb = torch.empty(M, dtype=torch.uint8, device=dev)
        dv.dv_stream_out_prompt(ca, 0, 0, L, t0, full, ga, M, stream)
        dv.dv_stream_out_prompt(cb, 0, 0, L, t0, full, gb, M, stream)
        torch.cuda.synchronize()
        ok = bool(torch.equal(ga, gb))
        del ga, gb
        return ok

    for _ in range(args.warmup):
        step(stream)
    eager_ms = timed(lambda: step(stream), args.steps)
    log(f"paged step, eager: {eager_ms:.3f} ms/step")
    checks = {"eager_pool_b_gathers_to_pool_a": pools_agree()}
    eager_wire = wire.clone()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        graph.replay()
    graph_ms = timed(graph.replay, args.steps)
    log(f"paged step, graph: {graph_ms:.3f} ms/step")
    pool_b.zero_()
    wire.zero_()
    graph.replay()
    torch.cuda.synchronize()
    checks["graph_pool_b_gathers_to_pool_a"] = pools_agree()
    checks["graph_wire_equals_eager_wire"] = bool(torch.equal(wire, eager_wire))
    del eager_wire, graph
    ms = eager_ms if args.eager else graph_ms

    # the bulk kernels alone; at least 20 launches averaged (single launches
    # vary by about 1 %)
    nk = max(args.steps, 20)
    kern = {
        "gather": back_to_back_ms(torch, stream, lambda: gather(stream), nk),
        "scatter_pool_order": back_to_back_ms(torch, stream, lambda: scatter(stream), nk),
        "scatter_table_order": back_to_back_ms(
            torch, stream, lambda: dv.dv_stream_in(cb_table, 0, 0, L, t0, t1, wire, P, stream),
            nk),
    }
    # ceilings, on the gather's own buffers (placement in HBM moves these
    # figures by several percent from one allocation to another): the first P
    # bytes of pool A copied contiguously into the buffer (the pack kernels'
    # copy ceiling), and the whole pool A copied into pool B block by block in
    # table A's order, random block reads (the gather's placement) and random
    # block writes (the table-order scatter's)
    kern["plain_copy"] = back_to_back_ms(
        torch, stream, lambda: baseline.plain_copy(wire, pool_a, P, stream), nk)
    checks["plain_copy_equals_source"] = bool(torch.equal(wire, pool_a[:P]))
    order = torch.from_numpy(block_order(w, w.block_table_a)).to(dev)
    nblk = int(order.numel())
    blk_bytes = H * bs * D * w.elem_bytes
    assert nblk * blk_bytes == pool_bytes
    for name, sc, src, dst in (("block_copy_random_reads", False, pool_a, pool_b),
                               ("block_copy_random_writes", True, pool_a, pool_b)):
        kern[name] = back_to_back_ms(
            torch, stream,
            lambda: baseline.block_copy(dst, src, order, nblk, blk_bytes, sc, stream), nk)
    step_bytes = 2 * P * 2 + w.steps * 2 * I * 2
    res = {"ms": ms, "eager_ms": eager_ms, "graph_ms": graph_ms, "P": P, "I": I,
           "pool_bytes": pool_bytes, "num_blocks": nb, "step_bytes": step_bytes,
           "value": step_bytes / (ms * 1e-3) / 1e9, "kern": kern, "checks": checks}
    del pool_a, pool_b, wire, inc, order
    torch.cuda.empty_cache()
    return w, res


def increments_bench(torch, dv, synth):
    """Per-call latency of decode-step increments (eager and graph-replayed)."""
    dev = torch.device("cuda:0")
    out = {}
    for idx in (1, 2, 4):
        w = synth.make_workload(idx)
        L, H, D, B = w.layers, w.heads, w.head_dim, w.batch
        stream = torch.cuda.current_stream()
        if w.paged:
            nbytes = w.pool_bytes()
            buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            bt = torch.from_numpy(w.block_table_a).to(dev)
            c = dv.Cache(dv.DV_PAGED, L, H, D, B, [buf], block_size=w.block_size,
                         num_blocks=w.num_blocks, max_blocks=w.max_blocks, block_tables=[bt])
        else:
            nbytes = w.dense_bytes()
            buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            c = dv.Cache(dv.DV_DENSE, L, H, D, B, [buf], max_seq=S_of(w))
        synth.device_fill(buf.data_ptr(), nbytes, w.data_seed, stream=stream.cuda_stream)
        p = w.step_positions(0)
        I = dv.dv_packed_bytes(c, 0, L, p, p + 1)
        inc = torch.empty(I, dtype=torch.uint8, device=dev)
        n = 200
        for _ in range(10):
            dv.dv_stream_out_token(c, 0, 0, L, p, inc, I, stream)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            dv.dv_stream_out_token(c, 0, 0, L, p, inc, I, stream)
        b.record(stream)
        torch.cuda.synchronize()
        eager_us = a.elapsed_time(b) / n * 1e3
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(stream)
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                for _ in range(n):
                    dv.dv_stream_out_token(c, 0, 0, L, p, inc, I, torch.cuda.current_stream())
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        a.record(stream)
        g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        graph_us = a.elapsed_time(b) / n * 1e3
        out[w.name] = {
            "bytes": I, "cache_state": "warm (back-to-back calls)",
            "eager_us_per_call": round(eager_us, 3),
            "graph_us_per_call": round(graph_us, 3),
            "eager_GBps_2x": round(2 * I / (eager_us * 1e-6) / 1e9, 1),
            "graph_GBps_2x": round(2 * I / (graph_us * 1e-6) / 1e9, 1),
            "hbm_roofline_us": round(2 * I / (HBM_PEAK_GBS * 1e9) * 1e6, 3),
        }
        del buf, inc, g
        torch.cuda.empty_cache()
    return out


def multi_token_bench(torch, dv, synth, ks=(1, 2, 4, 8, 16, 32)):
    """Decode steps that add K tokens per sequence (speculative decoding that
    accepts several tokens, or replication batched over K steps): stream-out
    then stream-in of [len, len + K) for every sequence, captured 50 times
    into a graph and replayed, on the OPT-13B stage and the LLaMA-2-70B paged
    pool.  K = 1 takes the single-token kernel, 2 <= K <= 16 the short-run
    kernel, K = 32 the tiled kernels."""
    dev = torch.device("cuda:0")
    out = {}
    for idx in (1, 4):
        w = synth.make_workload(idx)
        L, H, D, B = w.layers, w.heads, w.head_dim, w.batch
        st = torch.cuda.current_stream()
        if w.paged:
            nbytes = w.pool_bytes()
            src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            dst = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
            bta = torch.from_numpy(w.block_table_a).to(dev)
            btb = torch.from_numpy(w.block_table_b).to(dev)
            cs = dv.Cache(dv.DV_PAGED, L, H, D, B, [src], block_size=w.block_size,
                          num_blocks=w.num_blocks, max_blocks=w.max_blocks, block_tables=[bta])
            cr = dv.Cache(dv.DV_PAGED, L, H, D, B, [dst], block_size=w.block_size,
                          num_blocks=w.num_blocks, max_blocks=w.max_blocks, block_tables=[btb])
        else:
            nbytes = w.dense_bytes()
            src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            dst = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
            cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [src], max_seq=w.max_seq)
            cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [dst], max_seq=w.max_seq)
        synth.device_fill(src.data_ptr(), nbytes, w.data_seed, stream=st.cuda_stream)
        p = w.step_positions(0).astype(np.int32)
        rows = {}
        for K in ks:
            t1 = (p + K).astype(np.int32)
            P = dv.dv_packed_bytes(cs, 0, L, p, t1)
            wire = torch.empty(P, dtype=torch.uint8, device=dev)
            n = 50
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(st)
            with torch.cuda.stream(side):
                with torch.cuda.graph(g, stream=side):
                    for _ in range(n):
                        cur = torch.cuda.current_stream()
                        dv.dv_stream_out_prompt(cs, 0, 0, L, p, t1, wire, P, cur)
                        dv.dv_stream_in(cr, 0, 0, L, p, t1, wire, P, cur)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(st)
            g.replay()
            b.record(st)
            torch.cuda.synchronize()
            us = a.elapsed_time(b) / n * 1e3
            rows[str(K)] = {"payload_bytes": P, "out_plus_in_us": round(us, 2),
                            "us_per_token_step": round(us / K, 3),
                            "GBps_2x": round(4 * P / (us * 1e-6) / 1e9, 1)}
            del g, wire
        out[w.name] = rows
        del src, dst
        torch.cuda.empty_cache()
    return out


def S_of(w):
    return w.max_seq


def bulk_bench(torch, dv, synth, idx, reps=20, ksplit=False):
    """Bulk stream-out and stream-in of one workload, timed per call (with
    ``ksplit``, the dense workload stored with the split-key layout)."""
    dev = torch.device("cuda:0")
    w = synth.make_workload(idx)
    L, H, D, B = w.layers, w.heads, w.head_dim, w.batch
    stream = torch.cuda.current_stream()
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    if w.paged:
        nbytes = w.pool_bytes()
        a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        r = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
        bta = torch.from_numpy(w.block_table_a).to(dev)
        btb = torch.from_numpy(w.block_table_b).to(dev)
        ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [a], block_size=w.block_size,
                      num_blocks=w.num_blocks, max_blocks=w.max_blocks, block_tables=[bta])
        # the receiver scatters in pool order through an owner-map workspace;
        # the same scatter in table order is timed beside it
        owners = torch.empty(w.num_blocks * 4, dtype=torch.uint8, device=dev)
        cr = dv.Cache(dv.DV_PAGED, L, H, D, B, [r], block_size=w.block_size,
                      num_blocks=w.num_blocks, max_blocks=w.max_blocks, block_tables=[btb],
                      block_owners=[owners])
        cr_table = dv.Cache(dv.DV_PAGED, L, H, D, B, [r], block_size=w.block_size,
                            num_blocks=w.num_blocks, max_blocks=w.max_blocks,
                            block_tables=[btb])
    else:
        nbytes = w.dense_bytes()
        a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        r = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
        kind = dv.DV_DENSE_KSPLIT if ksplit else dv.DV_DENSE
        ca = dv.Cache(kind, L, H, D, B, [a], max_seq=w.max_seq)
        cr = dv.Cache(kind, L, H, D, B, [r], max_seq=w.max_seq)
    synth.device_fill(a.data_ptr(), nbytes, w.data_seed, stream=stream.cuda_stream)
    t0, t1 = w.prompt_ranges()
    P = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = torch.empty(P, dtype=torch.uint8, device=dev)
    tp, tu, tt = Timer(torch, stream), Timer(torch, stream), Timer(torch, stream)
    for i in range(reps + 2):
        flush_l2(torch, scratch)
        if i >= 2:
            with tp:
                dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, P, stream)
        else:
            dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, P, stream)
        flush_l2(torch, scratch)
        if i >= 2:
            with tu:
                dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, P, stream)
        else:
            dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, P, stream)
        if w.paged:
            flush_l2(torch, scratch)
            if i >= 2:
                with tt:
                    dv.dv_stream_in(cr_table, 0, 0, L, t0, t1, wire, P, stream)
            else:
                dv.dv_stream_in(cr_table, 0, 0, L, t0, t1, wire, P, stream)
    torch.cuda.synchronize()
    res = {"payload_bytes": P}
    # invariants after timing: the receiver holds the sender's ranges (dense:
    # directly; paged and split key: re-packed, since a stream of any layout
    # is in one canonical order)
    if w.paged or ksplit:
        again = torch.empty_like(wire)
        dv.dv_stream_out_prompt(cr, 0, 0, L, t0, t1, again, P, stream)
        torch.cuda.synchronize()
        res["check_receiver_repacks_to_wire"] = bool(torch.equal(again, wire))
        del again
    else:
        res["check_receiver_equals_sender_on_ranges"] = ranges_match(
            torch, r, a, L, B, H, w.max_seq, D, t0, t1)
    timers = [("stream_out", tp), ("stream_in", tu)]
    if w.paged:
        timers.append(("stream_in_table_order", tt))
    for name, t in timers:
        ms = t.mean_ms()
        gbs = 2 * P / (ms * 1e-3) / 1e9
        res[name] = {"ms": round(ms, 4), "median_ms": round(t.median_ms(), 4),
                     "min_ms": round(t.min_ms(), 4),
                     "GBps_2x": round(gbs, 1), "payload_GBps": round(gbs / 2, 1),
                     "frac_hbm": round(gbs / HBM_PEAK_GBS, 4)}
    res["cache_state"] = "cold: 512 MB written between calls"
    del a, r, wire, scratch
    torch.cuda.empty_cache()
    return w, res


def tiny_bench(torch, dv, synth, reps=20):
    """The tiny correctness workload (2 layers, 4 heads x 64, batch 2, prompts of
    100): prompt stream-out / stream-in and 16 increments, cold (512 MB
    written before each call) and warm (back to back).  Latency-bound: a
    fraction of HBM peak means nothing at 409 600 bytes."""
    dev = torch.device("cuda:0")
    w = synth.make_workload(0)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    stream = torch.cuda.current_stream()
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    a = torch.empty(w.dense_bytes(), dtype=torch.uint8, device=dev)
    r = torch.zeros_like(a)
    synth.device_fill(a.data_ptr(), a.numel(), w.data_seed, stream=stream.cuda_stream)
    ca = dv.Cache(dv.DV_DENSE, L, H, D, B, [a], max_seq=S)
    cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [r], max_seq=S)
    t0, t1 = w.prompt_ranges()
    P = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = torch.empty(P, dtype=torch.uint8, device=dev)
    p = w.step_positions(0)
    I = dv.dv_packed_bytes(ca, 0, L, p, p + 1)
    inc = torch.empty(I, dtype=torch.uint8, device=dev)
    ops = {
        "prompt_out": lambda: dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, P, stream),
        "prompt_in": lambda: dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, P, stream),
        "increment_out": lambda: dv.dv_stream_out_token(ca, 0, 0, L, p, inc, I, stream),
        "increment_in": lambda: dv.dv_stream_in(cr, 0, 0, L, p, p + 1, inc, I, stream),
    }
    res = {"payload_prompt_bytes": P, "payload_increment_bytes": I,
           "note": "latency-bound; % of HBM peak not meaningful"}
    for name, op in ops.items():
        op()
        cold, warm = Timer(torch, stream), Timer(torch, stream)
        for _ in range(reps):
            flush_l2(torch, scratch)
            with cold:
                op()
        for _ in range(reps):
            with warm:
                op()
        torch.cuda.synchronize()
        res[name] = {"cold_us": round(cold.mean_ms() * 1e3, 2),
                     "warm_us": round(warm.mean_ms() * 1e3, 2)}
    del scratch, a, r, wire, inc
    torch.cuda.empty_cache()
    return res


def bulk_all(torch, dv, synth):
    """Bulk stream-out / stream-in of the OPT-66B microbatch, the BLOOM shard,
    the LLaMA paged pool and the split-key OPT-13B stage."""
    log("extras: bulk workloads")
    out = {}
    for idx in (2, 3, 4):
        wk, res = bulk_bench(torch, dv, synth, idx)
        out[wk.name] = res
    wk, res = bulk_bench(torch, dv, synth, 1, ksplit=True)
    out[wk.name + " split-key"] = res
    return out


def swap_bench(torch, dv, synth, reps=3):
    """OPT-66B stage microbatch swap over the host link (one slot, valid prefix)."""
    dev = torch.device("cuda:0")
    w = synth.make_workload(2)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    S_host = 1024
    nb_dev = w.dense_bytes()
    nb_host = w.dense_bytes(S_host)
    slots = [torch.empty(nb_dev, dtype=torch.uint8, device=dev) for _ in range(2)]
    for i, s in enumerate(slots):
        synth.device_fill(s.data_ptr(), nb_dev, w.data_seed + i)
    hosts = [torch.empty(nb_host, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    for h in hosts:
        h.fill_(0)
    ds = dv.Cache(dv.DV_DENSE, L, H, D, B, slots, max_seq=S)
    hh = dv.Cache(dv.DV_DENSE, L, H, D, B, [h.data_ptr() for h in hosts], max_seq=S_host,
                  mem=dv.DV_MEM_HOST_PINNED)
    zero = np.zeros(B, np.int32)
    lens = w.lens.astype(np.int32)
    P = dv.dv_packed_bytes(ds, 0, L, zero, lens)
    s_out, s_in = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    res = {"payload_bytes": P, "rows": 2 * L * B * H, "row_bytes": int(lens[0]) * D * 2,
           "device_pitch": S * D * 2, "host_pitch": S_host * D * 2}
    # swap-out alone, swap-in alone, then both directions at once.  The first
    # copy of each direction touches the freshly pinned pages and is timed
    # apart (reported as the first call); the steady-state mean follows.
    first_o, first_i = Timer(torch, s_out), Timer(torch, s_in)
    with first_o:
        dv.dv_swap_out(ds, 0, hh, 0, 0, L, zero, lens, s_out)
    s_out.synchronize()
    with first_i:
        dv.dv_swap_in(hh, 1, ds, 1, 0, L, zero, lens, s_in)
    s_in.synchronize()
    res["first_call_ms"] = {"swap_out": round(first_o.mean_ms(), 3),
                            "swap_in": round(first_i.mean_ms(), 3)}
    to, ti = Timer(torch, s_out), Timer(torch, s_in)
    for _ in range(reps):
        with to:
            dv.dv_swap_out(ds, 0, hh, 0, 0, L, zero, lens, s_out)
        s_out.synchronize()
    for _ in range(reps):
        with ti:
            dv.dv_swap_in(hh, 1, ds, 1, 0, L, zero, lens, s_in)
        s_in.synchronize()
    out_ms, in_ms = to.mean_ms(), ti.mean_ms()
    res["swap_out"] = {"ms": round(out_ms, 3), "GBps": round(P / (out_ms * 1e-3) / 1e9, 2)}
    res["swap_in"] = {"ms": round(in_ms, 3), "GBps": round(P / (in_ms * 1e-3) / 1e9, 2)}
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(s_out)
    s_in.wait_event(a)
    dv.dv_swap_out(ds, 0, hh, 0, 0, L, zero, lens, s_out)
    dv.dv_swap_in(hh, 1, ds, 1, 0, L, zero, lens, s_in)
    s_out.wait_stream(s_in)
    b.record(s_out)
    torch.cuda.synchronize()
    bi_ms = a.elapsed_time(b)
    res["bidirectional"] = {"ms": round(bi_ms, 3),
                            "GBps_total": round(2 * P / (bi_ms * 1e-3) / 1e9, 2)}
    del t_start
    # decode-step increment packs on the compute stream, idle and while both
    # swap directions run on their own streams (slot 0 is read by both the
    # packs and the swap-out; the swap-in writes slot 1)
    comp = torch.cuda.current_stream()
    I = dv.dv_packed_bytes(ds, 0, L, lens, lens + 1)
    inc = torch.empty(I, dtype=torch.uint8, device=dev)
    n_inc = 200

    def time_incs():
        t = Timer(torch, comp)
        with t:
            for _ in range(n_inc):
                dv.dv_stream_out_token(ds, 0, 0, L, lens, inc, I, comp)
        return t

    time_incs()
    torch.cuda.synchronize()
    idle = time_incs()
    torch.cuda.synchronize()
    dv.dv_swap_in(hh, 1, ds, 1, 0, L, zero, lens, s_in)
    dv.dv_swap_out(ds, 0, hh, 0, 0, L, zero, lens, s_out)
    busy = time_incs()
    comp.synchronize()
    still_running = not s_in.query()
    torch.cuda.synchronize()
    res["increments_under_swap"] = {
        "increment_bytes": I, "calls": n_inc,
        "idle_us_per_call": round(idle.mean_ms() * 1e3 / n_inc, 3),
        "during_swaps_us_per_call": round(busy.mean_ms() * 1e3 / n_inc, 3),
        "swaps_still_running_after_packs": still_running,
    }
    # host-link calibration: one contiguous copy of the same byte count
    flat_d = slots[0][:P]
    flat_h = hosts[0][:P]
    tc_o, tc_i = Timer(torch, s_out), Timer(torch, s_in)
    for _ in range(reps):
        with tc_o:
            with torch.cuda.stream(s_out):
                flat_h.copy_(flat_d, non_blocking=True)
        s_out.synchronize()
        with tc_i:
            with torch.cuda.stream(s_in):
                flat_d.copy_(flat_h, non_blocking=True)
        s_in.synchronize()
    res["calibration_contiguous"] = {
        "d2h_GBps": round(P / (tc_o.mean_ms() * 1e-3) / 1e9, 2),
        "h2d_GBps": round(P / (tc_i.mean_ms() * 1e-3) / 1e9, 2)}
    link = read_link()
    res["link"] = link
    res["peak_GBps"] = PCIE_PEAK_GBS
    res["frac_link"] = round(min(res["swap_out"]["GBps"], res["swap_in"]["GBps"]) /
                             PCIE_PEAK_GBS, 4)
    del slots, hosts
    torch.cuda.empty_cache()
    return res


def on_own_stream(torch, fn):
    """Run ``fn`` with a compute stream of its own as torch's current
    stream, as a serving loop would.  The swap scheduler and the streamer
    then put their side streams on hardware queues of their own; from the
    legacy null stream they would share HIP's pooled queues, where a side
    stream can land on the compute stream's queue and serialise with it."""
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        out = fn()
    torch.cuda.synchronize()
    out["compute_stream"] = "a stream of its own (side streams on hardware queues of their own)"
    return out


def swap_protocol_bench(torch, dv, synth, swap_in_gbs):
    """The paper's microbatch swapping protocol on the OPT-66B stage through
    the swap scheduler: 4 host microbatches, 2 device slots, 2 rounds.  Each
    step prefetches the next microbatch, writes one token per layer, runs an
    emulated decode step (a spin kernel, its length measured with events),
    packs the increment and swaps out only the step's update.  Swap-ins
    share the one host link, so the steady-state period should be the
    longer of the step and one swap-in (App. E's max(t, transf_i)); the
    App. E break-even step time for 128 generated tokens is reported too."""
    from paper_2403_01876_amd import swap_model as SM
    dev = torch.device("cuda:0")
    w = synth.make_workload(2)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    M, S_host = w.microbatches, 1024
    compute = torch.cuda.current_stream()
    slots = [torch.empty(w.dense_bytes(), dtype=torch.uint8, device=dev) for _ in range(2)]
    synth.device_fill(slots[0].data_ptr(), w.dense_bytes(), w.data_seed,
                      stream=compute.cuda_stream)
    hosts = [torch.empty(w.dense_bytes(S_host), dtype=torch.uint8, pin_memory=True)
             for _ in range(M)]
    ds = dv.Cache(dv.DV_DENSE, L, H, D, B, slots, max_seq=S)
    hh = dv.Cache(dv.DV_DENSE, L, H, D, B, [h.data_ptr() for h in hosts], max_seq=S_host,
                  mem=dv.DV_MEM_HOST_PINNED)
    zero = np.zeros(B, np.int32)
    for x in range(M):
        dv.dv_swap_out(ds, 0, hh, x, 0, L, zero, w.lens.astype(np.int32), compute)
    I = dv.dv_packed_bytes(ds, 0, L, zero, np.ones(B, np.int32))
    tok = torch.empty(I, dtype=torch.uint8, device=dev)
    inc = torch.empty(I, dtype=torch.uint8, device=dev)
    synth.device_fill(tok.data_ptr(), I, 5, stream=compute.cuda_stream)
    torch.cuda.synchronize()
    # spin-kernel calibration: cycles per ms
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(compute)
    torch.cuda._sleep(10_000_000)
    b.record(compute)
    torch.cuda.synchronize()
    cyc_per_ms = 10_000_000 / a.elapsed_time(b)
    res = {"microbatches": M, "slots": 2, "steps": 2 * M, "increment_bytes": I}
    kv_token = L * 2 * H * D * w.elem_bytes
    bw = swap_in_gbs * 1e9
    runs = []
    transf_ms = SM.transfer_time(int(w.lens[0]), B, kv_token, bw) * 1e3
    # emulated steps below and above the swap-in time: the period must follow
    # the swap-in when it is longer and the step when the step is longer
    for t_ms in (0.0, 40.0, 100.0, 200.0):
        lens = [w.lens.astype(np.int32).copy() for _ in range(M)]
        sw = dv.Swapper(ds, hh)
        sched = list(SM.swap_schedule(M, 2))
        steps = len(sched)
        sw.prefetch(sched[0][0], lens[sched[0][0]])
        torch.cuda.synchronize()
        marks = []
        for x, xn, _ in sched:
            if xn is not None:
                sw.prefetch(xn, lens[xn])
            slot = sw.begin_step(x, compute)
            c0 = torch.cuda.Event(enable_timing=True)
            c1 = torch.cuda.Event(enable_timing=True)
            c0.record(compute)
            pos = lens[x]
            dv.dv_stream_in(ds, slot, 0, L, pos, pos + 1, tok, I, compute)
            if t_ms > 0:
                torch.cuda._sleep(int(t_ms * cyc_per_ms))
            dv.dv_stream_out_token(ds, slot, 0, L, pos, inc, I, compute)
            c1.record(compute)
            sw.end_step(x, pos, pos + 1, compute)
            lens[x] = pos + 1
            marks.append((c0, c1))
        sw.sync()
        torch.cuda.synchronize()
        sw.close()
        if os.environ.get("DV_BENCH_TIMELINE"):
            for k, (c0, c1) in enumerate(marks):
                log(f"  t={t_ms} step {k}: start {marks[0][0].elapsed_time(c0):9.2f} ms, "
                    f"end {marks[0][0].elapsed_time(c1):9.2f} ms")
        compute_ms = sum(c0.elapsed_time(c1) for c0, c1 in marks) / steps
        # steady-state period: between the ends of consecutive steps
        period = marks[0][1].elapsed_time(marks[-1][1]) / (steps - 1)
        runs.append({"emulated_step_ms": round(compute_ms, 3),
                     "measured_period_ms": round(period, 3),
                     "model_period_ms": round(max(compute_ms, transf_ms), 3)})
    res["swap_in_ms_model"] = round(transf_ms, 3)
    res["runs"] = runs
    res["swap_in_GBps_used"] = swap_in_gbs
    res["breakeven_step_ms_128_tokens"] = round(
        SM.breakeven_step_time(128, int(w.lens[0]), B, kv_token, bw) * 1e3, 3)
    del slots, hosts, tok, inc
    torch.cuda.empty_cache()
    return res


def buffered_vs_per_region(torch, dv, synth):
    """The paper's buffered copies (pack into one temporary GPU buffer, then
    one copy) against one copy call per contiguous region (Sec. 5.1, where
    buffered copies were 95x faster streaming to remote CPU memory).  Here
    on the OPT-13B stage, to pinned host memory and within HBM."""
    from paper_2403_01876_amd import baseline
    dev = torch.device("cuda:0")
    w = synth.make_workload(1)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    st = torch.cuda.current_stream()
    cache = torch.empty(w.dense_bytes(), dtype=torch.uint8, device=dev)
    synth.device_fill(cache.data_ptr(), w.dense_bytes(), w.data_seed, stream=st.cuda_stream)
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    out = {}
    cases = {"increment": (w.step_positions(0), w.step_positions(0) + 1),
             "prompt": w.prompt_ranges()}
    for name, (t0, t1) in cases.items():
        n = dv.dv_packed_bytes(c, 0, L, t0, t1)
        stage = torch.empty(n, dtype=torch.uint8, device=dev)
        dst_d = torch.empty(n, dtype=torch.uint8, device=dev)
        dst_h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
        reps = 20 if name == "increment" else 3

        def run(fn):
            fn()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            t_host = time.perf_counter()
            a.record(st)
            for _ in range(reps):
                fn()
            b.record(st)
            torch.cuda.synchronize()
            return min(a.elapsed_time(b), (time.perf_counter() - t_host) * 1e3) / reps, \
                (time.perf_counter() - t_host) * 1e3 / reps

        res = {"bytes": n}
        for where, dst in (("to_host", dst_h), ("in_hbm", dst_d)):
            def per_region():
                baseline.per_region_copy(c, 0, 0, L, t0, t1, dst.data_ptr(), n, st)

            def buffered():
                if name == "increment":
                    dv.dv_stream_out_token(c, 0, 0, L, t0, stage if where == "to_host" else dst,
                                           n, st)
                else:
                    dv.dv_stream_out_prompt(c, 0, 0, L, t0, t1,
                                            stage if where == "to_host" else dst, n, st)
                if where == "to_host":
                    dst.copy_(stage, non_blocking=True)

            _, pr = run(per_region)
            _, bf = run(buffered)
            res[where] = {"per_region_ms": round(pr, 4), "buffered_ms": round(bf, 4),
                          "speedup": round(pr / bf, 1),
                          "regions": 2 * L * H * int((np.asarray(t1) > np.asarray(t0)).sum())}
        out[name] = res
        del stage, dst_d, dst_h
    del cache
    torch.cuda.empty_cache()
    return out


def overlap_bench(torch, dv, synth):
    """Streaming overlapped with computation (the paper's optimisations 2
    and 3 with a background thread), on the OPT-13B stage with emulated
    compute of a 13B model's layer sizes (hidden 5120, 12 h^2 weights per
    layer, bf16 GEMMs): a prompt pass over the stage's 10 layers, each
    followed by streaming that layer's prompt cache to pinned host memory,
    then 32 decode steps, each followed by streaming its increment.

    Three runs: compute alone; compute with the background streamer
    (overlapped); compute with the same packs and copies issued inline on
    the compute stream (not overlapped).  Three interleaved rounds; each
    phase reports its median over them."""
    dev = torch.device("cuda:0")
    w = synth.make_workload(1)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    hidden = H * D
    st = torch.cuda.current_stream()
    cache = torch.empty(w.dense_bytes(), dtype=torch.uint8, device=dev)
    synth.device_fill(cache.data_ptr(), w.dense_bytes(), w.data_seed, stream=st.cuda_stream)
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t0, t1 = w.prompt_ranges()
    P = dv.dv_packed_bytes(c, 0, L, t0, t1)
    staging = torch.empty(P, dtype=torch.uint8, device=dev)
    host = torch.empty(P, dtype=torch.uint8, pin_memory=True)
    ntok = int(np.sum(t1))
    g = torch.Generator(device=dev).manual_seed(0)
    Wt = torch.randn(hidden, 12 * hidden, device=dev, dtype=torch.bfloat16, generator=g)
    Xp = torch.randn(ntok, hidden, device=dev, dtype=torch.bfloat16, generator=g)
    Xt = torch.randn(B, hidden, device=dev, dtype=torch.bfloat16, generator=g)
    layer_off = []
    off = 0
    for l in range(L):
        layer_off.append(off)
        off += dv.dv_packed_bytes(c, l, l + 1, t0, t1)
    steps = 32
    pos = [w.step_positions(i) for i in range(steps)]
    I = dv.dv_packed_bytes(c, 0, L, pos[0], pos[0] + 1)
    ring = 4

    def prompt_compute():
        return torch.mm(Xp, Wt)

    def token_compute():
        for _ in range(L):
            torch.mm(Xt, Wt)

    for _ in range(2):  # warm the GEMMs
        prompt_compute()
        token_compute()
    torch.cuda.synchronize()

    # One streamer, made and used once before the runs, as a serving loop
    # keeps one.  Made inside a run, the GPU idles while the host sets it up
    # and the prompt pass that follows starts at lowered clocks (measured:
    # +5 % on the pass, +8 % with a 0.2 s pause after creation).
    shared = dv.Streamer(c, 0, staging, P, host.data_ptr(), P)
    shared.push(0, 1, t0, t1, 0, stream=st)
    shared.flush()

    def run(mode):
        streamer = None
        if mode == "overlapped":
            streamer = shared
        a = torch.cuda.Event(enable_timing=True)
        m = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(st)
        for l in range(L):
            prompt_compute()
            n = dv.dv_packed_bytes(c, l, l + 1, t0, t1)
            if mode == "overlapped":
                streamer.push(l, l + 1, t0, t1, layer_off[l], stream=st)
            elif mode == "inline":
                dv.dv_stream_out_prompt(c, 0, l, l + 1, t0, t1,
                                        staging[layer_off[l]:], n, st)
                host[layer_off[l]:layer_off[l] + n].copy_(
                    staging[layer_off[l]:layer_off[l] + n], non_blocking=True)
        m.record(st)
        for i in range(steps):
            token_compute()
            if mode == "overlapped":
                streamer.push(0, L, pos[i], pos[i] + 1, (i % ring) * I, (i % ring) * I,
                              stream=st)
            elif mode == "inline":
                so = (i % ring) * I
                dv.dv_stream_out_token(c, 0, 0, L, pos[i], staging[so:], I, st)
                host[so:so + I].copy_(staging[so:so + I], non_blocking=True)
        b.record(st)
        torch.cuda.synchronize()
        if streamer is not None:
            streamer.flush()
        tail = torch.cuda.Event(enable_timing=True)
        tail.record(st)
        torch.cuda.synchronize()
        return {"prompt_ms": a.elapsed_time(m), "token_ms_per_step": m.elapsed_time(b) / steps}

    out = {"prompt_payload_bytes": P, "increment_bytes": I, "decode_steps": steps}
    samples = {}
    for _ in range(3):  # interleaved rounds; each phase's median over them
        for mode in ("compute-only", "overlapped", "inline"):
            samples.setdefault(mode, []).append(run(mode))
    runs = {mode: {k: float(np.median([r[k] for r in rs])) for k in rs[0]}
            for mode, rs in samples.items()}
    for mode, r in runs.items():
        out[mode] = {k: round(v, 4) for k, v in r.items()}
    base, ov, inl = runs["compute-only"], runs["overlapped"], runs["inline"]
    out["prompt_slowdown_overlapped"] = round(ov["prompt_ms"] / base["prompt_ms"] - 1, 4)
    out["prompt_slowdown_inline"] = round(inl["prompt_ms"] / base["prompt_ms"] - 1, 4)
    out["token_slowdown_overlapped"] = round(ov["token_ms_per_step"] /
                                             base["token_ms_per_step"] - 1, 4)
    out["token_slowdown_inline"] = round(inl["token_ms_per_step"] /
                                         base["token_ms_per_step"] - 1, 4)
    # share of the streaming time (what inline streaming adds) that the
    # background streamer hides behind the computation
    for ph, key in (("prompt", "prompt_ms"), ("token", "token_ms_per_step")):
        added = inl[key] - base[key]
        out[f"{ph}_hidden_fraction"] = (round(1 - (ov[key] - base[key]) / added, 4)
                                        if added > 0 else None)
    shared.close()
    del cache, staging, host, Wt, Xp, Xt
    torch.cuda.empty_cache()
    return out


def ring_recovery_bench(torch, dv, synth):
    """Ring replication and the four-step recovery (Sec. 4.2.3) on one GPU:
    four pipeline stages shaped like the BLOOM-176B shard (10 layers, 14 heads
    x 128, batch 16) with two microbatches each, prompts of the shard
    workload clipped to 1024 tokens, 16 decode steps with every step's
    increment streamed to the next stage.  Stage 1 fails after computing
    microbatch 1's step 12 and before streaming it; the recovery transfers
    (replica back, predecessor's cache to the failed stage's replica slot)
    are timed."""
    from paper_2403_01876_amd.ring import RingSim
    w = synth.make_workload(3)
    lens = np.minimum(w.lens, 1024).astype(np.int32)
    lens2 = np.minimum(w.lens[::-1], 1024).astype(np.int32)
    sim = RingSim(workers=4, microbatches=2, layers=10, heads=14, head_dim=128, batch=16,
                  max_seq=1024 + 16, prompt_lens=[lens, lens2], seed=3)
    st = torch.cuda.current_stream()
    sim.prefill()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(st)
    stopped = sim.run((0, 0), (0, 16), fail_at=(1, 1, 12))
    b.record(st)
    torch.cuda.synchronize()
    assert stopped
    per_step = a.elapsed_time(b) / (12 * 2 + 2)
    # bytes the recovery moves: stage 1's valid cache (from its replica) and
    # stage 0's (into stage 1's replica slot)
    zero = np.zeros(16, np.int32)
    moved = 0
    for j in range(2):
        held = sim.table.steps_held(2, j)
        moved += dv.dv_packed_bytes(sim.c[1], 0, 10, zero, sim.prompt[j] + held)
        moved += dv.dv_packed_bytes(sim.c[0], 0, 10, zero,
                                    sim.prompt[j] + sim._steps(sim.done[0], j))
    sim.fail(1)
    torch.cuda.synchronize()
    a.record(st)
    resume = sim.recover(1)
    b.record(st)
    torch.cuda.synchronize()
    rec_ms = a.elapsed_time(b)
    sim.run(resume, (0, 16))
    torch.cuda.synchronize()
    out = {"stages": 4, "microbatches": 2, "steps": 16, "failed_stage": 1,
           "fail_after": [1, 12], "resume_point": list(resume),
           "ms_per_step_all_stages_with_replication": round(per_step, 4),
           "recovery_ms": round(rec_ms, 4), "recovery_bytes": moved,
           "recovery_GBps_2x": round(2 * moved / (rec_ms * 1e-3) / 1e9, 1)}
    del sim
    torch.cuda.empty_cache()
    return out


def device_facts(torch):
    """What the runtime reports about the GPU the numbers come from."""
    p = torch.cuda.get_device_properties(0)
    out = {"name": p.name, "compute_units": p.multi_processor_count,
           "hbm_bytes": p.total_memory}
    for k in ("gcnArchName", "L2_cache_size", "shared_memory_per_block"):
        if hasattr(p, k):
            out[k] = getattr(p, k)
    return out


def read_link():
    """PCIe link speed/width of the GPU from sysfs (best effort)."""
    import glob
    out = {}
    for d in glob.glob("/sys/class/drm/card*/device"):
        try:
            vendor = open(os.path.join(d, "vendor")).read().strip()
            if vendor != "0x1002":
                continue
            for k in ("current_link_speed", "current_link_width", "max_link_speed",
                      "max_link_width"):
                p = os.path.join(d, k)
                if os.path.exists(p):
                    out[k] = open(p).read().strip()
            if out:
                break
        except OSError:
            continue
    return out or None


def copy_calibration(torch, nbytes=4 << 30):
    """Device-to-device copy of a known size: torch copy kernel and DMA."""
    dev = torch.device("cuda:0")
    a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    b = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    a.fill_(1)
    stream = torch.cuda.current_stream()
    t = Timer(torch, stream)
    for i in range(6):
        if i >= 2:
            with t:
                b.copy_(a)
        else:
            b.copy_(a)
    torch.cuda.synchronize()
    ms = t.mean_ms()
    del a, b
    torch.cuda.empty_cache()
    return {"bytes": nbytes, "ms": round(ms, 4),
            "GBps_2x": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}


def cpu_baseline(torch, dv, synth, reps=3):
    """The oracle on the host cores, on the headline workload (the LLaMA-2-70B
    paged pool): paged gather through table A, then scatter of that buffer
    into a zeroed pool through table B.

    * Multi-threaded: all 20 layers, one oracle call per layer [l, l+1) on as
      many host threads as the process's CPU affinity allows (layer ranges
      concatenate, so the slabs are independent); the oracle's code is the
      same.  This is ``value``.
    * Single-threaded: layers [0, 2), one oracle call per operation.
    Each is the median of ``reps`` runs, in the step's GB/s (2 x payload per
    operation).  The multi-threaded run's gather buffer and pool are then
    compared over every byte with one gather and one pool-order scatter of
    the GPU on the same generated pool."""
    import oracle
    from oracle import par

    w = synth.make_workload(4)
    orc = oracle.get()
    threads = par.host_threads()
    la = oracle.Layout(oracle.PAGED, w.layers, w.heads, w.head_dim, w.batch,
                       block_size=w.block_size, num_blocks=w.num_blocks,
                       block_table=w.block_table_a)
    lb = oracle.Layout(oracle.PAGED, w.layers, w.heads, w.head_dim, w.batch,
                       block_size=w.block_size, num_blocks=w.num_blocks,
                       block_table=w.block_table_b)
    t0, t1 = w.prompt_ranges()
    pool = synth.fill_bytes_parallel(la.storage_bytes(), w.data_seed)
    recv = np.zeros(lb.storage_bytes(), np.uint8)

    def timed(fn):
        a = time.perf_counter()
        out = fn()
        return time.perf_counter() - a, out

    # multi-threaded, all layers
    mt = []
    wire = None
    for _ in range(reps):
        tg, wire = timed(lambda: par.pack(orc, la, pool, 0, w.layers, t0, t1, threads))
        recv[:] = 0
        ts, _ = timed(lambda: par.unpack(orc, lb, recv, 0, w.layers, t0, t1, wire, threads))
        mt.append((tg, ts))
    P = wire.nbytes
    # single-threaded, layers [0, 2)
    l1 = 2
    st = []
    for _ in range(reps):
        part = np.empty(orc.wire_elems(la, 0, l1, t0, t1) * 2, np.uint8)
        tg, _ = timed(lambda: orc.pack_into(la, pool, 0, l1, t0, t1, part))
        scratch = np.zeros(lb.storage_bytes() // w.layers * l1, np.uint8)
        lb2 = oracle.Layout(oracle.PAGED, l1, w.heads, w.head_dim, w.batch,
                            block_size=w.block_size, num_blocks=w.num_blocks,
                            block_table=w.block_table_b)
        ts, _ = timed(lambda: orc.unpack(lb2, scratch, 0, l1, t0, t1, part))
        st.append((tg, ts))
    Pst = part.nbytes
    del scratch, part
    med = lambda xs: float(np.median(xs))  # noqa: E731
    mt_s = med([g + x for g, x in mt])
    st_s = med([g + x for g, x in st])

    # the GPU on the same generated pool, compared over every byte
    dev = torch.device("cuda:0")
    s = torch.cuda.current_stream()
    pa = torch.empty(la.storage_bytes(), dtype=torch.uint8, device=dev)
    synth.device_fill(pa.data_ptr(), la.storage_bytes(), w.data_seed, stream=s.cuda_stream)
    pb = torch.zeros(lb.storage_bytes(), dtype=torch.uint8, device=dev)
    own = torch.empty(w.num_blocks * 4, dtype=torch.uint8, device=dev)
    kw = dict(block_size=w.block_size, num_blocks=w.num_blocks, max_blocks=w.max_blocks)
    ca = dv.Cache(dv.DV_PAGED, w.layers, w.heads, w.head_dim, w.batch, [pa],
                  block_tables=[torch.from_numpy(w.block_table_a).to(dev)], **kw)
    cb = dv.Cache(dv.DV_PAGED, w.layers, w.heads, w.head_dim, w.batch, [pb],
                  block_tables=[torch.from_numpy(w.block_table_b).to(dev)], block_owners=[own],
                  **kw)
    gw = torch.empty(P, dtype=torch.uint8, device=dev)
    dv.dv_stream_out_prompt(ca, 0, 0, w.layers, t0, t1, gw, P, s)
    dv.dv_stream_in(cb, 0, 0, w.layers, t0, t1, gw, P, s)
    torch.cuda.synchronize()
    gw_h, pb_h = gw.cpu().numpy(), pb.cpu().numpy()
    del pa, pb, gw, own, ca, cb
    torch.cuda.empty_cache()
    parity = {"gather_buffer_bytes": P,
              "gather_buffer_equal": bool(np.array_equal(gw_h, wire)),
              "scattered_pool_bytes": int(recv.nbytes),
              "scattered_pool_equal": bool(np.array_equal(pb_h, recv))}
    del gw_h, pb_h, wire, recv, pool
    return {
        "value": round(2 * 2 * P / mt_s / 1e9, 3), "unit": "GB/s", "cores": threads,
        "kind": "oracle",
        "sample": (f"LLaMA-2-70B paged pool, all {w.layers} layers: gather through table A "
                   f"({P} B) + scatter into a zeroed pool through table B; one oracle call "
                   f"per layer on {threads} threads; median of {reps} "
                   f"({med([g for g, _ in mt]):.2f} s gather, {med([x for _, x in mt]):.2f} s "
                   f"scatter)"),
        "single_thread": {
            "value": round(2 * 2 * Pst / st_s / 1e9, 3), "unit": "GB/s", "cores": 1,
            "sample": (f"the same, layers [0, {l1}) ({Pst} B), one call per operation; median "
                       f"of {reps} ({med([g for g, _ in st]):.2f} s gather, "
                       f"{med([x for _, x in st]):.2f} s scatter)")},
        "parity_vs_gpu": parity,
        "host_cpu": cpu_model(),
        "affinity_cores": threads,
        "per_op": cpu_baseline_per_op(orc),
    }


def cpu_baseline_per_op(orc):
    """The oracle, single-threaded, on the other operations the benchmark
    times, each on a bounded sample of its workload (layer 0 of the stage, or
    one decode step), in the same 2 x payload GB/s."""
    import oracle
    import synth

    out = {}

    def rate(nbytes, fn):
        a = time.perf_counter()
        fn()
        return round(2 * nbytes / (time.perf_counter() - a) / 1e9, 3)

    # OPT-13B stage prompt, all 10 layers, one call each way
    w = synth.make_workload(1)
    ld = oracle.Layout(oracle.DENSE, w.layers, w.heads, w.head_dim, w.batch, seq_cap=w.max_seq)
    cache = synth.fill_bytes_parallel(ld.storage_bytes(), w.data_seed)
    t0, t1 = w.prompt_ranges()
    box = {}
    po = rate(orc.wire_elems(ld, 0, w.layers, t0, t1) * 2,
              lambda: box.setdefault("wire", orc.pack(ld, cache, 0, w.layers, t0, t1)))
    recv = np.zeros_like(cache)
    pi = rate(box["wire"].nbytes, lambda: orc.unpack(ld, recv, 0, w.layers, t0, t1, box["wire"]))
    out["opt13b-stage prompt"] = {"pack_GBps_2x": po, "unpack_GBps_2x": pi,
                                  "sample": f"all {w.layers} layers, {box['wire'].nbytes} B"}
    del cache, recv, box
    # split key: OPT-13B stage, layer 0 of 10
    lk = oracle.Layout(oracle.KSPLIT, 1, w.heads, w.head_dim, w.batch, seq_cap=w.max_seq)
    cache = synth.fill_bytes(lk.storage_bytes(), w.data_seed)
    t0, t1 = w.prompt_ranges()
    box = {}
    pk = rate(orc.wire_elems(lk, 0, 1, t0, t1) * 2,
              lambda: box.setdefault("wire", orc.pack(lk, cache, 0, 1, t0, t1)))
    recv = np.zeros_like(cache)
    uk = rate(box["wire"].nbytes, lambda: orc.unpack(lk, recv, 0, 1, t0, t1, box["wire"]))
    out["opt13b-stage split-key"] = {"pack_GBps_2x": pk, "unpack_GBps_2x": uk,
                                     "sample": f"layer 0 of {w.layers}, {box['wire'].nbytes} B "
                                               "payload"}
    # one decode-step increment of the OPT-13B stage, layer 0 (the split-key
    # sample's value half is dense, so its cache serves as a dense layer)
    ld = oracle.Layout(oracle.DENSE, 1, w.heads, w.head_dim, w.batch, seq_cap=w.max_seq)
    p = w.step_positions(0)
    inc = orc.wire_elems(ld, 0, 1, p, p + 1) * 2
    box = {}
    ti = rate(inc, lambda: [box.setdefault(k, orc.pack(ld, cache, 0, 1, p, p + 1))
                            for k in range(10)])
    out["opt13b-stage increment"] = {"pack_GBps_2x": round(ti * 10, 3),
                                     "sample": f"one step of layer 0, {inc} B, 10 calls"}
    del cache, recv, box
    # swap copy: OPT-66B microbatch, layer 0 of 16, slot to a 1024-token mirror
    w = synth.make_workload(2)
    sd = oracle.Layout(oracle.DENSE, 1, w.heads, w.head_dim, w.batch, seq_cap=w.max_seq)
    hd = oracle.Layout(oracle.DENSE, 1, w.heads, w.head_dim, w.batch, seq_cap=1024)
    slot = synth.fill_bytes(sd.storage_bytes(), w.data_seed)
    host = np.zeros(hd.storage_bytes(), np.uint8)
    t0, t1 = w.prompt_ranges()
    moved = orc.wire_elems(sd, 0, 1, t0, t1) * 2
    sw = rate(moved, lambda: orc.copy_ranges(sd, slot, hd, host, 0, 1, t0, t1))
    out["opt66b-stage swap copy"] = {"GBps_2x": sw, "sample": f"layer 0 of {w.layers}, "
                                                              f"{moved} B"}
    return out


def counted_traffic(profile: str, key: str):
    """HBM bytes per launch from the ``key`` line of the committed counter
    summary ``profiles/<profile>``, or None if the kernel sources changed
    since the counters were taken (the summary records their hash)."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", profile)
    try:
        text = open(path).read()
    except OSError:
        return None
    m_sha = re.search(r"^kernel_source_sha256: ([0-9a-f]{64})$", text, re.M)
    m_t = re.search(r"^%s: (\d+)$" % re.escape(key), text, re.M)
    if not (m_sha and m_t):
        return None
    return int(m_t.group(1)) if kernel_source_sha256() == m_sha.group(1) else None


def kernel_source_sha256() -> str:
    """Hash of the streaming kernels' sources (the kernels and their launch
    descriptors), recorded with each counter summary."""
    import hashlib
    h = hashlib.sha256()
    for f in ("dv_kernels.hip", "dv_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2403_01876_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


import numpy as np  # noqa: E402


DENSE_TRAFFIC = "dense_runs_hbm_traffic_opt13b_stage.md"
PAGED_TRAFFIC = "paged_kernel_hbm_traffic_llama2_70b_paged.md"


def gbs2(nbytes, ms):
    """Algorithmic GB/s of an operation moving ``nbytes`` of payload (each
    byte read once and written once) in ``ms``."""
    return 2 * nbytes / (ms * 1e-3) / 1e9


def opt13b_step(args, torch, dv, synth):
    """The OPT-13B stage step with its dense pack kernel's roofline and copy
    ceiling."""
    w, r = main_step_bench(args, torch, dv, synth)
    pack_gbs, unpack_gbs, copy_gbs = (gbs2(r["P"], r[k]) for k in ("pack_ms", "unpack_ms",
                                                                      "copy_ms"))
    return {
        "workload": ("opt13b-stage: 10 layers x 40 heads x 128 dims, batch 8, capacity 2048, "
                     "fp16 dense [layer][K|V][batch][head][seq][dim], prompts U[512,1024] from "
                     "seed 1; step = prompt stream-out + stream-in + 128 x (increment out + "
                     "in)"),
        "value": round(r["value"], 2), "unit": "GB/s", "ms_per_step": round(r["ms"], 4),
        "eager_ms_per_step": round(r["eager_ms"], 4), "graph_ms_per_step": round(r["graph_ms"], 4),
        "payload_prompt_bytes": r["P"], "payload_increment_bytes": r["I"],
        "algorithmic_bytes_per_step": r["step_bytes"], "checks": r["checks"],
        "roofline": {
            "kernel": "dense_runs_kernel<pack> (prompt stream-out)", "bound": "hbm",
            "achieved": round(pack_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(pack_gbs / HBM_PEAK_GBS, 4),
            "traffic": counted_traffic(DENSE_TRAFFIC, "traffic_bytes_per_launch"),
            "avg_ms": round(r["pack_ms"], 4), "bytes_per_launch": 2 * r["P"],
            "copy_ceiling": {
                "what": "plain contiguous 16-byte copy of the same P bytes in the pack "
                        "kernel's launch shape (libdv_baseline dvb_plain_copy)",
                "avg_ms": round(r["copy_ms"], 4), "GBps": round(copy_gbs, 1),
                "frac": round(copy_gbs / HBM_PEAK_GBS, 4),
                "kernel_vs_copy": round(pack_gbs / copy_gbs, 4)},
        },
        "dense_runs_kernel<unpack>": {
            "avg_ms": round(r["unpack_ms"], 4), "GBps_2x": round(unpack_gbs, 1),
            "frac_hbm": round(unpack_gbs / HBM_PEAK_GBS, 4),
            "kernel_vs_copy": round(unpack_gbs / copy_gbs, 4),
            "traffic": counted_traffic(DENSE_TRAFFIC, "traffic_bytes_per_launch_unpack")},
    }


def roofline_rows(out, paged):
    """One row per (workload, bulk operation) measured in this run: the
    kernel, its GB/s and its fraction of the roofline (HBM, or the host link
    for swaps)."""
    rows = []

    def row(cfg, op, kernel, gbs, peak=HBM_PEAK_GBS, bound="hbm", cache="warm, back to back"):
        rows.append({"config": cfg, "op": op, "kernel": kernel, "bound": bound,
                     "GBps": round(gbs, 1), "peak": peak, "frac": round(gbs / peak, 4),
                     "cache_state": cache})

    k, P = paged["kern"], paged["P"]
    row("llama2-70b-paged", "paged gather (table order)", "paged_kernel<pack>",
        gbs2(P, k["gather"]))
    row("llama2-70b-paged", "paged scatter, pool order (owner map included)",
        "owner_clear/build + paged_kernel<unpack>", gbs2(P, k["scatter_pool_order"]))
    row("llama2-70b-paged", "paged scatter, table order", "paged_kernel<unpack>",
        gbs2(P, k["scatter_table_order"]))
    step = out.get("opt13b_step")
    if step:
        row("opt13b-stage", "prompt stream-out", "dense_runs_kernel<pack>",
            step["roofline"]["achieved"])
        row("opt13b-stage", "prompt stream-in", "dense_runs_kernel<unpack>",
            step["dense_runs_kernel<unpack>"]["GBps_2x"])
    cold = "cold: 512 MB written between calls"
    for name, res in out.get("bulk", {}).items():
        for op in ("stream_out", "stream_in", "stream_in_table_order"):
            if op in res:
                row(name, op, "paged_kernel" if "paged" in name else
                    ("ksplit_kernel + dense_runs_kernel" if "split" in name
                     else "dense_runs_kernel"), res[op]["GBps_2x"], cache=cold)
    sw = out.get("swap")
    if sw:
        for op in ("swap_out", "swap_in"):
            row("opt66b-stage-swap", op, "hipMemcpy2DAsync (DMA)", sw[op]["GBps"],
                peak=PCIE_PEAK_GBS, bound="host link", cache="n/a")
    tiny = out.get("tiny")
    if tiny:
        rows.append({"config": "tiny-dense", "op": "prompt stream-out / stream-in",
                     "kernel": "dense_runs_kernel", "bound": "latency",
                     "frac": None, "note": tiny["note"]})
    return rows


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: the streaming path has no cross-GPU step "
              f"here (asked for --gpus {args.gpus}, WORLD_SIZE {world})", file=sys.stderr)
        sys.exit(2)
    import torch

    import synth
    from paper_2403_01876_amd import dv

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    log(f"device: {torch.cuda.get_device_name(0)}")
    w, r = paged_step_bench(args, torch, dv, synth)
    k, P = r["kern"], r["P"]
    g_gbs = gbs2(P, k["gather"])
    copy_gbs = gbs2(P, k["plain_copy"])
    rr_gbs = gbs2(r["pool_bytes"], k["block_copy_random_reads"])
    rw_gbs = gbs2(r["pool_bytes"], k["block_copy_random_writes"])
    sp_gbs = gbs2(P, k["scatter_pool_order"])
    st_gbs = gbs2(P, k["scatter_table_order"])
    out = {
        "metric": METRIC,
        "value": round(r["value"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u16",
        "data": "synthetic",
        "device": device_facts(torch),
        "config": {
            "workload": (f"llama2-70b-paged: 20 of 80 layers x 8 KV heads x 128 dims, block 16 "
                         f"tokens, 32 sequences U[128,4096] from seed 4, fp16 pool "
                         f"[layer][K|V][block][head][slot][dim] of {r['num_blocks']} blocks, "
                         f"tables A and B random permutations of it; step = paged gather "
                         f"through table A + scatter through table B (pool order) + 128 x "
                         f"(tail-block increment out of pool A + into pool B)"),
            "payload_gather_bytes": P,
            "payload_increment_bytes": r["I"],
            "pool_bytes": r["pool_bytes"],
            "algorithmic_bytes_per_step": r["step_bytes"],
            "step_issue": "eager" if args.eager else "hip graph replay",
            "eager_ms_per_step": round(r["eager_ms"], 4),
            "graph_ms_per_step": round(r["graph_ms"], 4),
            "checks": r["checks"],
        },
        "roofline": {
            "kernel": "paged_kernel<pack> (paged gather through table A)",
            "bound": "hbm",
            "achieved": round(g_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(g_gbs / HBM_PEAK_GBS, 4),
            "traffic": counted_traffic(PAGED_TRAFFIC, "traffic_bytes_per_launch"),
            "avg_ms": round(k["gather"], 4),
            "bytes_per_launch": 2 * P,
            "copy_ceiling": {
                "what": "plain contiguous 16-byte copy of P bytes from pool A into the "
                        "gather's buffer, in the dense kernels' launch shape (dvb_plain_copy)",
                "avg_ms": round(k["plain_copy"], 4), "GBps": round(copy_gbs, 1),
                "frac": round(copy_gbs / HBM_PEAK_GBS, 4),
                "kernel_vs_copy": round(g_gbs / copy_gbs, 4)},
            "block_order_ceiling": {
                "what": "plain copy of the whole pool block by block in table A's order, "
                        "random 32 KB block reads and sequential writes, in the paged "
                        "kernel's launch shape (dvb_block_copy): the gather's block "
                        "placement without its ranges and head split",
                "bytes": 2 * r["pool_bytes"],
                "avg_ms": round(k["block_copy_random_reads"], 4), "GBps": round(rr_gbs, 1),
                "frac": round(rr_gbs / HBM_PEAK_GBS, 4),
                "kernel_vs_ceiling": round(g_gbs / rr_gbs, 4)},
        },
        "kernels": {
            "paged scatter, pool order (owner map + paged_kernel<unpack>)": {
                "avg_ms": round(k["scatter_pool_order"], 4), "GBps_2x": round(sp_gbs, 1),
                "frac_hbm": round(sp_gbs / HBM_PEAK_GBS, 4),
                "traffic": counted_traffic(PAGED_TRAFFIC,
                                           "traffic_bytes_per_launch_scatter_pool_order")},
            "paged scatter, table order (paged_kernel<unpack>)": {
                "avg_ms": round(k["scatter_table_order"], 4), "GBps_2x": round(st_gbs, 1),
                "frac_hbm": round(st_gbs / HBM_PEAK_GBS, 4),
                "traffic": counted_traffic(PAGED_TRAFFIC,
                                           "traffic_bytes_per_launch_scatter_table_order"),
                "block_order_ceiling": {
                    "what": "the same block copy with random block writes and sequential "
                            "reads: the table-order scatter's placement",
                    "avg_ms": round(k["block_copy_random_writes"], 4),
                    "GBps": round(rw_gbs, 1), "frac": round(rw_gbs / HBM_PEAK_GBS, 4),
                    "kernel_vs_ceiling": round(st_gbs / rw_gbs, 4)}},
        },
    }
    extras = "none" if args.no_extras else args.extras
    errors = {}

    def extra(key, label, fn):
        """Run one extra measurement.  A Python-level failure (an allocation
        refused on a box with less pinned memory, say) is recorded in the
        line's ``errors`` and on stderr instead of losing the line."""
        if label:
            log(f"extras: {label}")
        try:
            out[key] = fn()
        except Exception as e:  # noqa: BLE001 -- reported, not swallowed
            errors[key] = f"{type(e).__name__}: {e}"
            log(f"extras: {key} failed: {errors[key]}")
            torch.cuda.synchronize()
            torch.cuda.empty_cache()

    if extras != "none":
        extra("opt13b_step", "OPT-13B stage step", lambda: opt13b_step(args, torch, dv, synth))
    if extras == "calib":
        extra("calibration_d2d_copy", "", lambda: copy_calibration(torch))
    if extras == "bulk":
        extra("bulk", "", lambda: bulk_all(torch, dv, synth))
        extra("calibration_d2d_copy", "", lambda: copy_calibration(torch))
    if extras == "swap":
        extra("swap", "swap", lambda: swap_bench(torch, dv, synth))
        if "swap" in out:
            extra("swap_protocol", "swap protocol", lambda: on_own_stream(
                torch, lambda: swap_protocol_bench(torch, dv, synth,
                                                   out["swap"]["swap_in"]["GBps"])))
    if extras == "all":
        extra("increments", "increments", lambda: increments_bench(torch, dv, synth))
        extra("multi_token_steps", "multi-token steps",
              lambda: multi_token_bench(torch, dv, synth))
        extra("tiny", "tiny workload", lambda: tiny_bench(torch, dv, synth))
        extra("bulk", "", lambda: bulk_all(torch, dv, synth))
        extra("swap", "swap", lambda: swap_bench(torch, dv, synth))
        if "swap" in out:
            extra("swap_protocol", "swap protocol", lambda: on_own_stream(
                torch, lambda: swap_protocol_bench(torch, dv, synth,
                                                   out["swap"]["swap_in"]["GBps"])))
        extra("overlap", "streaming overlapped with compute",
              lambda: on_own_stream(torch, lambda: overlap_bench(torch, dv, synth)))
        extra("ring_recovery", "ring replication and recovery",
              lambda: ring_recovery_bench(torch, dv, synth))
        extra("buffered_vs_per_region", "buffered vs per-region copies",
              lambda: buffered_vs_per_region(torch, dv, synth))
        extra("calibration_d2d_copy", "copy calibration", lambda: copy_calibration(torch))
    out["rooflines"] = roofline_rows(out, r)
    if not args.no_cpu_baseline:
        extra("cpu_baseline", "cpu baseline (oracle)", lambda: cpu_baseline(torch, dv, synth))
    if errors:
        out["errors"] = errors
    # device memory the run held at its peak (every cache, pool and buffer is
    # a torch allocation; pinned host mirrors are not device memory)
    out["device"]["peak_allocated_bytes"] = int(torch.cuda.max_memory_allocated())
    print(json.dumps(out), flush=True)
    failed = [k for k, v in r["checks"].items() if not v]
    failed += [f"opt13b_step: {k}" for k, v in out.get("opt13b_step", {}).get("checks",
                                                                            {}).items() if not v]
    for name, res in out.get("bulk", {}).items():
        failed += [f"{name}: {k}" for k, v in res.items() if k.startswith("check_") and not v]
    par = out.get("cpu_baseline", {}).get("parity_vs_gpu", {})
    failed += [f"cpu_baseline: {k}" for k, v in par.items() if k.endswith("_equal") and not v]
    if failed:
        log("checks failed, numbers invalid: " + ", ".join(failed))
        sys.exit(1)


if __name__ == "__main__":
    main()

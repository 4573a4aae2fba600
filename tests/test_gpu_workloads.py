"""The five synthetic workloads at full size, in the launch configuration the
benchmark times, compared with the oracle over every byte.

Each GPU input is the seeded generator's device fill; the oracle reads the
same generator's host fill (the two fills are independent implementations of
one definition).  The oracle runs one layer per call on host threads
(``oracle/par.py``; layer ranges concatenate), and each GPU result --
contiguous buffer, receiver cache or paged pool -- is compared with the
oracle's whole result on the device.  Receivers start from a sentinel byte,
so bytes a stream must leave alone are compared too.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2403_01876_amd import dv  # noqa: E402
from tests import gpu_util as G  # noqa: E402
from oracle import par as OP  # noqa: E402

SENTINEL = 0xA5


def stream():
    return torch.cuda.current_stream()


def say(msg):
    print(msg, flush=True)


def dense_layout(w, kind=oracle.DENSE):
    return oracle.Layout(kind, w.layers, w.heads, w.head_dim, w.batch, seq_cap=w.max_seq,
                         elem_bytes=w.elem_bytes)


def paged_layout(w, table):
    return oracle.Layout(oracle.PAGED, w.layers, w.heads, w.head_dim, w.batch,
                         elem_bytes=w.elem_bytes, block_size=w.block_size,
                         num_blocks=w.num_blocks, block_table=table)


def filled_pair(nbytes, seed):
    """The generator's bytes on the host (oracle input) and on the device
    (GPU input)."""
    return synth.fill_bytes_parallel(nbytes, seed), G.dev_filled(nbytes, seed)


def test_tiny_workload_bit_exact(oracle_lib):
    """Prompt of 100 tokens for both sequences, 16 increments, empty receiver."""
    w = synth.make_workload(0)
    lay = dense_layout(w)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    zero = np.zeros(B, np.int32)
    hi = (w.lens + w.steps).astype(np.int32)
    gen = synth.fill_bytes(lay.storage_bytes(), w.data_seed)
    sender_h = np.zeros(lay.storage_bytes(), np.uint8)
    oracle_lib.unpack(lay, sender_h, 0, L, zero, hi, oracle_lib.pack(lay, gen, 0, L, zero, hi))
    sender = G.to_dev(sender_h)
    recv = G.dev_const(lay.storage_bytes(), 0)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [sender], max_seq=S)
    cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S)
    t0, t1 = w.prompt_ranges()
    wire = torch.empty(409600, dtype=torch.uint8, device=G.DEV)
    assert dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, wire.numel(), stream()) == 409600
    dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, 409600, stream())
    torch.cuda.synchronize()
    assert G.host(wire).tobytes() == oracle_lib.pack(lay, sender_h, 0, L, t0, t1).tobytes()
    inc = torch.empty(4096, dtype=torch.uint8, device=G.DEV)
    for i in range(w.steps):
        p = w.step_positions(i)
        assert dv.dv_stream_out_token(cs, 0, 0, L, p, inc, 4096, stream()) == 4096
        dv.dv_stream_in(cr, 0, 0, L, p, p + 1, inc, 4096, stream())
        torch.cuda.synchronize()
        assert G.host(inc).tobytes() == oracle_lib.pack(lay, sender_h, 0, L, p, p + 1).tobytes()
    assert G.host(recv).tobytes() == sender_h.tobytes()


def increments_both_sides(orc, lay, recv_lay, gen_h, recv_exp, w, cs, cr, L):
    """The workload's decode steps: on the GPU each step's increment is packed
    out of the sender into its own slot of one buffer and streamed into the
    receiver; on the host the oracle packs the same steps from the generator
    (sender layout ``lay``) and unpacks them into the expected receiver
    (layout ``recv_lay``).  Returns the GPU buffer of all increments and the
    oracle's."""
    p0 = w.step_positions(0)
    inc_n = dv.dv_packed_bytes(cs, 0, L, p0, p0 + 1)
    incs = torch.empty(w.steps * inc_n, dtype=torch.uint8, device=G.DEV)
    for i in range(w.steps):
        p = w.step_positions(i)
        slot = incs[i * inc_n:(i + 1) * inc_n]
        assert dv.dv_stream_out_token(cs, 0, 0, L, p, slot, inc_n, stream()) == inc_n
        dv.dv_stream_in(cr, 0, 0, L, p, p + 1, slot, inc_n, stream())
    exp = np.empty(w.steps * inc_n, np.uint8)
    for i in range(w.steps):
        p = w.step_positions(i)
        part = exp[i * inc_n:(i + 1) * inc_n]
        part[:] = OP.pack(orc, lay, gen_h, 0, L, p, p + 1)
        OP.unpack(orc, recv_lay, recv_exp, 0, L, p, p + 1, part)
    return incs, exp, inc_n


def test_opt13b_stage_prompt_and_increments(oracle_lib):
    """Prompt stream-out and stream-in into a sentinel receiver, then 128
    decode steps: the prompt buffer, every increment and the final receiver
    against the oracle."""
    w = synth.make_workload(1)
    lay = dense_layout(w)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    gen_h, cache = filled_pair(lay.storage_bytes(), w.data_seed)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    recv = G.dev_const(lay.storage_bytes(), SENTINEL)
    cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S)
    t0, t1 = w.prompt_ranges()
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    assert dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, n, stream()) == n
    dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, n, stream())
    exp_wire = OP.pack(oracle_lib, lay, gen_h, 0, L, t0, t1)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, "prompt stream-out")
    recv_exp = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, recv_exp, 0, L, t0, t1, exp_wire)
    del exp_wire
    incs, exp_incs, inc_n = increments_both_sides(oracle_lib, lay, lay, gen_h, recv_exp, w,
                                                  cs, cr, L)
    assert inc_n == 1638400
    torch.cuda.synchronize()
    G.assert_same_bytes(incs, exp_incs, "128 increments")
    G.assert_same_bytes(recv, recv_exp, "receiver after prompt + 128 increments")


def test_opt13b_stage_split_key_full_size(oracle_lib):
    """The OPT-13B stage stored with the split-key layout, as the benchmark
    times it: stream-out, and stream-in into a sentinel receiver."""
    w = synth.make_workload(1)
    lay = dense_layout(w, oracle.KSPLIT)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    gen_h, cache = filled_pair(lay.storage_bytes(), w.data_seed)
    cs = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [cache], max_seq=S)
    t0, t1 = w.prompt_ranges()
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, n, stream())
    recv = G.dev_const(lay.storage_bytes(), SENTINEL)
    cr = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [recv], max_seq=S)
    dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, n, stream())
    exp_wire = OP.pack(oracle_lib, lay, gen_h, 0, L, t0, t1)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, "split-key stream-out")
    recv_exp = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, recv_exp, 0, L, t0, t1, exp_wire)
    G.assert_same_bytes(recv, recv_exp, "split-key receiver")


def test_opt66b_microbatch_prompt_full_size(oracle_lib):
    """One OPT-66B stage microbatch (4.7 GB payload) streamed out and into a
    sentinel receiver, as the benchmark's bulk measurement times it."""
    w = synth.make_workload(2)
    lay = dense_layout(w)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    gen_h, cache = filled_pair(lay.storage_bytes(), w.data_seed)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t0, t1 = w.prompt_ranges()
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    assert n == 4718592000
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, n, stream())
    recv = G.dev_const(lay.storage_bytes(), SENTINEL)
    cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S)
    dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, n, stream())
    exp_wire = OP.pack(oracle_lib, lay, gen_h, 0, L, t0, t1)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, "OPT-66B microbatch stream-out")
    del gen_h
    recv_exp = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, recv_exp, 0, L, t0, t1, exp_wire)
    G.assert_same_bytes(recv, recv_exp, "OPT-66B receiver")


def test_bloom_shard_replicate_and_restore(oracle_lib):
    """Full valid cache -> contiguous replica; the cache is lost (poisoned);
    restore from the replica."""
    w = synth.make_workload(3)
    lay = dense_layout(w)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    gen_h, cache = filled_pair(lay.storage_bytes(), w.data_seed)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t0, t1 = w.prompt_ranges()
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    replica = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, replica, n, stream())
    exp_rep = OP.pack(oracle_lib, lay, gen_h, 0, L, t0, t1)
    torch.cuda.synchronize()
    G.assert_same_bytes(replica, exp_rep, "BLOOM replica")
    cache.fill_(SENTINEL)  # the worker's cache is lost
    dv.dv_stream_in(cs, 0, 0, L, t0, t1, replica, n, stream())
    exp = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, exp, 0, L, t0, t1, exp_rep)
    torch.cuda.synchronize()
    G.assert_same_bytes(cache, exp, "BLOOM restored cache")


def test_bloom_shard_restore_from_random_replica(oracle_lib):
    """Restore from a replica of generated bytes (every wire element
    distinct from the cache's own values) into a sentinel cache."""
    w = synth.make_workload(3)
    lay = dense_layout(w)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    t0, t1 = w.prompt_ranges()
    cache = G.dev_const(lay.storage_bytes(), SENTINEL)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    rep_h, replica = filled_pair(n, 0xBEEF)
    dv.dv_stream_in(cs, 0, 0, L, t0, t1, replica, n, stream())
    exp = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, exp, 0, L, t0, t1, rep_h)
    torch.cuda.synchronize()
    G.assert_same_bytes(cache, exp, "BLOOM cache restored from a generated replica")


def test_llama_paged_gather_scatter_and_tail_increments(oracle_lib):
    """Paged gather through table A; scatter into a sentinel pool through the
    freshly permuted table B in pool order (owner-map workspace) and in table
    order; 128 tail-block increments from pool A into pool B."""
    w = synth.make_workload(4)
    L, H, D, B, nb = w.layers, w.heads, w.head_dim, w.batch, w.num_blocks
    bs, mbk = w.block_size, w.max_blocks
    la, lb = paged_layout(w, w.block_table_a), paged_layout(w, w.block_table_b)
    gen_h, pool_a = filled_pair(la.storage_bytes(), w.data_seed)
    pool_b = G.dev_const(lb.storage_bytes(), SENTINEL)
    pool_t = G.dev_const(lb.storage_bytes(), SENTINEL)
    bta, btb = G.to_dev(w.block_table_a), G.to_dev(w.block_table_b)
    ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_a], block_size=bs, num_blocks=nb,
                  max_blocks=mbk, block_tables=[bta])
    owners = G.dev_const(nb * 4, 0x7E)
    cb = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_b], block_size=bs, num_blocks=nb,
                  max_blocks=mbk, block_tables=[btb], block_owners=[owners])
    ct = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_t], block_size=bs, num_blocks=nb,
                  max_blocks=mbk, block_tables=[btb])
    t0, t1 = w.prompt_ranges()
    n = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, n, stream())
    dv.dv_stream_in(cb, 0, 0, L, t0, t1, wire, n, stream())  # pool order
    dv.dv_stream_in(ct, 0, 0, L, t0, t1, wire, n, stream())  # table order
    say(f"paged: gather + both scatters of {n} B enqueued")
    exp_wire = OP.pack(oracle_lib, la, gen_h, 0, L, t0, t1)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, "paged gather")
    assert (G.host(owners).view(np.int32) ==
            G.owner_map_expected(w.block_table_b, nb, bs, t0, t1)).all()
    exp_b = np.full(lb.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lb, exp_b, 0, L, t0, t1, exp_wire)
    del exp_wire
    G.assert_same_bytes(pool_b, exp_b, "paged scatter, pool order")
    G.assert_same_bytes(pool_t, exp_b, "paged scatter, table order")
    del pool_t, ct
    say("paged: gather and both scatters equal the oracle")
    incs, exp_incs, inc_n = increments_both_sides(oracle_lib, la, lb, gen_h, exp_b, w,
                                                  ca, cb, L)
    assert inc_n == 2621440
    torch.cuda.synchronize()
    G.assert_same_bytes(incs, exp_incs, "128 tail-block increments")
    G.assert_same_bytes(pool_b, exp_b, "pool B after the scatter and 128 increments")
    del incs, exp_incs, exp_b
    # pool A gathered over [0, len + 128): the prompt and every tail block
    full = (t1 + w.steps).astype(np.int32)
    m = dv.dv_packed_bytes(ca, 0, L, t0, full)
    ga = torch.empty(m, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(ca, 0, 0, L, t0, full, ga, m, stream())
    exp_ga = OP.pack(oracle_lib, la, gen_h, 0, L, t0, full)
    torch.cuda.synchronize()
    G.assert_same_bytes(ga, exp_ga, "paged gather of [0, len + 128)")


def multi_token_case(oracle_lib, w, K):
    L, H, D, B = w.layers, w.heads, w.head_dim, w.batch
    p = w.step_positions(0).astype(np.int32)
    t0, t1 = p, (p + K).astype(np.int32)
    if w.paged:
        lay = paged_layout(w, w.block_table_a)
        gen_h, src = filled_pair(lay.storage_bytes(), w.data_seed)
        bta = G.to_dev(w.block_table_a)
        recv = G.dev_const(lay.storage_bytes(), SENTINEL)
        kw = dict(block_size=w.block_size, num_blocks=w.num_blocks, max_blocks=w.max_blocks,
                  block_tables=[bta])
        cs = dv.Cache(dv.DV_PAGED, L, H, D, B, [src], **kw)
        cr = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], **kw)
    else:
        lay = dense_layout(w)
        gen_h, src = filled_pair(lay.storage_bytes(), w.data_seed)
        recv = G.dev_const(lay.storage_bytes(), SENTINEL)
        cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [src], max_seq=w.max_seq)
        cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=w.max_seq)
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    assert dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, n, stream()) == n
    dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, n, stream())
    exp_wire = OP.pack(oracle_lib, lay, gen_h, 0, L, t0, t1)
    del gen_h
    exp_recv = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, exp_recv, 0, L, t0, t1, exp_wire)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, f"{w.name} K={K} stream-out")
    G.assert_same_bytes(recv, exp_recv, f"{w.name} K={K} receiver")
    return n


@pytest.mark.parametrize("K", [2, 4, 8, 16])
@pytest.mark.parametrize("idx", [1, 4])
def test_multi_token_steps(oracle_lib, idx, K):
    """Decode steps that each add K tokens per sequence (speculative decoding
    accepting several tokens, or replication batched over K steps) on the
    OPT-13B stage and the LLaMA-2-70B paged pool.  They go through the
    short-run kernel: one unit per lane below 2^19 units a launch (OPT-13B
    K = 2, 4; LLaMA K = 2), two units per lane from there on."""
    w = synth.make_workload(idx)
    n = multi_token_case(oracle_lib, w, K)
    units = n // 16
    assert (units >= 1 << 19) == ((idx, K) not in ((1, 2), (1, 4), (4, 2)))
    torch.cuda.empty_cache()


def short_run_launch_units(kind, L, H, du, nt):
    """Units of each launch the library makes for these token counts: one
    launch per group of 64 sequences over all (layer, K|V) slabs; a split-key
    cache makes two per group (keys, values), each over L slabs."""
    per_slab = [int(np.sum(nt[g:g + 64])) * H * du for g in range(0, len(nt), 64)]
    return [u * (L if kind == "ksplit" else 2 * L) for u in per_slab]


@pytest.mark.parametrize("kind", ["dense", "paged", "ksplit"])
@pytest.mark.parametrize("size", ["below", "above", "two-groups"])
def test_short_runs_random_shapes_across_unroll_threshold(oracle_lib, kind, size):
    """The short-run kernel on random shapes whose launches fall on either
    side of 2^19 units (one unit per lane below, two from there on), with
    ragged runs of 0-16 tokens, sentinel receivers and, for "two-groups",
    more than 64 sequences (two launch groups): stream-out and stream-in
    against the oracle."""
    r = np.random.default_rng(9100 + 10 * ["below", "above", "two-groups"].index(size)
                              + ["dense", "paged", "ksplit"].index(kind))
    L, H, B = {"below": (1, 8, 37), "above": (4, 48, 64), "two-groups": (3, 48, 100)}[size]
    D = int(r.choice([64, 128, 256]))
    E = 2
    du = D * E // 16
    kmax = min(16, 256 // du)  # every run within the short-run bound
    t0 = r.integers(0, 40, size=B).astype(np.int32)
    nt = r.integers(0, kmax + 1, size=B)
    nt[int(r.integers(0, B))] = kmax  # at least one run of the longest length
    t1 = (t0 + nt).astype(np.int32)
    units = short_run_launch_units(kind, L, H, du, nt)
    assert (units[0] >= 1 << 19) == (size != "below"), units
    cap = 40 + kmax
    if kind == "paged":
        bs = int(r.choice([4, 16]))
        maxb = (cap + bs - 1) // bs
        bt, nb = synth.make_paged_tables(int(r.integers(0, 1000)), [cap] * B, bs, maxb)
        lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                            num_blocks=nb, block_table=bt)
        kw = dict(block_size=bs, num_blocks=nb, max_blocks=maxb, block_tables=[G.to_dev(bt)])
        dk = dv.DV_PAGED
    else:
        lay = oracle.Layout(oracle.KSPLIT if kind == "ksplit" else oracle.DENSE, L, H, D, B,
                            seq_cap=cap, elem_bytes=E)
        kw = dict(max_seq=cap)
        dk = dv.DV_DENSE_KSPLIT if kind == "ksplit" else dv.DV_DENSE
    gen_h, src = filled_pair(lay.storage_bytes(), 500 + int(r.integers(0, 1000)))
    recv = G.dev_const(lay.storage_bytes(), SENTINEL)
    cs = dv.Cache(dk, L, H, D, B, [src], **kw)
    cr = dv.Cache(dk, L, H, D, B, [recv], **kw)
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, n, stream())
    dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, n, stream())
    exp_wire = OP.pack(oracle_lib, lay, gen_h, 0, L, t0, t1)
    exp_recv = np.full(lay.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(oracle_lib, lay, exp_recv, 0, L, t0, t1, exp_wire)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, f"{kind} short runs stream-out")
    G.assert_same_bytes(recv, exp_recv, f"{kind} short runs receiver")
    say(f"{kind} {size}: L{L} H{H} D{D} B{B}, launch units {units}")

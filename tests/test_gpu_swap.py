"""Microbatch swapping between device slots and pinned host mirrors."""
import zlib

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2403_01876_amd import dv, swap_model  # noqa: E402
from tests import gpu_util as G  # noqa: E402
from oracle import par as OP  # noqa: E402


def pinned(nbytes: int, byte: int) -> torch.Tensor:
    t = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    t.fill_(byte)
    return t


@pytest.mark.parametrize("seed", range(10))
def test_swap_out_in_matches_oracle(oracle_lib, seed):
    r = np.random.default_rng(500 + seed)
    L, H, B = int(r.integers(1, 4)), int(r.integers(1, 6)), int(r.integers(1, 9))
    D, E = int(r.choice([64, 128])), 2
    S_dev = int(r.integers(8, 300))
    S_host = int(r.integers(S_dev // 2, S_dev + 50))
    cap = min(S_dev, S_host)
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_dev, elem_bytes=E)
    hl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_host, elem_bytes=E)
    slot_h = synth.fill_bytes(dl.storage_bytes(), seed)
    slot = G.to_dev(slot_h)
    host = pinned(hl.storage_bytes(), 0x77)
    d = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot], max_seq=S_dev)
    h = dv.Cache(dv.DV_DENSE, L, H, D, B, [host.data_ptr()], max_seq=S_host,
                 mem=dv.DV_MEM_HOST_PINNED)
    if seed % 2 == 0:  # uniform ranges: one 2-D copy
        a = int(r.integers(0, cap))
        t0 = np.full(B, a, np.int32)
        t1 = np.full(B, int(r.integers(a, cap + 1)), np.int32)
    else:
        t0 = r.integers(0, cap // 2 + 1, size=B).astype(np.int32)
        t1 = np.minimum(t0 + r.integers(0, cap, size=B), cap).astype(np.int32)
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    side = torch.cuda.Stream()
    dv.dv_swap_out(d, 0, h, 0, l0, l1, t0, t1, side)
    side.synchronize()
    exp_host = np.full(hl.storage_bytes(), 0x77, np.uint8)
    oracle_lib.copy_ranges(dl, slot_h, hl, exp_host, l0, l1, t0, t1)
    assert host.numpy().tobytes() == exp_host.tobytes()
    # swap back into a sentinel slot
    slot2 = G.dev_const(dl.storage_bytes(), 0xA5)
    d2 = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot2], max_seq=S_dev)
    dv.dv_swap_in(h, 0, d2, 0, l0, l1, t0, t1, side)
    side.synchronize()
    exp_slot = np.full(dl.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.copy_ranges(hl, exp_host, dl, exp_slot, l0, l1, t0, t1)
    assert G.host(slot2).tobytes() == exp_slot.tobytes()


@pytest.mark.parametrize("E", [1, 4])
def test_swap_kernel_engine_many_sequences_other_element_sizes(oracle_lib, E):
    """The copy-kernel engine with 100 sequences (two launch groups), 1- and
    4-byte elements and a layer sub-range, both directions."""
    L, H, B = 3, 2, 100
    D = 64 if E == 4 else 128  # 256 or 128 bytes per token
    S_dev, S_host = 40, 33
    r = np.random.default_rng(600 + E)
    t0 = r.integers(0, 20, size=B).astype(np.int32)
    t1 = np.minimum(t0 + r.integers(0, 14, size=B), S_host).astype(np.int32)
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_dev, elem_bytes=E)
    hl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_host, elem_bytes=E)
    slot_h = synth.fill_bytes(dl.storage_bytes(), 31 + E)
    slot = G.to_dev(slot_h)
    host = pinned(hl.storage_bytes(), 0x77)
    d = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot], max_seq=S_dev, elem_bytes=E)
    h = dv.Cache(dv.DV_DENSE, L, H, D, B, [host.data_ptr()], max_seq=S_host, elem_bytes=E,
                 mem=dv.DV_MEM_HOST_PINNED)
    side = torch.cuda.Stream()
    dv.dv_swap_out(d, 0, h, 0, 1, 3, t0, t1, side)
    side.synchronize()
    exp_host = np.full(hl.storage_bytes(), 0x77, np.uint8)
    oracle_lib.copy_ranges(dl, slot_h, hl, exp_host, 1, 3, t0, t1)
    assert host.numpy().tobytes() == exp_host.tobytes()
    host_h = synth.fill_bytes(hl.storage_bytes(), 41 + E)
    host.copy_(torch.from_numpy(host_h))
    slot2 = G.dev_const(dl.storage_bytes(), 0xA5)
    d2 = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot2], max_seq=S_dev, elem_bytes=E)
    dv.dv_swap_in(h, 0, d2, 0, 1, 3, t0, t1, side)
    side.synchronize()
    exp_slot = np.full(dl.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.copy_ranges(hl, host_h, dl, exp_slot, 1, 3, t0, t1)
    assert G.host(slot2).tobytes() == exp_slot.tobytes()


@pytest.mark.parametrize("case", ["delta-uniform", "delta-ragged", "wide-uniform",
                                  "wide-ragged", "mixed"])
def test_swap_engines_match_oracle(oracle_lib, case):
    """Both engines: narrow rows (copy kernel) and rows of 64 KB or more (DMA)."""
    L, H, D, B, E = 2, 3, 128, 5, 2
    S_dev, S_host = 600, 520
    # a fixed seed per case (str hashes change from process to process)
    r = np.random.default_rng(zlib.crc32(case.encode()))
    if case == "delta-uniform":
        t0 = np.full(B, 300, np.int32)
        t1 = t0 + 1
    elif case == "delta-ragged":
        t0 = r.integers(0, 519, size=B).astype(np.int32)
        t1 = t0 + 1
        t1[2] = t0[2]  # an inactive sequence
    elif case == "wide-uniform":
        t0 = np.zeros(B, np.int32)
        t1 = np.full(B, 500, np.int32)  # 128000-byte rows
    elif case == "wide-ragged":
        t0 = r.integers(0, 100, size=B).astype(np.int32)
        t1 = (t0 + 256 + r.integers(0, 160, size=B)).astype(np.int32)
    else:  # one wide row makes the whole call DMA; others narrow or empty
        t0 = np.array([0, 5, 7, 0, 100], np.int32)
        t1 = np.array([400, 6, 7, 3, 101], np.int32)
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_dev, elem_bytes=E)
    hl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_host, elem_bytes=E)
    slot_h = synth.fill_bytes(dl.storage_bytes(), 3)
    slot = G.to_dev(slot_h)
    host = pinned(hl.storage_bytes(), 0x77)
    d = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot], max_seq=S_dev)
    h = dv.Cache(dv.DV_DENSE, L, H, D, B, [host.data_ptr()], max_seq=S_host,
                 mem=dv.DV_MEM_HOST_PINNED)
    side = torch.cuda.Stream()
    dv.dv_swap_out(d, 0, h, 0, 0, L, t0, t1, side)
    side.synchronize()
    exp_host = np.full(hl.storage_bytes(), 0x77, np.uint8)
    oracle_lib.copy_ranges(dl, slot_h, hl, exp_host, 0, L, t0, t1)
    assert host.numpy().tobytes() == exp_host.tobytes()
    # swap a different host content back in
    host_h = synth.fill_bytes(hl.storage_bytes(), 4)
    host.copy_(torch.from_numpy(host_h))
    slot2 = G.dev_const(dl.storage_bytes(), 0xA5)
    d2 = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot2], max_seq=S_dev)
    dv.dv_swap_in(h, 0, d2, 0, 0, L, t0, t1, side)
    side.synchronize()
    exp_slot = np.full(dl.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.copy_ranges(hl, host_h, dl, exp_slot, 0, L, t0, t1)
    assert G.host(slot2).tobytes() == exp_slot.tobytes()


@pytest.mark.parametrize("engine", ["kernel", "dma"])
def test_swaps_replay_from_a_graph(oracle_lib, engine):
    """Swap-out then swap-in captured once and replayed three times, with the
    slot and the mirror rewritten between replays: narrow rows (one-token
    updates, the copy kernel) and whole prompts (2-D copies on the DMA
    engines).  Every replay moves the oracle's bytes."""
    L, H, D, B, S = 2, 3, 64, 4, 96
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    if engine == "kernel":
        t0 = np.array([5, 17, 0, 40], np.int32)
        t1 = t0 + 1
    else:  # the DMA engines take rows of 64 KB or more: 1 KB tokens, runs of 64-77
        D, S = 512, 80
        dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
        t0 = np.array([0, 3, 0, 10], np.int32)
        t1 = np.array([70, 80, 64, 75], np.int32)
    slot = G.dev_const(dl.storage_bytes(), 0)
    back = G.dev_const(dl.storage_bytes(), 0)
    host = pinned(dl.storage_bytes(), 0)
    d = dv.Cache(dv.DV_DENSE, L, H, D, B, [slot], max_seq=S)
    d2 = dv.Cache(dv.DV_DENSE, L, H, D, B, [back], max_seq=S)
    h = dv.Cache(dv.DV_DENSE, L, H, D, B, [host.data_ptr()], max_seq=S,
                 mem=dv.DV_MEM_HOST_PINNED)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            cur = torch.cuda.current_stream()
            dv.dv_swap_out(d, 0, h, 0, 0, L, t0, t1, cur)
            dv.dv_swap_in(h, 0, d2, 0, 0, L, t0, t1, cur)
    torch.cuda.synchronize()
    for rep in range(3):
        slot_h = synth.fill_bytes(dl.storage_bytes(), 70 + rep)
        slot.copy_(torch.from_numpy(slot_h))
        host.fill_(0x40 + rep)
        back.fill_(0x90 + rep)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        exp_host = np.full(dl.storage_bytes(), 0x40 + rep, np.uint8)
        oracle_lib.copy_ranges(dl, slot_h, dl, exp_host, 0, L, t0, t1)
        assert host.numpy().tobytes() == exp_host.tobytes(), rep
        exp_back = np.full(dl.storage_bytes(), 0x90 + rep, np.uint8)
        oracle_lib.copy_ranges(dl, exp_host, dl, exp_back, 0, L, t0, t1)
        assert G.host(back).tobytes() == exp_back.tobytes(), rep


@pytest.mark.timeout(900)
def test_opt66b_round_robin_swapping(oracle_lib):
    """Four microbatches through two device slots, two rounds.

    Before microbatch x's step its whole cache has been prefetched into its
    slot; the step writes one token per layer (emulated by streaming in a
    generated increment) and packs that increment on the compute stream;
    after the step only the step's token is swapped out, while the next
    microbatch is swapped in on another stream.  At the end every host
    mirror equals the oracle's over every byte: the generator's prompt cache
    copied to the mirror's layout, then each of the microbatch's step tokens
    unpacked at its position.
    """
    w = synth.make_workload(2)
    L, H, D, B, S, E = w.layers, w.heads, w.head_dim, w.batch, w.max_seq, w.elem_bytes
    M = w.microbatches
    S_host = 1024
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    hl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_host, elem_bytes=E)
    seeds = [synth.derived_seed(w.seed, 0x100 + x) for x in range(M)]
    slots = [G.dev_const(dl.storage_bytes(), 0) for _ in range(w.device_slots)]
    hosts = [pinned(hl.storage_bytes(), 0) for _ in range(M)]
    ds = dv.Cache(dv.DV_DENSE, L, H, D, B, slots, max_seq=S)
    hh = dv.Cache(dv.DV_DENSE, L, H, D, B, [t.data_ptr() for t in hosts], max_seq=S_host,
                  mem=dv.DV_MEM_HOST_PINNED)
    prompt = np.full(B, 1000, np.int32)
    lens = [prompt.copy() for _ in range(M)]
    zero = np.zeros(B, np.int32)
    compute, s_out, s_in = torch.cuda.current_stream(), torch.cuda.Stream(), torch.cuda.Stream()

    # the prompt caches start on the host: each generated in slot 0, swapped out
    for x in range(M):
        synth.device_fill(slots[0].data_ptr(), dl.storage_bytes(), seeds[x],
                          stream=compute.cuda_stream)
        dv.dv_swap_out(ds, 0, hh, x, 0, L, zero, lens[x], compute)
        compute.synchronize()

    inc_n = L * 2 * B * H * D * E
    assert inc_n == 4718592
    inc = torch.empty(inc_n, dtype=torch.uint8, device=G.DEV)
    tok = torch.empty(inc_n, dtype=torch.uint8, device=G.DEV)
    swapped_in = [torch.cuda.Event() for _ in range(w.device_slots)]
    slot_free = [torch.cuda.Event() for _ in range(w.device_slots)]
    for e in slot_free:
        e.record(compute)
    # prefetch microbatch 0 into slot 0
    s_in.wait_event(slot_free[0])
    dv.dv_swap_in(hh, 0, ds, 0, 0, L, zero, lens[0], s_in)
    swapped_in[0].record(s_in)
    steps = 2 * M
    written = [[] for _ in range(M)]  # (position, token seed) of each step, per microbatch
    for k in range(steps):
        x, slot, nxt = k % M, k % 2, (k + 1) % 2
        # prefetch the next microbatch into the other slot once its previous
        # occupant's update has reached the host
        if k + 1 < steps:
            s_in.wait_event(slot_free[nxt])
            xn = (k + 1) % M
            dv.dv_swap_in(hh, xn, ds, nxt, 0, L, zero, lens[xn], s_in)
            swapped_in[nxt].record(s_in)
        # the step itself on the compute stream
        compute.wait_event(swapped_in[slot])
        pos = lens[x]
        tok_seed = synth.derived_seed(w.seed, 0x200 + k)
        synth.device_fill(tok.data_ptr(), inc_n, tok_seed, stream=compute.cuda_stream)
        dv.dv_stream_in(ds, slot, 0, L, pos, pos + 1, tok, inc_n, compute)
        dv.dv_stream_out_token(ds, slot, 0, L, pos, inc, inc_n, compute)
        done = torch.cuda.Event()
        done.record(compute)
        # swap out only the step's update, then free the slot
        s_out.wait_event(done)
        dv.dv_swap_out(ds, slot, hh, x, 0, L, pos, pos + 1, s_out)
        slot_free[slot].record(s_out)
        written[x].append((pos.copy(), tok_seed))
        lens[x] = pos + 1
        # the packed increment is the generated token just written
        compute.synchronize()
        G.assert_same_bytes(inc, synth.fill_bytes(inc_n, tok_seed), f"increment of step {k}")
    torch.cuda.synchronize()
    del slots, inc, tok
    torch.cuda.empty_cache()
    for x in range(M):
        exp = np.zeros(hl.storage_bytes(), np.uint8)
        gen = synth.fill_bytes_parallel(dl.storage_bytes(), seeds[x])
        OP.copy_ranges(oracle_lib, dl, gen, hl, exp, 0, L, zero, prompt)
        del gen
        for pos, tok_seed in written[x]:
            OP.unpack(oracle_lib, hl, exp, 0, L, pos, pos + 1,
                      synth.fill_bytes(inc_n, tok_seed))
        got = hosts[x].numpy()
        if not np.array_equal(got, exp):
            bad = np.flatnonzero(got != exp)
            raise AssertionError(f"mirror {x}: {bad.size} bytes differ, first at {bad[0]}")
        del exp


@pytest.mark.parametrize("compute_kind", ["null", "own", "alternating"])
def test_swapper_round_robin(oracle_lib, compute_kind):
    """The scheduler runs the protocol of the previous test by itself: five
    microbatches (an odd count, so slots alternate differently each round)
    through two slots, three rounds, ragged per-sequence positions.  The
    compute stream is the legacy null stream (pooled side streams), a stream
    of its own (side streams on hardware queues of their own), or the two in
    turn, step by step (the scheduler switching forms mid-protocol)."""
    L, H, D, B, E = 3, 4, 128, 3, 2
    S, S_host, M = 64, 48, 5
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    hl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S_host, elem_bytes=E)
    slots = [G.dev_const(dl.storage_bytes(), 0) for _ in range(2)]
    refs = [G.dev_filled(dl.storage_bytes(), 70 + x) for x in range(M)]
    hosts = [pinned(hl.storage_bytes(), 0) for _ in range(M)]
    ds = dv.Cache(dv.DV_DENSE, L, H, D, B, slots, max_seq=S)
    dr = dv.Cache(dv.DV_DENSE, L, H, D, B, refs, max_seq=S)
    hh = dv.Cache(dv.DV_DENSE, L, H, D, B, [t.data_ptr() for t in hosts], max_seq=S_host,
                  mem=dv.DV_MEM_HOST_PINNED)
    zero = np.zeros(B, np.int32)
    lens = [np.array([20, 25, 30], np.int32) + x for x in range(M)]
    null = torch.cuda.default_stream()
    own = torch.cuda.Stream()
    own.wait_stream(torch.cuda.current_stream())
    compute = null
    for x in range(M):
        dv.dv_swap_out(dr, x, hh, x, 0, L, zero, lens[x], compute)
    compute.synchronize()
    sw = dv.Swapper(ds, hh)
    n = dv.dv_packed_bytes(ds, 0, L, lens[0], lens[0] + 1)
    tok = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    inc = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    # the paper's order (swap_schedule): while x runs, prefetch x + 1; x's
    # update leaves after its step, while x + 1 runs
    sched = list(swap_model.swap_schedule(M, 3))
    sw.prefetch(sched[0][0], lens[sched[0][0]])
    for k, (x, xn, _) in enumerate(sched):
        compute = {"null": null, "own": own}.get(compute_kind, null if k % 2 == 0 else own)
        if xn is not None:
            sw.prefetch(xn, lens[xn])
        slot = sw.begin_step(x, compute)
        pos = lens[x]
        synth.device_fill(tok.data_ptr(), n, 900 + k, stream=compute.cuda_stream)
        dv.dv_stream_in(ds, slot, 0, L, pos, pos + 1, tok, n, compute)
        dv.dv_stream_in(dr, x, 0, L, pos, pos + 1, tok, n, compute)
        dv.dv_stream_out_token(ds, slot, 0, L, pos, inc, n, compute)
        sw.end_step(x, pos, pos + 1, compute)
        lens[x] = pos + 1
        compute.synchronize()
        assert torch.equal(inc, tok), k
    sw.sync()
    # every host mirror equals its reference on [0, len) (oracle copy map)
    for x in range(M):
        exp = np.zeros(hl.storage_bytes(), np.uint8)
        oracle_lib.copy_ranges(dl, G.host(refs[x]), hl, exp, 0, L, zero, lens[x])
        m = np.zeros(hl.storage_bytes(), np.uint8)
        oracle_lib.copy_ranges(hl, hosts[x].numpy(), hl, m, 0, L, zero, lens[x])
        assert m.tobytes() == exp.tobytes(), x
    sw.close()


def test_swapper_refuses_refill_before_step_end():
    L, H, D, B = 1, 1, 64, 1
    slots = [G.dev_const(L * 2 * B * H * 16 * D * 2, 0) for _ in range(2)]
    hosts = [pinned(L * 2 * B * H * 16 * D * 2, 0) for _ in range(3)]
    ds = dv.Cache(dv.DV_DENSE, L, H, D, B, slots, max_seq=16)
    hh = dv.Cache(dv.DV_DENSE, L, H, D, B, [t.data_ptr() for t in hosts], max_seq=16,
                  mem=dv.DV_MEM_HOST_PINNED)
    sw = dv.Swapper(ds, hh)
    lens = np.array([4], np.int32)
    assert sw.prefetch(0, lens) == dv.DV_OK
    assert sw.prefetch(1, lens) == dv.DV_OK
    # both slots hold microbatches whose steps have not ended
    assert sw.prefetch(2, lens, check=False) == dv.DV_ERR_INVALID
    with pytest.raises(dv.DvError):
        sw.begin_step(2)  # not prefetched
    # begin_step and end_step refuse a stream under graph capture, and the
    # capture goes on
    scratch = G.dev_const(64, 0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            scratch.add_(1)
            cap = torch.cuda.current_stream()
            with pytest.raises(dv.DvError) as e:
                sw.begin_step(0, stream=cap)
            assert e.value.status == dv.DV_ERR_INVALID
            assert sw.end_step(0, [3], [4], stream=cap, check=False) == dv.DV_ERR_INVALID
    g.replay()
    torch.cuda.synchronize()
    assert int(scratch[0]) == 1
    assert sw.begin_step(0) == 0
    sw.end_step(0, [3], [4])
    assert sw.prefetch(2, lens) == dv.DV_OK  # slot 0 is free again
    sw.sync()
    sw.close()


def test_swapper_rejects_bad_ranges_without_changing_state():
    """A prefetch or end_step whose ranges do not fit the slots or the host
    mirrors is refused before anything is enqueued, and the scheduler's
    state is as before: the same calls with good ranges then work."""
    L, H, D, B = 1, 1, 64, 2
    S, S_host = 16, 8
    slots = [G.dev_const(L * 2 * B * H * S * D * 2, 0) for _ in range(2)]
    hosts = [pinned(L * 2 * B * H * S_host * D * 2, 0) for _ in range(3)]
    ds = dv.Cache(dv.DV_DENSE, L, H, D, B, slots, max_seq=S)
    hh = dv.Cache(dv.DV_DENSE, L, H, D, B, [t.data_ptr() for t in hosts], max_seq=S_host,
                  mem=dv.DV_MEM_HOST_PINNED)
    sw = dv.Swapper(ds, hh)
    good = np.array([4, 5], np.int32)
    for bad in (np.array([9, 1], np.int32), np.array([-1, 1], np.int32)):
        assert sw.prefetch(0, bad, check=False) == dv.DV_ERR_RANGE  # 9 > host capacity 8
    assert sw.prefetch(0, good) == dv.DV_OK
    assert sw.prefetch(1, good) == dv.DV_OK
    assert sw.begin_step(0) == 0
    assert sw.end_step(0, [4, 5], [9, 6], check=False) == dv.DV_ERR_RANGE
    assert sw.end_step(0, [5, 4], [4, 5], check=False) == dv.DV_ERR_RANGE  # t1 < t0
    # the refused end_step did not free slot 0
    assert sw.prefetch(2, good, check=False) == dv.DV_ERR_INVALID
    assert sw.end_step(0, [4, 5], [5, 6]) == dv.DV_OK
    assert sw.prefetch(2, good) == dv.DV_OK
    sw.sync()
    sw.close()

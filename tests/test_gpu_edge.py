"""Edge cases of the HIP path, each compared with the CPU oracle byte for byte."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2403_01876_amd import dv  # noqa: E402
from tests import gpu_util as G  # noqa: E402


def stream():
    return torch.cuda.current_stream()


def dense_roundtrip(orc, L, H, D, B, S, E, l0, l1, t0, t1, seed=0, kind=dv.DV_DENSE):
    okind = {dv.DV_DENSE: oracle.DENSE, dv.DV_DENSE_KSPLIT: oracle.KSPLIT}[kind]
    lay = oracle.Layout(okind, L, H, D, B, seq_cap=S, elem_bytes=E)
    host = synth.fill_bytes(lay.storage_bytes(), seed)
    cache = G.to_dev(host)
    c = dv.Cache(kind, L, H, D, B, [cache], max_seq=S, elem_bytes=E)
    exp = orc.pack(lay, host, l0, l1, t0, t1)
    wire = G.dev_const(exp.nbytes + 32, 0x5C)
    n = dv.dv_stream_out_prompt(c, 0, l0, l1, t0, t1, wire, exp.nbytes, stream())
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    r = dv.Cache(kind, L, H, D, B, [recv], max_seq=S, elem_bytes=E)
    if n:
        dv.dv_stream_in(r, 0, l0, l1, t0, t1, wire, n, stream())
    torch.cuda.synchronize()
    w = G.host(wire)
    assert n == exp.nbytes and w[:n].tobytes() == exp.tobytes() and (w[n:] == 0x5C).all()
    exp_recv = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    orc.unpack(lay, exp_recv, l0, l1, t0, t1, exp)
    assert G.host(recv)[: lay.storage_bytes()].tobytes() == exp_recv.tobytes()


def test_one_unit_per_token(oracle_lib):
    """head_dim * elem_bytes == 16: one 16-byte unit per token."""
    B = 5
    t0 = np.array([0, 3, 0, 7, 2], np.int32)
    t1 = np.array([9, 3, 1, 31, 30], np.int32)
    dense_roundtrip(oracle_lib, 2, 3, 8, B, 31, 2, 0, 2, t0, t1)
    dense_roundtrip(oracle_lib, 2, 3, 8, B, 31, 2, 0, 2, t0, t1, kind=dv.DV_DENSE_KSPLIT)
    dense_roundtrip(oracle_lib, 1, 2, 16, B, 31, 1, 0, 1, t0, t1)


def test_many_heads_and_long_runs(oracle_lib):
    """128 heads; runs of 3000 tokens span many tiles with a ragged tail."""
    B = 2
    t0 = np.array([0, 5], np.int32)
    t1 = np.array([3000, 2999], np.int32)
    dense_roundtrip(oracle_lib, 1, 128, 128, B, 3001, 2, 0, 1, t0, t1)


def test_two_hundred_sequences_with_an_empty_group(oracle_lib):
    """Sequences 64..127 stream nothing: their launch is skipped, later groups
    still land at the right wire offsets."""
    B = 200
    r = np.random.default_rng(3)
    t0 = r.integers(0, 20, size=B).astype(np.int32)
    t1 = (t0 + r.integers(0, 20, size=B)).astype(np.int32)
    t1[64:128] = t0[64:128]
    dense_roundtrip(oracle_lib, 2, 2, 64, B, 40, 2, 0, 2, t0, t1)
    # and single tokens with the same empty group
    p = r.integers(0, 40, size=B).astype(np.int32)
    e = (p + 1).astype(np.int32)
    e[64:128] = p[64:128]
    dense_roundtrip(oracle_lib, 2, 2, 64, B, 40, 2, 1, 2, p, e)


def test_ranges_at_capacity_end(oracle_lib):
    S = 77
    t0 = np.array([76, 0, 77, 40], np.int32)
    t1 = np.array([77, 77, 77, 77], np.int32)
    dense_roundtrip(oracle_lib, 3, 4, 64, 4, S, 2, 1, 3, t0, t1)
    dense_roundtrip(oracle_lib, 3, 4, 64, 4, S, 2, 1, 3, t0, t1, kind=dv.DV_DENSE_KSPLIT)


def test_head_dim_512(oracle_lib):
    """64 units per token (split key is limited to 32 and rejects it)."""
    t0 = np.array([0, 1], np.int32)
    t1 = np.array([33, 2], np.int32)
    dense_roundtrip(oracle_lib, 1, 2, 512, 2, 40, 2, 0, 1, t0, t1)
    cache, dst = G.dev_const(1 << 20, 0), G.dev_const(1 << 20, 0)
    lay = dv.Cache(dv.DV_DENSE_KSPLIT, 1, 2, 512, 2, [cache], max_seq=40)
    rc, _ = dv.dv_stream_out_prompt(lay, 0, 0, 1, t0, t1, dst, 1 << 20, check=False)
    assert rc == dv.DV_ERR_UNSUPPORTED


@pytest.mark.parametrize("bs", [1, 64])
def test_paged_block_sizes(oracle_lib, bs):
    L, H, D, B, E = 2, 3, 128, 4, 2
    lens = [130, 0, 1, 64]
    maxb = max((n + bs - 1) // bs for n in lens) + 1
    bt, nb = synth.make_paged_tables(bs, lens, bs, maxb)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    host = synth.fill_bytes(lay.storage_bytes(), bs)
    pool = G.to_dev(host)
    btd = G.to_dev(bt)
    c = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=bs, num_blocks=nb,
                 max_blocks=maxb, block_tables=[btd])
    t0 = np.array([3, 0, 0, 10], np.int32)
    t1 = np.array([130, 0, 1, 64], np.int32)
    exp = oracle_lib.pack(lay, host, 0, L, t0, t1)
    wire = G.dev_const(exp.nbytes, 0)
    dv.dv_stream_out_prompt(c, 0, 0, L, t0, t1, wire, exp.nbytes, stream())
    torch.cuda.synchronize()
    assert G.host(wire).tobytes() == exp.tobytes()


def test_paged_unmapped_entries_are_skipped(oracle_lib):
    """Table entries outside [0, num_blocks) inside the ranges: the kernels
    skip those tokens -- their wire bytes stay unwritten on pack and the pool
    is untouched on unpack -- and every other token is exact.

    Expected values come from the oracle over a pool with one extra block per
    (layer, K|V) slab that the invalid entries are pointed at: filled with the
    wire sentinel for pack, and dropped again after unpack.  Three range
    shapes reach the three paged paths: runs longer than 4 KB per head (tiled
    kernel, pool order with the workspace), single tokens, and runs of 4 KB
    (short-run kernel)."""
    L, H, D, B, E, bs = 2, 2, 512, 3, 2, 4
    bt = np.array([[0, 1, 2], [3, -1, 4], [5, 99, 6]], np.int32)
    nb = 7
    blk = H * bs * D * E  # bytes per block per slab
    bad = (bt < 0) | (bt >= nb)
    bt_x = np.where(bad, nb, bt).astype(np.int32)
    ext = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                        num_blocks=nb + 1, block_table=bt_x)

    def with_extra(pool_real, fill):
        x = pool_real.reshape(L * 2, nb * blk)
        pad = np.full((L * 2, blk), fill, np.uint8)
        return np.concatenate([x, pad], axis=1).reshape(-1)

    def drop_extra(pool_ext):
        return pool_ext.reshape(L * 2, (nb + 1) * blk)[:, : nb * blk].reshape(-1)

    host = synth.fill_bytes(L * 2 * nb * blk, 11)
    pool = G.to_dev(host)
    btd = G.to_dev(bt)
    c = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=bs, num_blocks=nb, max_blocks=3,
                 block_tables=[btd])
    for case in ("long", "single", "short"):
        single = case == "single"
        if single:
            t0 = np.array([5, 5, 5], np.int32)  # logical block 1 of each sequence
            t1 = t0 + 1
        elif case == "long":
            t0 = np.array([0, 1, 2], np.int32)
            t1 = np.array([12, 9, 11], np.int32)
        else:  # 4 tokens x 64 units = 4 KB per head, across the unmapped entries
            t0 = np.array([2, 3, 4], np.int32)
            t1 = t0 + 4
        n = dv.dv_packed_bytes(c, 0, L, t0, t1)
        wire = G.dev_const(n, 0x5C)
        if single:
            dv.dv_stream_out_token(c, 0, 0, L, t0, wire, n, stream())
        else:
            dv.dv_stream_out_prompt(c, 0, 0, L, t0, t1, wire, n, stream())
        torch.cuda.synchronize()
        exp = oracle_lib.pack(ext, with_extra(host, 0x5C), 0, L, t0, t1)
        assert G.host(wire).tobytes() == exp.tobytes()
        # unpack a generated wire into a sentinel pool
        wh = synth.fill_bytes(n, 21)
        recv = G.dev_const(L * 2 * nb * blk, 0xA5)
        rc = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], block_size=bs, num_blocks=nb,
                      max_blocks=3, block_tables=[btd])
        dv.dv_stream_in(rc, 0, 0, L, t0, t1, G.to_dev(wh), n, stream())
        torch.cuda.synchronize()
        exp_pool = with_extra(np.full(L * 2 * nb * blk, 0xA5, np.uint8), 0xA5)
        oracle_lib.unpack(ext, exp_pool, 0, L, t0, t1, wh)
        assert G.host(recv).tobytes() == drop_extra(exp_pool).tobytes()
        # the same scatter in pool order (an owner-map workspace given)
        ws = G.dev_const(nb * 4, 0x7E)
        recv2 = G.dev_const(L * 2 * nb * blk, 0xA5)
        rc2 = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv2], block_size=bs, num_blocks=nb,
                       max_blocks=3, block_tables=[btd], block_owners=[ws])
        dv.dv_stream_in(rc2, 0, 0, L, t0, t1, G.to_dev(wh), n, stream())
        torch.cuda.synchronize()
        assert G.host(recv2).tobytes() == drop_extra(exp_pool).tobytes()
        if case == "long":  # 9 logical blocks streamed, 7 pool blocks: pool order taken
            assert G.host(ws).view(np.int32).tolist() == [0, 1, 2, 3, 5, 6, 8]
        else:  # token and short-run kernels scatter in stream order
            assert (G.host(ws) == 0x7E).all()


def test_graph_replay_paged_pool_order_and_split_key(oracle_lib):
    """Captured: a paged gather, a pool-order scatter (owner map rebuilt by
    kernels inside the graph), tail-block increments, and a split-key
    round trip.  Each replay starts from a sentinel receiver and a garbage
    owner workspace and must give the oracle's result."""
    L, H, D, B, bs = 2, 3, 128, 5, 16
    lens = [40, 17, 64, 1, 33]
    steps = 4
    maxb = max((n + steps + bs - 1) // bs for n in lens) + 1
    bt, nb = synth.make_paged_tables(77, [n + steps for n in lens], bs, maxb)
    valid = bt >= 0
    bt_b = bt.copy()
    bt_b[valid] = np.random.default_rng(3).permutation(bt[valid])
    la = oracle.Layout(oracle.PAGED, L, H, D, B, block_size=bs, num_blocks=nb, block_table=bt)
    lb = oracle.Layout(oracle.PAGED, L, H, D, B, block_size=bs, num_blocks=nb, block_table=bt_b)
    host = synth.fill_bytes(la.storage_bytes(), 78)
    pool_a = G.to_dev(host)
    pool_b = G.dev_const(lb.storage_bytes(), 0)
    owners = G.dev_const(nb * 4, 0x7E)
    bta, btb = G.to_dev(bt), G.to_dev(bt_b)
    ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_a], block_size=bs, num_blocks=nb,
                  max_blocks=maxb, block_tables=[bta])
    cb = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_b], block_size=bs, num_blocks=nb,
                  max_blocks=maxb, block_tables=[btb], block_owners=[owners])
    t0 = np.zeros(B, np.int32)
    t1 = np.array(lens, np.int32)
    P = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = G.dev_const(P, 0)
    I = dv.dv_packed_bytes(ca, 0, L, t1, t1 + 1)
    inc = G.dev_const(I, 0)
    S = 96
    kl = oracle.Layout(oracle.KSPLIT, L, H, D, B, seq_cap=S)
    khost = synth.fill_bytes(kl.storage_bytes(), 79)
    ks = G.to_dev(khost)
    kr = G.dev_const(kl.storage_bytes(), 0)
    ck = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [ks], max_seq=S)
    ckr = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [kr], max_seq=S)
    kt1 = np.minimum(t1, S).astype(np.int32)
    KP = dv.dv_packed_bytes(ck, 0, L, t0, kt1)
    kwire = G.dev_const(KP, 0)

    def step(st):
        dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, P, st)
        dv.dv_stream_in(cb, 0, 0, L, t0, t1, wire, P, st)
        for i in range(steps):
            p = t1 + i
            dv.dv_stream_out_token(ca, 0, 0, L, p, inc, I, st)
            dv.dv_stream_in(cb, 0, 0, L, p, p + 1, inc, I, st)
        dv.dv_stream_out_prompt(ck, 0, 0, L, t0, kt1, kwire, KP, st)
        dv.dv_stream_in(ckr, 0, 0, L, t0, kt1, kwire, KP, st)

    exp_b = np.full(lb.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lb, exp_b, 0, L, t0, t1, oracle_lib.pack(la, host, 0, L, t0, t1))
    for i in range(steps):
        p = t1 + i
        oracle_lib.unpack(lb, exp_b, 0, L, p, p + 1, oracle_lib.pack(la, host, 0, L, p, p + 1))
    exp_k = np.full(kl.storage_bytes(), 0x3C, np.uint8)
    oracle_lib.unpack(kl, exp_k, 0, L, t0, kt1, oracle_lib.pack(kl, khost, 0, L, t0, kt1))

    side = torch.cuda.Stream()
    side.wait_stream(stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(4):
        pool_b.fill_(0xA5)
        owners.fill_(0x40 + rep)
        kr.fill_(0x3C)
        wire.fill_(rep)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert G.host(pool_b).tobytes() == exp_b.tobytes(), rep
        assert G.host(kr).tobytes() == exp_k.tobytes(), rep
        assert (G.host(owners).view(np.int32) == G.owner_map_expected(bt_b, nb, bs, t0, t1)).all()


def test_graph_replay_matches_eager(oracle_lib):
    """A captured step replayed several times, with eager work and syncs in
    between, gives the eager result every time."""
    w = synth.make_workload(0)
    L, H, D, B, S = w.layers, w.heads, w.head_dim, w.batch, w.max_seq
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    host = synth.fill_bytes(lay.storage_bytes(), 5)
    src = G.to_dev(host)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [src], max_seq=S)
    recv = G.dev_const(lay.storage_bytes(), 0)
    cr = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S)
    t0, t1 = w.prompt_ranges()
    P = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = G.dev_const(P, 0)
    inc = G.dev_const(4096, 0)

    def step(st):
        dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, P, st)
        dv.dv_stream_in(cr, 0, 0, L, t0, t1, wire, P, st)
        for i in range(w.steps):
            p = w.step_positions(i)
            dv.dv_stream_out_token(cs, 0, 0, L, p, inc, 4096, st)
            dv.dv_stream_in(cr, 0, 0, L, p, p + 1, inc, 4096, st)

    step(stream())
    torch.cuda.synchronize()
    eager_recv, eager_wire, eager_inc = recv.clone(), wire.clone(), inc.clone()
    side = torch.cuda.Stream()
    side.wait_stream(stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(4):
        recv.fill_(rep + 1)
        wire.fill_(0x11 * rep)
        inc.fill_(0x22)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        exp = np.full(lay.storage_bytes(), rep + 1, np.uint8)
        oracle_lib.unpack(lay, exp, 0, L, t0, t1, oracle_lib.pack(lay, host, 0, L, t0, t1))
        for i in range(w.steps):
            p = w.step_positions(i)
            oracle_lib.unpack(lay, exp, 0, L, p, p + 1,
                              oracle_lib.pack(lay, host, 0, L, p, p + 1))
        assert G.host(recv).tobytes() == exp.tobytes(), rep
        assert torch.equal(wire, eager_wire) and torch.equal(inc, eager_inc), rep
    del eager_recv


@pytest.mark.parametrize("kind", ["dense", "paged"])
def test_graph_replay_short_runs(oracle_lib, kind):
    """Multi-token steps (3 tokens per sequence, the short-run kernel)
    captured once and replayed four times, with eager work and syncs in
    between: every replay leaves each step's wire and the receiver equal to
    the oracle's."""
    r = np.random.default_rng(11)
    L, H, D, B, K, steps = 2, 4, 64, 5, 3, 5
    if kind == "dense":
        S = 64
        lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
        extents = dict(max_seq=S)
        kd = dv.DV_DENSE
    else:
        bs, maxb = 16, 4
        bt, nb = synth.make_paged_tables(9, [maxb * bs] * B, bs, maxb)
        lay = oracle.Layout(oracle.PAGED, L, H, D, B, block_size=bs, num_blocks=nb,
                            block_table=bt)
        extents = dict(block_size=bs, num_blocks=nb, max_blocks=maxb,
                       block_tables=[G.to_dev(bt)])
        kd = dv.DV_PAGED
    host = synth.fill_bytes(lay.storage_bytes(), 13)
    cs = dv.Cache(kd, L, H, D, B, [G.to_dev(host)], **extents)
    recv = G.dev_const(lay.storage_bytes(), 0)
    cr = dv.Cache(kd, L, H, D, B, [recv], **extents)
    p0 = r.integers(0, 40, size=B).astype(np.int32)
    rng = [(p0 + K * i, p0 + K * (i + 1)) for i in range(steps)]
    n = dv.dv_packed_bytes(cs, 0, L, *rng[0])
    wires = [G.dev_const(n, 0) for _ in range(steps)]

    def step(st):
        for (a, e), wb in zip(rng, wires):
            dv.dv_stream_out_prompt(cs, 0, 0, L, a, e, wb, n, st)
            dv.dv_stream_in(cr, 0, 0, L, a, e, wb, n, st)

    side = torch.cuda.Stream()
    side.wait_stream(stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    exp_wires = [oracle_lib.pack(lay, host, 0, L, a, e) for a, e in rng]
    for rep in range(4):
        recv.fill_(rep + 7)
        for wb in wires:
            wb.fill_(0x33)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        exp = np.full(lay.storage_bytes(), rep + 7, np.uint8)
        for (a, e), ew in zip(rng, exp_wires):
            oracle_lib.unpack(lay, exp, 0, L, a, e, ew)
        for wb, ew in zip(wires, exp_wires):
            assert G.host(wb).tobytes() == ew.tobytes(), rep
        assert G.host(recv).tobytes() == exp.tobytes(), rep


@pytest.mark.parametrize("seed", range(4))
def test_per_region_baseline_matches_buffered(oracle_lib, seed):
    """The comparison baseline (one copy per contiguous region) yields the same
    bytes as the buffered path, to device memory and to pinned host memory."""
    from paper_2403_01876_amd import baseline
    r = np.random.default_rng(40 + seed)
    L, H, D, B, S = 2, int(r.integers(1, 5)), 128, int(r.integers(1, 7)), 90
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    host = synth.fill_bytes(lay.storage_bytes(), seed)
    cache = G.to_dev(host)
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t0 = r.integers(0, 40, size=B).astype(np.int32)
    t1 = (t0 + r.integers(0, 50, size=B)).astype(np.int32)
    if seed == 3:
        t1 = (t0 + 1).astype(np.int32)  # single tokens
    exp = oracle_lib.pack(lay, host, 0, L, t0, t1)
    n = exp.nbytes
    d_buf = G.dev_const(max(n, 16), 0)
    h_buf = torch.zeros(max(n, 16), dtype=torch.uint8, pin_memory=True)
    calls = baseline.per_region_copy(c, 0, 0, L, t0, t1, d_buf, n, stream())
    assert calls == 2 * L * H * int((t1 > t0).sum())
    baseline.per_region_copy(c, 0, 0, L, t0, t1, h_buf.data_ptr(), n, stream())
    torch.cuda.synchronize()
    assert G.host(d_buf)[:n].tobytes() == exp.tobytes()
    assert h_buf.numpy()[:n].tobytes() == exp.tobytes()


@pytest.mark.parametrize("units", [1, 255, 512, 513, 8 * 512 + 7, 5 * 8 * 512 + 300])
def test_plain_copy_baseline(units):
    """The copy ceiling the benchmark sets the pack kernel against copies
    exactly its bytes: sizes below one 8 KB tile, at and past tile edges, and
    tile counts that do not divide by the 8 XCDs (the workgroup renumbering
    must stay a bijection); the bytes past the end stay untouched."""
    from paper_2403_01876_amd import baseline
    n = units * 16
    src = G.to_dev(synth.fill_bytes(n, units))
    dst = G.dev_const(n + 64, 0x5C)
    baseline.plain_copy(dst, src, n, stream())
    torch.cuda.synchronize()
    assert torch.equal(dst[:n], src)
    assert bool((dst[n:] == 0x5C).all())


@pytest.mark.parametrize("scatter", [False, True])
@pytest.mark.parametrize("block_kb", [8, 32])
def test_block_copy_baseline(scatter, block_kb):
    """The paged kernels' ceiling copies whole blocks in a permutation's
    order: checked against numpy's block permutation; an out-of-range order
    entry skips its block (its destination keeps the sentinel)."""
    from paper_2403_01876_amd import baseline
    nb, bb = 37, block_kb * 1024
    src_h = synth.fill_bytes(nb * bb, block_kb + 100 * scatter)
    order = np.random.default_rng(block_kb).permutation(nb).astype(np.int32)
    order[5] = nb  # skipped
    dst = G.dev_const(nb * bb, 0x5C)
    baseline.block_copy(dst, G.to_dev(src_h), G.to_dev(order), nb, bb, scatter, stream())
    torch.cuda.synchronize()
    s = src_h.reshape(nb, bb)
    exp = np.full((nb, bb), 0x5C, np.uint8)
    ok = order < nb
    if scatter:
        exp[order[ok]] = s[ok]
    else:
        exp[ok] = s[order[ok]]
    assert G.host(dst).tobytes() == exp.tobytes()


def test_binding_follows_torchs_current_stream(oracle_lib):
    """stream=None means torch's current stream: under torch.cuda.stream(s)
    the pack runs after the work already queued on s (here a long spin and
    then the fill of its source), never on a stream unordered with it."""
    L, H, D, B, S = 2, 4, 128, 3, 64
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    host = synth.fill_bytes(lay.storage_bytes(), 91)
    cache = G.dev_const(lay.storage_bytes(), 0)
    staged = G.to_dev(host)
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t0 = np.zeros(B, np.int32)
    t1 = np.array([64, 10, 33], np.int32)
    n = dv.dv_packed_bytes(c, 0, L, t0, t1)
    wire = G.dev_const(n, 0)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        torch.cuda._sleep(50_000_000)  # tens of ms on the side stream
        cache.copy_(staged)
        dv.dv_stream_out_prompt(c, 0, 0, L, t0, t1, wire, n)  # stream=None
    torch.cuda.synchronize()
    assert G.host(wire).tobytes() == oracle_lib.pack(lay, host, 0, L, t0, t1).tobytes()

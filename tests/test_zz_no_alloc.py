"""dv_stream_in_noalloc, the allocation-free stream-in, through the C ABI.

It must write exactly what dv_stream_in with a caller-owned owner-map
workspace writes.  Two calls in a row on one GPU share the library's static
owner map: the first is the LLaMA-2-70B paged scatter at full size (pool
order, as the benchmark times it), the second a smaller pool whose map
covers fewer blocks, so stale entries of the first call lie past its end.
Both results are compared over every byte with the workspace call's and with
the oracle's; the caller's workspace passed in the noalloc call's descriptor
is left untouched.  Graph replays of the call are checked too, including a
process whose very first call is made under capture.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("no GPU", allow_module_level=True)

from paper_2403_01876_amd import dv  # noqa: E402
from tests import gpu_util as G  # noqa: E402
from oracle import par as OP  # noqa: E402

SENTINEL = 0xA5


def scatter_both_ways(orc, L, H, D, B, bs, nb, maxb, bta, btb, lens, seed):
    """Gather through table A; scatter the buffer into sentinel pools through
    table B with dv_stream_in (workspace) and dv_stream_in_noalloc; compare."""
    E = 2
    la = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                       block_table=bta)
    lb = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                       block_table=btb)
    gen_h = synth.fill_bytes_parallel(la.storage_bytes(), seed)
    pool_a = G.dev_filled(la.storage_bytes(), seed)
    ta, tb = G.to_dev(bta), G.to_dev(btb)
    kw = dict(block_size=bs, num_blocks=nb, max_blocks=maxb)
    ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_a], block_tables=[ta], **kw)
    t0 = np.zeros(B, np.int32)
    t1 = np.asarray(lens, np.int32)
    n = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    assert dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, n) == n
    pool_w = G.dev_const(lb.storage_bytes(), SENTINEL)
    pool_n = G.dev_const(lb.storage_bytes(), SENTINEL)
    ws = G.dev_const(nb * 4, 0x7E)
    untouched = G.dev_const(nb * 4, 0x3C)
    cw = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_w], block_tables=[tb], block_owners=[ws], **kw)
    cn = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_n], block_tables=[tb],
                  block_owners=[untouched], **kw)
    assert dv.dv_stream_in(cw, 0, 0, L, t0, t1, wire, n) == dv.DV_OK
    assert dv.dv_stream_in_noalloc(cn, 0, 0, L, t0, t1, wire, n) == dv.DV_OK
    exp_wire = OP.pack(orc, la, gen_h, 0, L, t0, t1)
    exp_pool = np.full(lb.storage_bytes(), SENTINEL, np.uint8)
    OP.unpack(orc, lb, exp_pool, 0, L, t0, t1, exp_wire)
    torch.cuda.synchronize()
    G.assert_same_bytes(wire, exp_wire, "gather")
    assert torch.equal(pool_n, pool_w), "noalloc scatter differs from the workspace scatter"
    G.assert_same_bytes(pool_n, exp_pool, "noalloc scatter")
    # the workspace call built its map in the caller's workspace; the
    # noalloc call left the workspace in its descriptor alone
    assert (G.host(ws).view(np.int32) == G.owner_map_expected(btb, nb, bs, t0, t1)).all()
    assert bool((untouched == 0x3C).all())
    return nb


def test_noalloc_scatter_matches_workspace_scatter_twice():
    orc = oracle.get()
    w = synth.make_workload(4)
    assert w.num_blocks <= dv.NOALLOC_MAX_BLOCKS
    nb1 = scatter_both_ways(orc, w.layers, w.heads, w.head_dim, w.batch, w.block_size,
                            w.num_blocks, w.max_blocks, w.block_table_a, w.block_table_b,
                            w.lens, w.data_seed)
    torch.cuda.empty_cache()
    # second call, smaller: 6 sequences, 2 layers, block size 8
    lens = [40, 7, 64, 1, 33, 90]
    bs, maxb = 8, 12
    bta, nb = synth.make_paged_tables(71, lens, bs, maxb)
    btb, nb2 = synth.make_paged_tables(72, lens, bs, maxb)
    assert nb == nb2 and nb < nb1
    scatter_both_ways(orc, 2, 4, 128, 6, bs, nb, maxb, bta, btb, lens, 73)


def test_noalloc_dense_receiver_is_stream_in():
    """A dense receiver uses no buffer: the same bytes as dv_stream_in."""
    L, H, D, B, S = 2, 3, 64, 4, 40
    t0 = np.array([0, 5, 9, 0], np.int32)
    t1 = np.array([30, 5, 40, 1], np.int32)
    src = G.dev_filled(L * 2 * B * H * S * D * 2, 81)
    cs = dv.Cache(dv.DV_DENSE, L, H, D, B, [src], max_seq=S)
    n = dv.dv_packed_bytes(cs, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(cs, 0, 0, L, t0, t1, wire, n)
    a = G.dev_const(src.numel(), SENTINEL)
    b = G.dev_const(src.numel(), SENTINEL)
    dv.dv_stream_in(dv.Cache(dv.DV_DENSE, L, H, D, B, [a], max_seq=S), 0, 0, L, t0, t1, wire, n)
    dv.dv_stream_in_noalloc(dv.Cache(dv.DV_DENSE, L, H, D, B, [b], max_seq=S), 0, 0, L, t0, t1,
                            wire, n)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("B", [6, 100])
def test_noalloc_scatter_replayed_from_a_graph(B):
    """The callers it is for capture it: a gather and a dv_stream_in_noalloc
    scatter captured into a HIP graph and replayed three times, with eager
    work and a fresh sentinel pool between replays; every replay against the
    oracle.  100 sequences take the pool-order launch over the whole call
    (more than 64 sequences), 6 the scan-based one."""
    orc = oracle.get()
    L, H, D, E, bs = 2, 4, 128, 2, 16
    r = np.random.default_rng(B)
    lens = [int(x) for x in r.integers(20, 120, size=B)]
    maxb = max((n + bs - 1) // bs for n in lens)
    bta, nb = synth.make_paged_tables(B + 1, lens, bs, maxb)
    btb, nb2 = synth.make_paged_tables(B + 2, lens, bs, maxb)
    assert nb == nb2
    la = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                       block_table=bta)
    lb = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                       block_table=btb)
    gen_h = synth.fill_bytes(la.storage_bytes(), 300 + B)
    pool_a = G.to_dev(gen_h)
    pool_b = G.dev_const(lb.storage_bytes(), SENTINEL)
    kw = dict(block_size=bs, num_blocks=nb, max_blocks=maxb)
    ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_a], block_tables=[G.to_dev(bta)], **kw)
    cb = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_b], block_tables=[G.to_dev(btb)], **kw)
    t0 = np.zeros(B, np.int32)
    t1 = np.array(lens, np.int32)
    n = dv.dv_packed_bytes(ca, 0, L, t0, t1)
    wire = G.dev_const(n, 0)
    exp_wire = orc.pack(la, gen_h, 0, L, t0, t1)
    exp_pool = np.full(lb.storage_bytes(), SENTINEL, np.uint8)
    orc.unpack(lb, exp_pool, 0, L, t0, t1, exp_wire)
    # one eager call first: the library looks its buffer's address up once
    assert dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, n) == n
    assert dv.dv_stream_in_noalloc(cb, 0, 0, L, t0, t1, wire, n) == dv.DV_OK
    torch.cuda.synchronize()
    G.assert_same_bytes(pool_b, exp_pool, "eager noalloc scatter")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            cur = torch.cuda.current_stream()
            dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, n, cur)
            dv.dv_stream_in_noalloc(cb, 0, 0, L, t0, t1, wire, n, cur)
    torch.cuda.synchronize()
    for rep in range(3):
        pool_b.fill_(SENTINEL)
        wire.fill_(rep + 1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        G.assert_same_bytes(wire, exp_wire, f"replay {rep}: gather")
        G.assert_same_bytes(pool_b, exp_pool, f"replay {rep}: noalloc scatter")
        # eager work between replays on the library's shared map: a smaller
        # stream-in (still over five ninths of the blocks, so in pool order)
        # that rebuilds the map for other ranges
        part = (t1 * 9 // 10).astype(np.int32)
        m = dv.dv_packed_bytes(cb, 0, L, t0, part)
        scratch = G.dev_const(lb.storage_bytes(), 0)
        cs = dv.Cache(dv.DV_PAGED, L, H, D, B, [scratch], block_tables=[G.to_dev(btb)], **kw)
        dv.dv_stream_in_noalloc(cs, 0, 0, L, t0, part, wire[:m], m)
        torch.cuda.synchronize()
        del scratch


def test_noalloc_first_call_under_graph_capture():
    """In a process of its own, the first allocation-free call is made under
    graph capture, so the library's one-time lookup of its buffer's address
    happens while the stream is being captured; the replays still scatter
    the oracle's bytes (tests/noalloc_capture_first.py)."""
    import os
    import subprocess
    import sys

    script = os.path.join(os.path.dirname(os.path.abspath(__file__)), "noalloc_capture_first.py")
    r = subprocess.run([sys.executable, "-u", script], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), \
        r.stdout[-2000:] + r.stderr[-4000:]

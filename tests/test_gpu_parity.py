"""HIP path vs the CPU oracle, byte for byte, on randomized small shapes.

Shapes span several tiles per run (runs longer than one workgroup's 2048
16-byte units), ragged tails, empty ranges, sub-ranges of layers, more than
64 sequences (several launches), 1/2/4-byte elements and head_dim 16..256.
Every call goes through the C ABI (paper_2403_01876_amd.dv).
"""
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


def rand_dense_shape(r, big_batch=False):
    L = int(r.integers(1, 4))
    H = int(r.integers(1, 7))
    E = int(r.choice([2, 2, 2, 1, 4]))
    D = int(r.choice([64, 128, 128, 256, 96])) if E == 2 else int(r.choice([16, 32, 64])) // E * 4
    D = max(16 // E, D - D % (16 // E))
    B = int(r.integers(65, 140)) if big_batch else int(r.integers(1, 12))
    S = int(r.integers(1, 400))
    return L, H, D, B, S, E


def rand_ranges(r, B, cap, p_empty=0.15):
    t0 = np.zeros(B, np.int32)
    t1 = np.zeros(B, np.int32)
    for b in range(B):
        if r.random() < 0.5:
            a, c = 0, int(r.integers(0, cap + 1))  # prompt-like prefix
        else:
            a, c = sorted(int(v) for v in r.integers(0, cap + 1, size=2))
        if r.random() < p_empty:
            c = a
        t0[b], t1[b] = a, c
    return t0, t1


def stream():
    return torch.cuda.current_stream()


def run_pack(cache_desc, l0, l1, t0, t1, nbytes):
    wire = G.dev_const(nbytes + 64, 0x5C)
    n = dv.dv_stream_out_prompt(cache_desc, 0, l0, l1, t0, t1, wire, nbytes, stream())
    assert n == nbytes
    torch.cuda.synchronize()
    w = G.host(wire)
    assert (w[nbytes:] == 0x5C).all(), "wrote past the stream"
    return w[:nbytes]


@pytest.mark.parametrize("seed", range(24))
def test_dense_pack_unpack(oracle_lib, seed):
    r = np.random.default_rng(seed)
    L, H, D, B, S, E = rand_dense_shape(r, big_batch=(seed % 6 == 5))
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    host_cache = synth.fill_bytes(lay.storage_bytes(), seed)
    cache = G.to_dev(host_cache)
    desc = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S, elem_bytes=E)
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    t0, t1 = rand_ranges(r, B, S)
    exp = oracle_lib.pack(lay, host_cache, l0, l1, t0, t1)
    got = run_pack(desc, l0, l1, t0, t1, exp.nbytes)
    assert got.tobytes() == exp.tobytes()
    # unpack a different wire into a sentinel receiver
    wire_h = synth.fill_bytes(exp.nbytes, seed + 1000)
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    rdesc = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S, elem_bytes=E)
    if exp.nbytes:
        dv.dv_stream_in(rdesc, 0, l0, l1, t0, t1, G.to_dev(wire_h), exp.nbytes, stream())
    torch.cuda.synchronize()
    exp_recv = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp_recv, l0, l1, t0, t1, wire_h)
    assert G.host(recv)[: lay.storage_bytes()].tobytes() == exp_recv.tobytes()


@pytest.mark.parametrize("seed", range(12))
def test_token_increments(oracle_lib, seed):
    """Single-token ranges (the decode-step path), some sequences inactive."""
    r = np.random.default_rng(100 + seed)
    L, H, D, B, S, E = rand_dense_shape(r, big_batch=(seed % 4 == 3))
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    host_cache = synth.fill_bytes(lay.storage_bytes(), seed)
    cache = G.to_dev(host_cache)
    desc = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S, elem_bytes=E)
    pos = r.integers(0, S, size=B).astype(np.int32)
    pos[r.random(B) < 0.25] = -1
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    a = np.maximum(pos, 0)
    e = np.where(pos >= 0, pos + 1, 0).astype(np.int32)
    exp = oracle_lib.pack(lay, host_cache, l0, l1, a, e)
    wire = G.dev_const(exp.nbytes + 64, 0x5C)
    n = dv.dv_stream_out_token(desc, 0, l0, l1, pos, wire, exp.nbytes, stream())
    assert n == exp.nbytes
    torch.cuda.synchronize()
    w = G.host(wire)
    assert w[:n].tobytes() == exp.tobytes() and (w[n:] == 0x5C).all()
    # stream the increment into a sentinel receiver
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    rdesc = dv.Cache(dv.DV_DENSE, L, H, D, B, [recv], max_seq=S, elem_bytes=E)
    if n:
        dv.dv_stream_in(rdesc, 0, l0, l1, a, e, wire, n, stream())
    torch.cuda.synchronize()
    exp_recv = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp_recv, l0, l1, a, e, exp)
    assert G.host(recv)[: lay.storage_bytes()].tobytes() == exp_recv.tobytes()


def paged_setup(r, seed, big_batch=False):
    L = int(r.integers(1, 4))
    H = int(r.integers(1, 12))
    E = int(r.choice([2, 2, 1, 4]))
    D = int(r.choice([64, 128, 256])) // E * 2  # 128, 256 or 512 bytes per token
    B = int(r.integers(65, 100)) if big_batch else int(r.integers(1, 10))
    bs = int(r.choice([1, 4, 16, 16, 32]))
    lens = [int(r.integers(0, 300)) for _ in range(B)]
    maxb = max(1, max((n + bs - 1) // bs for n in lens)) + int(r.integers(0, 3))
    bt, nb = synth.make_paged_tables(seed, lens, bs, maxb)
    nb = max(nb, 1)
    return L, H, D, B, E, bs, lens, maxb, bt, nb


@pytest.mark.parametrize("seed", range(16))
def test_paged_gather_scatter(oracle_lib, seed):
    r = np.random.default_rng(200 + seed)
    L, H, D, B, E, bs, lens, maxb, bt, nb = paged_setup(r, seed, big_batch=(seed % 8 == 7))
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    host_pool = synth.fill_bytes(lay.storage_bytes(), seed)
    pool = G.to_dev(host_pool)
    bt_dev = G.to_dev(bt)
    desc = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], elem_bytes=E, block_size=bs,
                    num_blocks=nb, max_blocks=maxb, block_tables=[bt_dev])
    t0 = np.zeros(B, np.int32)
    t1 = np.zeros(B, np.int32)
    for b in range(B):
        a, c = sorted(int(v) for v in r.integers(0, lens[b] + 1, size=2))
        if r.random() < 0.5:
            a = 0
        t0[b], t1[b] = a, c
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    exp = oracle_lib.pack(lay, host_pool, l0, l1, t0, t1)
    got = run_pack(desc, l0, l1, t0, t1, exp.nbytes)
    assert got.tobytes() == exp.tobytes()
    # scatter into a fresh permutation of the same pool size, sentinel-filled
    bt_b = bt.copy()
    valid = bt >= 0
    bt_b[valid] = r.permutation(bt[valid])
    lay_b = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                          block_table=bt_b)
    recv = G.dev_const(lay_b.storage_bytes(), 0xA5)
    bt_b_dev = G.to_dev(bt_b)
    rdesc = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], elem_bytes=E, block_size=bs,
                     num_blocks=nb, max_blocks=maxb, block_tables=[bt_b_dev])
    if exp.nbytes:
        dv.dv_stream_in(rdesc, 0, l0, l1, t0, t1, G.to_dev(exp), exp.nbytes, stream())
    torch.cuda.synchronize()
    exp_recv = np.full(lay_b.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay_b, exp_recv, l0, l1, t0, t1, exp)
    assert G.host(recv)[: lay_b.storage_bytes()].tobytes() == exp_recv.tobytes()


@pytest.mark.parametrize("seed", range(12))
def test_paged_scatter_pool_order(oracle_lib, seed):
    """Scatter with an owner-map workspace: the pool equals the oracle's
    unpack whichever order the library picks; when the header's conditions
    hold (some run longer than 256 16-byte units, at most 256 sequences, at
    least five ninths of the pool's blocks written) the workspace holds the owner
    map afterwards, otherwise it is untouched.  A second call with another
    table reuses the stale workspace."""
    r = np.random.default_rng(900 + seed)
    L, H, D, B, E, bs, lens, maxb, bt, nb = paged_setup(r, seed, big_batch=(seed % 6 == 5))
    kind = seed % 3
    t0 = np.zeros(B, np.int32)
    t1 = np.array(lens, np.int32)
    for b in range(B):
        if kind == 1:
            a, c = sorted(int(v) for v in r.integers(0, lens[b] + 1, size=2))
            t0[b], t1[b] = a, c
        elif kind == 2 and r.random() < 0.2:
            t1[b] = 0
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    ws = G.dev_const(nb * 4 + 64, 0x7E)
    valid = bt >= 0
    for call in range(2):
        bt_b = bt.copy()
        bt_b[valid] = r.permutation(bt[valid])
        lay_b = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                              num_blocks=nb, block_table=bt_b)
        n = dv.dv_packed_bytes(dv.Cache(dv.DV_PAGED, L, H, D, B, [0], elem_bytes=E,
                                        block_size=bs, num_blocks=nb, max_blocks=maxb,
                                        block_tables=[0]), l0, l1, t0, t1)
        wire_h = synth.fill_bytes(n, 1000 + seed * 2 + call)
        recv = G.dev_const(lay_b.storage_bytes(), 0xA5)
        bt_b_dev = G.to_dev(bt_b)
        rdesc = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], elem_bytes=E, block_size=bs,
                         num_blocks=nb, max_blocks=maxb, block_tables=[bt_b_dev],
                         block_owners=[ws])
        wire = G.to_dev(wire_h)
        if n:
            dv.dv_stream_in(rdesc, 0, l0, l1, t0, t1, wire, n, stream())
        torch.cuda.synchronize()
        exp_recv = np.full(lay_b.storage_bytes(), 0xA5, np.uint8)
        oracle_lib.unpack(lay_b, exp_recv, l0, l1, t0, t1, wire_h)
        assert G.host(recv)[: lay_b.storage_bytes()].tobytes() == exp_recv.tobytes()
        blocks = sum((t1[b] + bs - 1) // bs - t0[b] // bs for b in range(B) if t1[b] > t0[b])
        du = D * E // 16
        # runs of at most 256 units per (sequence, head) take the short-run
        # kernel, which scatters in stream order
        pool_order = (n > 0 and B <= 256 and (t1 - t0).max() > 1 and
                      (t1 - t0).max() * du > 256 and 9 * blocks >= 5 * nb)
        w = G.host(ws)
        assert (w[nb * 4:] == 0x7E).all(), "wrote past the workspace"
        if pool_order:
            assert (w[: nb * 4].view(np.int32) ==
                    G.owner_map_expected(bt_b, nb, bs, t0, t1)).all()
        elif call == 0:
            assert (w[: nb * 4] == 0x7E).all()


@pytest.mark.parametrize("written", [4, 5])
def test_paged_scatter_pool_order_threshold(oracle_lib, written):
    """The five-ninths rule at its boundary: a pool of 9 blocks with an
    owner-map workspace, one sequence streaming 5 blocks (5/9: pool order,
    the workspace holds the table's inverse) or 4 blocks (table order, the
    workspace untouched).  The pool equals the oracle's unpack either way."""
    L, H, D, B, E, bs, nb, maxb = 2, 2, 128, 1, 2, 16, 9, 9
    r = np.random.default_rng(77 + written)
    bt = r.permutation(nb).astype(np.int32).reshape(1, maxb)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    t0 = np.zeros(B, np.int32)
    t1 = np.array([written * bs], np.int32)  # runs of 1024-1280 16-byte units: tiled kernels
    n = oracle_lib.wire_elems(lay, 0, L, t0, t1) * E
    wire_h = synth.fill_bytes(n, 500 + written)
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    ws = G.dev_const(nb * 4, 0x7E)
    c = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], elem_bytes=E, block_size=bs, num_blocks=nb,
                 max_blocks=maxb, block_tables=[G.to_dev(bt)], block_owners=[ws])
    dv.dv_stream_in(c, 0, 0, L, t0, t1, G.to_dev(wire_h), n, stream())
    torch.cuda.synchronize()
    exp = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp, 0, L, t0, t1, wire_h)
    assert G.host(recv).tobytes() == exp.tobytes()
    if 9 * written >= 5 * nb:
        assert (G.host(ws).view(np.int32) == G.owner_map_expected(bt, nb, bs, t0, t1)).all()
    else:
        assert (G.host(ws) == 0x7E).all()


@pytest.mark.parametrize("B", [130, 256, 257])
def test_paged_scatter_pool_order_many_sequences(oracle_lib, B):
    """Pool order over several launch groups: one owner map for the whole
    call (sequence indices past 64 included) and one launch over the pool,
    up to 256 sequences; 257 sequences scatter in table order and leave the
    workspace untouched.  Against the oracle over the whole pool, with
    sequences of every length including empty ones."""
    r = np.random.default_rng(4000 + B)
    L, H, D, E, bs = 2, 3, 128, 2, 16
    lens = [int(x) for x in r.integers(0, 90, size=B)]
    lens[5] = 0
    maxb = max((n + bs - 1) // bs for n in lens) + 1
    bt, nb = synth.make_paged_tables(B, lens, bs, maxb)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    t0 = np.zeros(B, np.int32)
    t1 = np.array(lens, np.int32)
    n = oracle_lib.wire_elems(lay, 0, L, t0, t1) * E
    wire_h = synth.fill_bytes(n, 4100 + B)
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    ws = G.dev_const(nb * 4, 0x7E)
    c = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], elem_bytes=E, block_size=bs, num_blocks=nb,
                 max_blocks=maxb, block_tables=[G.to_dev(bt)], block_owners=[ws])
    dv.dv_stream_in(c, 0, 0, L, t0, t1, G.to_dev(wire_h), n, stream())
    torch.cuda.synchronize()
    exp = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp, 0, L, t0, t1, wire_h)
    assert G.host(recv).tobytes() == exp.tobytes()
    if B <= 256:
        assert (G.host(ws).view(np.int32) == G.owner_map_expected(bt, nb, bs, t0, t1)).all()
    else:
        assert (G.host(ws) == 0x7E).all()


@pytest.mark.parametrize("seed", range(6))
def test_block_claims_count_table_entries(seed):
    """dv_block_claims against a plain count of the table entries over the
    ranges, with duplicated and unmapped entries planted in the table, and
    more than 64 sequences for some seeds."""
    r = np.random.default_rng(1500 + seed)
    L, H, D, B, E, bs, lens, maxb, bt, nb = paged_setup(r, seed, big_batch=(seed % 3 == 2))
    bt = bt.copy()
    valid = np.argwhere(bt >= 0)
    for _ in range(3):  # duplicates
        if len(valid) >= 2:
            a, b = valid[r.integers(0, len(valid), size=2)]
            bt[a[0], a[1]] = bt[b[0], b[1]]
    if len(valid):
        k = valid[r.integers(0, len(valid))]
        bt[k[0], k[1]] = nb + 5  # unmapped: outside the pool
    t0 = np.zeros(B, np.int32)
    t1 = np.zeros(B, np.int32)
    for b in range(B):
        a, c = sorted(int(v) for v in r.integers(0, lens[b] + 1, size=2))
        t0[b], t1[b] = a, c
    exp = np.zeros(nb, np.int64)
    for b in range(B):
        if t1[b] > t0[b]:
            for j in range(t0[b] // bs, (t1[b] - 1) // bs + 1):
                if 0 <= bt[b, j] < nb:
                    exp[bt[b, j]] += 1
    pool = G.dev_const(L * 2 * nb * H * bs * D * E, 0)
    btd = G.to_dev(bt)
    c = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], elem_bytes=E, block_size=bs, num_blocks=nb,
                 max_blocks=maxb, block_tables=[btd])
    counts = G.dev_const(nb * 4 + 64, 0x7E)
    dv.dv_block_claims(c, 0, t0, t1, counts, stream())
    torch.cuda.synchronize()
    got = G.host(counts)
    assert (got[nb * 4:] == 0x7E).all(), "wrote past the counts"
    assert np.array_equal(got[: nb * 4].view(np.int32), exp.astype(np.int32))


@pytest.mark.parametrize("seed", range(8))
def test_paged_token_increments(oracle_lib, seed):
    r = np.random.default_rng(300 + seed)
    L, H, D, B, E, bs, lens, maxb, bt, nb = paged_setup(r, seed)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    host_pool = synth.fill_bytes(lay.storage_bytes(), seed)
    pool = G.to_dev(host_pool)
    bt_dev = G.to_dev(bt)
    desc = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], elem_bytes=E, block_size=bs,
                    num_blocks=nb, max_blocks=maxb, block_tables=[bt_dev])
    pos = np.array([int(r.integers(0, n)) if n > 0 else -1 for n in lens], np.int32)
    a = np.maximum(pos, 0)
    e = np.where(pos >= 0, pos + 1, 0).astype(np.int32)
    exp = oracle_lib.pack(lay, host_pool, 0, L, a, e)
    wire = G.dev_const(exp.nbytes + 64, 0x5C)
    n = dv.dv_stream_out_token(desc, 0, 0, L, pos, wire, exp.nbytes, stream())
    torch.cuda.synchronize()
    assert n == exp.nbytes and G.host(wire)[:n].tobytes() == exp.tobytes()
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    rdesc = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], elem_bytes=E, block_size=bs,
                     num_blocks=nb, max_blocks=maxb, block_tables=[bt_dev])
    if n:
        dv.dv_stream_in(rdesc, 0, 0, L, a, e, wire, n, stream())
    torch.cuda.synchronize()
    exp_recv = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp_recv, 0, L, a, e, exp)
    assert G.host(recv)[: lay.storage_bytes()].tobytes() == exp_recv.tobytes()


@pytest.mark.parametrize("seed", range(24))
def test_ksplit_pack_unpack(oracle_lib, seed):
    r = np.random.default_rng(400 + seed)
    L, H, D, B, S, E = rand_dense_shape(r)
    if 16 % E:
        E = 2
    D = min(D, 256 // max(E // 2, 1))
    D = max(16 // E, D - D % (16 // E))
    lay = oracle.Layout(oracle.KSPLIT, L, H, D, B, seq_cap=S, elem_bytes=E)
    host_cache = synth.fill_bytes(lay.storage_bytes(), seed)
    cache = G.to_dev(host_cache)
    desc = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [cache], max_seq=S, elem_bytes=E)
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    t0, t1 = rand_ranges(r, B, S)
    if seed % 3 == 2:  # single-token ranges take the increment path
        t1 = np.minimum(t0 + 1, S).astype(np.int32)
    exp = oracle_lib.pack(lay, host_cache, l0, l1, t0, t1)
    got = run_pack(desc, l0, l1, t0, t1, exp.nbytes)
    assert got.tobytes() == exp.tobytes()
    wire_h = synth.fill_bytes(exp.nbytes, seed + 5)
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    rdesc = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [recv], max_seq=S, elem_bytes=E)
    if exp.nbytes:
        dv.dv_stream_in(rdesc, 0, l0, l1, t0, t1, G.to_dev(wire_h), exp.nbytes, stream())
    torch.cuda.synchronize()
    exp_recv = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp_recv, l0, l1, t0, t1, wire_h)
    assert G.host(recv)[: lay.storage_bytes()].tobytes() == exp_recv.tobytes()


@pytest.mark.parametrize("D", [8, 32, 64, 128, 192, 256])
def test_ksplit_group_counts(oracle_lib, D):
    """Every count of 16-byte groups per token the split-key kernel takes in
    one or several 4-unit passes (1 .. 32 groups; 16 and more get the padded
    LDS request), with ragged 64-token tiles."""
    r = np.random.default_rng(D)
    L, H, B, S, E = 2, 3, 4, 150, 2
    lay = oracle.Layout(oracle.KSPLIT, L, H, D, B, seq_cap=S, elem_bytes=E)
    host_cache = synth.fill_bytes(lay.storage_bytes(), D + 1)
    cache = G.to_dev(host_cache)  # the descriptor holds its address only
    desc = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [cache], max_seq=S)
    t0 = np.array([0, 5, 63, 0], np.int32)
    t1 = np.array([150, 70, 64, int(r.integers(2, 150))], np.int32)
    exp = oracle_lib.pack(lay, host_cache, 0, L, t0, t1)
    assert run_pack(desc, 0, L, t0, t1, exp.nbytes).tobytes() == exp.tobytes()
    wire_h = synth.fill_bytes(exp.nbytes, D + 2)
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    rdesc = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [recv], max_seq=S)
    wire = G.to_dev(wire_h)
    dv.dv_stream_in(rdesc, 0, 0, L, t0, t1, wire, exp.nbytes, stream())
    torch.cuda.synchronize()
    exp_recv = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    oracle_lib.unpack(lay, exp_recv, 0, L, t0, t1, wire_h)
    assert G.host(recv)[: lay.storage_bytes()].tobytes() == exp_recv.tobytes()


def test_cross_layout_stream(oracle_lib):
    """Dense sender -> paged receiver and split-key receiver, then back."""
    r = np.random.default_rng(7)
    L, H, D, B, S, E = 3, 5, 128, 6, 200, 2
    dl = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    host_cache = synth.fill_bytes(dl.storage_bytes(), 3)
    cache = G.to_dev(host_cache)
    d = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t1 = r.integers(0, S + 1, size=B).astype(np.int32)
    t0 = np.zeros(B, np.int32)
    n = dv.dv_packed_bytes(d, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(d, 0, 0, L, t0, t1, wire, n, stream())
    bs = 16
    bt, nb = synth.make_paged_tables(9, list(t1), bs, (S + bs - 1) // bs)
    pl = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                       block_table=bt)
    pool = G.dev_const(pl.storage_bytes(), 0)
    btd = G.to_dev(bt)
    p = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=bs, num_blocks=nb,
                 max_blocks=bt.shape[1], block_tables=[btd])
    dv.dv_stream_in(p, 0, 0, L, t0, t1, wire, n, stream())
    ks = G.dev_const(dl.storage_bytes(), 0)
    k = dv.Cache(dv.DV_DENSE_KSPLIT, L, H, D, B, [ks], max_seq=S)
    dv.dv_stream_in(k, 0, 0, L, t0, t1, wire, n, stream())
    w2 = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    w3 = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(p, 0, 0, L, t0, t1, w2, n, stream())
    dv.dv_stream_out_prompt(k, 0, 0, L, t0, t1, w3, n, stream())
    torch.cuda.synchronize()
    exp = oracle_lib.pack(dl, host_cache, 0, L, t0, t1)
    for x in (wire, w2, w3):
        assert G.host(x).tobytes() == exp.tobytes()


def test_layer_by_layer_equals_whole(oracle_lib):
    """Streaming one layer per call into consecutive wire chunks equals one call."""
    L, H, D, B, S = 4, 3, 128, 5, 300
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    cache = G.dev_filled(lay.storage_bytes(), 11)
    d = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    t1 = np.array([300, 1, 0, 129, 77], np.int32)
    t0 = np.zeros(B, np.int32)
    n = dv.dv_packed_bytes(d, 0, L, t0, t1)
    whole = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    parts = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(d, 0, 0, L, t0, t1, whole, n, stream())
    off = 0
    for l in range(L):
        k = dv.dv_packed_bytes(d, l, l + 1, t0, t1)
        dv.dv_stream_out_prompt(d, 0, l, l + 1, t0, t1, parts[off:], k, stream())
        off += k
    torch.cuda.synchronize()
    assert off == n and torch.equal(whole, parts)


def test_device_fill_equals_host_fill():
    for nbytes, first in [(16, 0), (4096, 0), (1 << 20, 160), (12345 * 16, 1 << 33)]:
        t = torch.empty(nbytes, dtype=torch.uint8, device=G.DEV)
        synth.device_fill(t.data_ptr(), nbytes, 0xC0FFEE, first_byte=first)
        torch.cuda.synchronize()
        assert G.host(t).tobytes() == synth.fill_bytes(nbytes, 0xC0FFEE, first_byte=first).tobytes()


@pytest.mark.parametrize("seed", range(24))
def test_short_runs(oracle_lib, seed):
    """Ranges of 0 to 20 tokens per sequence -- a decode step that accepts
    several tokens, or replication batched over a few steps -- through the
    short-run kernel (longest run at most 256 16-byte units) and, for some
    seeds, just past that limit through the tiled kernels.  Dense, paged and
    split-key senders and receivers, 1/2/4-byte elements, more than 64
    sequences for some seeds; pack and sentinel-receiver unpack against the
    oracle byte for byte."""
    r = np.random.default_rng(2500 + seed)
    E = int(r.choice([2, 2, 1, 4]))
    du = int(r.choice([1, 2, 8, 16, 32]))
    D = du * 16 // E
    L = int(r.integers(1, 4))
    H = int(r.integers(1, 9))
    B = int(r.integers(65, 80)) if seed % 6 == 5 else int(r.integers(1, 10))
    kinds = [(dv.DV_DENSE, oracle.DENSE), (dv.DV_PAGED, oracle.PAGED),
             (dv.DV_DENSE_KSPLIT, oracle.KSPLIT)]
    kind, okind = kinds[seed % 3]
    rkind, rokind = kinds[(seed // 3) % 3]
    limit = 256 // du  # longest run (tokens) the short-run kernel takes
    nmax = limit + 1 if seed % 4 == 3 else min(20, limit)
    S = max(64, nmax + 8)
    t0 = r.integers(0, S - nmax, size=B).astype(np.int32)
    n = r.integers(0, nmax + 1, size=B).astype(np.int32)
    n[r.random(B) < 0.2] = 0
    if seed % 4 == 3:
        n[int(r.integers(0, B))] = nmax  # one run just past the limit
    t1 = (t0 + n).astype(np.int32)
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))

    def layout(k, ok, sd, fill):
        if k == dv.DV_PAGED:
            bs = int(r.choice([1, 4, 16]))
            maxb = -(-S // bs)
            bt, nb = synth.make_paged_tables(sd, [maxb * bs] * B, bs, maxb)
            lay = oracle.Layout(ok, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                                block_table=bt)
            host = synth.fill_bytes(lay.storage_bytes(), sd) if fill is None else \
                np.full(lay.storage_bytes(), fill, np.uint8)
            dev = G.to_dev(host)
            desc = dv.Cache(k, L, H, D, B, [dev], elem_bytes=E, block_size=bs, num_blocks=nb,
                            max_blocks=maxb, block_tables=[G.to_dev(bt)])
        else:
            lay = oracle.Layout(ok, L, H, D, B, seq_cap=S, elem_bytes=E)
            host = synth.fill_bytes(lay.storage_bytes(), sd) if fill is None else \
                np.full(lay.storage_bytes(), fill, np.uint8)
            dev = G.to_dev(host)
            desc = dv.Cache(k, L, H, D, B, [dev], max_seq=S, elem_bytes=E)
        return lay, host, dev, desc

    lay, host, dev, desc = layout(kind, okind, seed, None)
    exp = oracle_lib.pack(lay, host, l0, l1, t0, t1)
    got = run_pack(desc, l0, l1, t0, t1, exp.nbytes)
    assert got.tobytes() == exp.tobytes()
    rlay, rhost, rdev, rdesc = layout(rkind, rokind, seed + 77, 0xA5)
    if exp.nbytes:
        dv.dv_stream_in(rdesc, 0, l0, l1, t0, t1, G.to_dev(exp), exp.nbytes, stream())
    torch.cuda.synchronize()
    oracle_lib.unpack(rlay, rhost, l0, l1, t0, t1, exp)
    assert G.host(rdev)[: rlay.storage_bytes()].tobytes() == rhost.tobytes()

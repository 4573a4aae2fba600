"""The largest extents the library accepts, on the GPU.

* a dense cache of 68 GiB, so cache addresses pass 2**32 16-byte units;
* the 2**24-token capacity with capacity * head_dim * elem_bytes at its
  2**34-byte limit (32 GiB), for a prompt range and a decode-step token at
  the last position;
* a paged table of 2**20 blocks per sequence (capacity 2**24), gathered and
  scattered in both orders;
* a split-key cache at capacity with the most 16-byte groups per token.

Every wire element is checked against the oracle's source map applied to the
generator (the caches are too large to copy to the host); a filled wire is
streamed back in and every cache element it should land on is checked the
same way, plus neighbours of the ranges that must keep their generated
values.  The paged pool is small and is compared with the oracle in full.
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

GIB = 1 << 30
WIRE_SEED = 77


@pytest.fixture(autouse=True)
def release_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def stream():
    return torch.cuda.current_stream()


def wire_sources(orc, lay, l0, l1, t0, t1):
    nel = orc.wire_elems(lay, l0, l1, t0, t1)
    w = np.arange(nel, dtype=np.int64)
    return w, orc.wire_to_storage(lay, l0, l1, t0, t1, w)


def check_wire(orc, lay, data_seed, wire, l0, l1, t0, t1):
    """Every wire element equals the generated element the oracle maps it to."""
    E = lay.elem_bytes
    w, src = wire_sources(orc, lay, l0, l1, t0, t1)
    assert (src >= 0).all()
    exp = synth.bytes_at(data_seed, src.astype(np.uint64) * np.uint64(E), E).astype(G.NDT[E])
    got = G.host(wire)[: w.size * E].view(G.NDT[E])
    bad = np.flatnonzero(got != exp)
    assert bad.size == 0, f"{bad.size} of {w.size} wire elements differ; first at {bad[0]}"


def check_landed(orc, lay, cache, l0, l1, t0, t1):
    """Every cache element the oracle maps a wire element to holds that wire
    element (the wire was filled from WIRE_SEED)."""
    E = lay.elem_bytes
    w, dst = wire_sources(orc, lay, l0, l1, t0, t1)
    exp = synth.bytes_at(WIRE_SEED, w.astype(np.uint64) * np.uint64(E), E).astype(G.NDT[E])
    got = G.gather(cache, dst, E)
    bad = np.flatnonzero(got != exp)
    assert bad.size == 0, f"{bad.size} of {w.size} cache elements differ"


def check_neighbours_kept(orc, lay, cache, data_seed, L, H, D, b, s):
    """Elements d = 0 and D-1 of token s of sequence b, every layer, K|V and
    head, still hold their generated values."""
    E = lay.elem_bytes
    idx = np.array([orc.elem_index(lay, l, kv, b, h, s, d) for l in range(L) for kv in (0, 1)
                    for h in range(H) for d in (0, D - 1)], np.int64)
    exp = synth.bytes_at(data_seed, idx.astype(np.uint64) * np.uint64(E), E).astype(G.NDT[E])
    assert np.array_equal(G.gather(cache, idx, E), exp)


def dense_limit_case(orc, kind, L, H, D, B, S, t0, t1, data_seed):
    E = 2
    okind = {dv.DV_DENSE: oracle.DENSE, dv.DV_DENSE_KSPLIT: oracle.KSPLIT}[kind]
    lay = oracle.Layout(okind, L, H, D, B, seq_cap=S, elem_bytes=E)
    cache = G.dev_filled(lay.storage_bytes(), data_seed)
    c = dv.Cache(kind, L, H, D, B, [cache], max_seq=S, elem_bytes=E)
    assert dv.dv_cache_bytes(c) == lay.storage_bytes()
    n = dv.dv_packed_bytes(c, 0, L, t0, t1)
    wire = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    assert dv.dv_stream_out_prompt(c, 0, 0, L, t0, t1, wire, n, stream()) == n
    torch.cuda.synchronize()
    check_wire(orc, lay, data_seed, wire, 0, L, t0, t1)

    # stream a filled wire in, then re-pack it
    wire2 = G.dev_filled(n, WIRE_SEED)
    dv.dv_stream_in(c, 0, 0, L, t0, t1, wire2, n, stream())
    torch.cuda.synchronize()
    check_landed(orc, lay, cache, 0, L, t0, t1)
    for b in range(B):
        if t0[b] > 0:
            check_neighbours_kept(orc, lay, cache, data_seed, L, H, D, b, int(t0[b]) - 1)
        if t1[b] < S:
            check_neighbours_kept(orc, lay, cache, data_seed, L, H, D, b, int(t1[b]))
    wire3 = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    dv.dv_stream_out_prompt(c, 0, 0, L, t0, t1, wire3, n, stream())
    torch.cuda.synchronize()
    assert torch.equal(wire3, wire2[:n])
    return lay, c, cache


def test_dense_cache_past_32_gib(oracle_lib):
    """17 heads x 1 GiB per K|V slab: the value slab's last head ends at
    34 GiB, past 2**31 16-byte units."""
    L, H, D, B, S = 1, 17, 512, 2, 1 << 20
    assert L * 2 * B * H * S * D * 2 >= 68 * GIB
    t0 = np.array([S - 300, 0], np.int32)
    t1 = np.array([S, 0], np.int32)  # sequence 1 (the upper 34 GiB) empty
    dense_limit_case(oracle_lib, dv.DV_DENSE, L, H, D, B, S, t0, t1, 3101)
    t0 = np.array([0, S - 129], np.int32)
    t1 = np.array([0, S - 1], np.int32)  # only sequence 1, ending 1 token short
    dense_limit_case(oracle_lib, dv.DV_DENSE, L, H, D, B, S, t0, t1, 3102)


def test_token_capacity_and_size_limits(oracle_lib):
    """max_seq = 2**24 with 64 units per token: capacity * units = 2**30,
    both at the limits; a prompt range and the last token."""
    L, H, D, B, S = 1, 1, 512, 1, 1 << 24
    t0 = np.array([S - 200], np.int32)
    t1 = np.array([S], np.int32)
    lay, c, cache = dense_limit_case(oracle_lib, dv.DV_DENSE, L, H, D, B, S, t0, t1, 3103)
    # the cache now holds the WIRE_SEED wire on [S-200, S): pack the last token
    pos = np.array([S - 1], np.int32)
    n = dv.dv_packed_bytes(c, 0, L, pos, pos + 1)
    inc = torch.empty(n, dtype=torch.uint8, device=G.DEV)
    assert dv.dv_stream_out_token(c, 0, 0, L, pos, inc, n, stream()) == n
    torch.cuda.synchronize()
    # token S-1 is element 199 of each slab's 200-token run on the first wire
    tok = D * 2
    w = G.host(G.dev_filled(2 * 200 * tok, WIRE_SEED))
    assert G.host(inc).tobytes() == w[199 * tok:200 * tok].tobytes() + \
        w[399 * tok:400 * tok].tobytes()
    # and a filled increment streamed in at S-1
    inc2 = G.dev_filled(n, WIRE_SEED)
    dv.dv_stream_in(c, 0, 0, L, pos, pos + 1, inc2, n, stream())
    torch.cuda.synchronize()
    check_landed(oracle_lib, lay, cache, 0, L, pos, pos + 1)


def test_split_key_at_capacity(oracle_lib):
    """Split key with 32 groups per token (the most) and max_seq = 2**24:
    group g of a head sits g * 2**24 units after group 0; ragged 64-token tiles."""
    L, H, D, B, S = 1, 2, 256, 1, 1 << 24
    t0 = np.array([S - 100], np.int32)
    t1 = np.array([S], np.int32)
    dense_limit_case(oracle_lib, dv.DV_DENSE_KSPLIT, L, H, D, B, S, t0, t1, 3104)


def test_paged_table_of_2_pow_20_blocks(oracle_lib):
    """Tables of 2**20 columns (capacity 2**24) with only the last columns
    mapped: gather, scatter into another permutation in table order and in
    pool order, and a decode-step token in the last slot."""
    L, H, D, B, E, bs = 2, 8, 128, 2, 2, 16
    maxb = 1 << 20
    cap = maxb * bs
    t0 = np.array([cap - 100, cap - 80], np.int32)
    t1 = np.array([cap, cap - 1], np.int32)
    cols = [np.arange((t0[b]) // bs, (t1[b] - 1) // bs + 1) for b in range(B)]
    nb = sum(len(x) for x in cols)
    assert nb == 12

    def table(seed):
        perm = synth.SplitMix64(seed).permutation(nb)
        bt = np.full((B, maxb), -1, np.int32)
        k = 0
        for b in range(B):
            for j in cols[b]:
                bt[b, j] = perm[k]
                k += 1
        return bt

    bt_a, bt_b = table(5), table(6)
    lay_a = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                          num_blocks=nb, block_table=bt_a)
    lay_b = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                          num_blocks=nb, block_table=bt_b)
    host = synth.fill_bytes(lay_a.storage_bytes(), 3105)
    pool = G.to_dev(host)
    bta, btb = G.to_dev(bt_a), G.to_dev(bt_b)
    ca = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=bs, num_blocks=nb,
                  max_blocks=maxb, block_tables=[bta])
    exp = oracle_lib.pack(lay_a, host, 0, L, t0, t1)
    wire = G.dev_const(exp.nbytes, 0)
    assert dv.dv_stream_out_prompt(ca, 0, 0, L, t0, t1, wire, exp.nbytes, stream()) == exp.nbytes
    torch.cuda.synchronize()
    assert G.host(wire).tobytes() == exp.tobytes()

    exp_b = np.full(lay_b.storage_bytes(), 0x3C, np.uint8)
    oracle_lib.unpack(lay_b, exp_b, 0, L, t0, t1, exp)
    owner = torch.full((nb,), 7, dtype=torch.int32, device=G.DEV)
    for owners in (None, [owner]):  # table order, then pool order
        pool_b = G.dev_const(lay_b.storage_bytes(), 0x3C)
        cb = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool_b], block_size=bs, num_blocks=nb,
                      max_blocks=maxb, block_tables=[btb], block_owners=owners)
        dv.dv_stream_in(cb, 0, 0, L, t0, t1, wire, exp.nbytes, stream())
        torch.cuda.synchronize()
        assert G.host(pool_b).tobytes() == exp_b.tobytes()
    # pool order ran: the workspace holds the table's inverse over the ranges
    assert np.array_equal(G.host(owner), G.owner_map_expected(bt_b, nb, bs, t0, t1))

    pos = np.array([cap - 1, cap - 2], np.int32)
    exp_t = oracle_lib.pack(lay_a, host, 0, L, pos, pos + 1)
    inc = G.dev_const(exp_t.nbytes, 0)
    assert dv.dv_stream_out_token(ca, 0, 0, L, pos, inc, exp_t.nbytes, stream()) == exp_t.nbytes
    torch.cuda.synchronize()
    assert G.host(inc).tobytes() == exp_t.tobytes()

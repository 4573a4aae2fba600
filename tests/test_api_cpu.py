"""The C-ABI library without a GPU: it loads, exports what include/dv.h
declares, sizes streams as the oracle does, and rejects bad arguments before
enqueuing anything (no call here reaches the HIP runtime)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2403_01876_amd import dv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "dv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert set(names) == set(dv.EXPORTS), names
    lib = ctypes.CDLL(dv.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert dv.dv_api_version() == dv.API_VERSION == 3


def test_status_strings():
    for s in (0, -1, -2, -3, -4, -5):
        assert dv.status_string(s) and dv.status_string(s) != "unknown status"
    assert dv.status_string(-99) == "unknown status"


FAKE = 1 << 40  # an aligned address never dereferenced by the host checks


def dense(L=2, H=3, D=64, B=4, S=50, E=2, bases=(FAKE,), kind=dv.DV_DENSE, mem=dv.DV_MEM_DEVICE):
    return dv.Cache(kind, L, H, D, B, list(bases), max_seq=S, elem_bytes=E, mem=mem)


@pytest.mark.parametrize("seed", range(20))
def test_packed_bytes_matches_oracle(seed, oracle_lib):
    r = np.random.default_rng(seed)
    L, H, B, S = int(r.integers(1, 5)), int(r.integers(1, 9)), int(r.integers(1, 80)), \
        int(r.integers(1, 300))
    E = int(r.choice([1, 2, 4]))
    D = int(r.choice([16, 32, 64, 128])) // E * E
    D = max(D - D % (16 // E), 16 // E)
    c = dense(L, H, D, B, S, E)
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    t0 = r.integers(0, S + 1, size=B).astype(np.int32)
    t1 = np.minimum(t0 + r.integers(0, S + 1, size=B), S).astype(np.int32)
    l0 = int(r.integers(0, L + 1))
    l1 = int(r.integers(l0, L + 1))
    assert dv.dv_packed_bytes(c, l0, l1, t0, t1) == oracle_lib.wire_elems(lay, l0, l1, t0, t1) * E
    assert dv.dv_cache_bytes(c) == lay.storage_bytes()


def test_packed_bytes_paged():
    bt = np.zeros((4, 10), np.int32)
    c = dv.Cache(dv.DV_PAGED, 3, 8, 128, 4, [FAKE], block_size=16, num_blocks=30,
                 max_blocks=10, block_tables=[FAKE])
    assert dv.dv_cache_bytes(c) == 3 * 2 * 30 * 8 * 16 * 128 * 2
    t1 = np.array([160, 0, 5, 17], np.int32)
    assert dv.dv_packed_bytes(c, 0, 3, None, t1) == 3 * 2 * 8 * 128 * 2 * int(t1.sum())
    rc, _ = dv.dv_packed_bytes(c, 0, 3, None, [161, 0, 0, 0], check=False)
    assert rc == dv.DV_ERR_RANGE
    del bt


def test_negative_microbatch_and_slot_are_rejected():
    """Every call that addresses a microbatch or slot rejects an index below
    zero with DV_ERR_RANGE before touching memory (a regression test: an
    index of -1 once reached the sizing-only path and passed a null base)."""
    c = dense(bases=(FAKE, FAKE + (1 << 32)))
    h = dense(bases=(FAKE + (1 << 34),), mem=dv.DV_MEM_HOST_PINNED)
    z = np.zeros(4, np.int32)
    t1 = np.full(4, 10, np.int32)
    wire = FAKE + (1 << 36)
    for mb in (-1, -2, 2):
        rc, _ = dv.dv_stream_out_prompt(c, mb, 0, 2, z, t1, wire, 1 << 30, check=False)
        assert rc == dv.DV_ERR_RANGE, mb
        rc, _ = dv.dv_stream_out_token(c, mb, 0, 2, t1, wire, 1 << 30, check=False)
        assert rc == dv.DV_ERR_RANGE, mb
        assert dv.dv_stream_in(c, mb, 0, 2, z, t1, wire, 1 << 30, check=False) == dv.DV_ERR_RANGE
        assert dv.dv_swap_out(c, mb, h, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_RANGE
        assert dv.dv_swap_in(h, 0, c, mb, 0, 2, z, t1, check=False) == dv.DV_ERR_RANGE
    for hb in (-1, 1):
        assert dv.dv_swap_out(c, 0, h, hb, 0, 2, z, t1, check=False) == dv.DV_ERR_RANGE
        assert dv.dv_swap_in(h, hb, c, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_RANGE
    # sizing calls take no microbatch and still work
    assert dv.dv_packed_bytes(c, 0, 2, z, t1) == 2 * 2 * 3 * 64 * 2 * 40
    assert dv.dv_cache_bytes(c) == 2 * 2 * 4 * 3 * 50 * 64 * 2


def test_block_claims_rejections():
    d = dense()
    z = np.zeros(4, np.int32)
    t1 = np.full(4, 10, np.int32)
    cnt = FAKE + (1 << 36)
    assert dv.dv_block_claims(d, 0, z, t1, cnt, check=False) == dv.DV_ERR_UNSUPPORTED
    p = dv.Cache(dv.DV_PAGED, 2, 3, 64, 4, [FAKE], block_size=16, num_blocks=8, max_blocks=4,
                 block_tables=[FAKE + (1 << 35)])
    assert dv.dv_block_claims(p, 1, z, t1, cnt, check=False) == dv.DV_ERR_RANGE
    assert dv.dv_block_claims(p, -1, z, t1, cnt, check=False) == dv.DV_ERR_RANGE
    assert dv.dv_block_claims(p, 0, z, np.full(4, 65, np.int32), cnt,
                              check=False) == dv.DV_ERR_RANGE
    assert dv.dv_block_claims(p, 0, z, t1, None, check=False) == dv.DV_ERR_INVALID
    assert dv.dv_block_claims(p, 0, z, t1, cnt + 2, check=False) == dv.DV_ERR_INVALID
    assert dv.dv_block_claims(p, 0, z, t1, FAKE + 64, check=False) == dv.DV_ERR_INVALID


def test_owner_workspace_rejections():
    """A paged receiver's owner-map workspace must be 4-byte aligned and must
    not overlap the pool or the source buffer; all checked on the host."""
    L, H, D, B, NB, MB = 2, 4, 64, 3, 12, 4
    pool = FAKE
    pool_bytes = L * 2 * NB * H * 16 * D * 2
    wire = FAKE + (1 << 34)
    t1 = np.array([16, 33, 0], np.int32)

    def paged(owner):
        return dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=16, num_blocks=NB,
                        max_blocks=MB, block_tables=[FAKE + (1 << 35)], block_owners=[owner])

    need = dv.dv_packed_bytes(paged(None), 0, L, None, t1)
    for owner, rc in ((FAKE + (1 << 36) + 2, dv.DV_ERR_INVALID),   # misaligned
                      (pool + pool_bytes - 16, dv.DV_ERR_INVALID),  # inside the pool
                      (wire + 64, dv.DV_ERR_INVALID)):              # inside the source
        assert dv.dv_stream_in(paged(owner), 0, 0, L, None, t1, wire, need,
                               check=False) == rc, hex(owner)
    # a pack through the same descriptor checks alignment too (the map is
    # then unused, so overlap with the pool is not an error for packs)
    rc, _ = dv.dv_stream_out_prompt(paged(FAKE + (1 << 36) + 2), 0, 0, L, None, t1, wire, need,
                                    check=False)
    assert rc == dv.DV_ERR_INVALID


def test_noalloc_stream_in_limits():
    """dv_stream_in_noalloc refuses a paged pool past its static owner map
    (DV_NOALLOC_MAX_BLOCKS blocks) before anything else; at the limit the
    call gets as far as the ordinary argument checks.  The workspace field
    of the descriptor is ignored, misaligned or not."""
    z, t1 = np.zeros(1, np.int32), np.ones(1, np.int32)

    def pool(nb, owner=None):
        return dv.Cache(dv.DV_PAGED, 1, 1, 64, 1, [FAKE], block_size=16, num_blocks=nb,
                        max_blocks=4, block_tables=[FAKE + (1 << 36)], block_owners=[owner])

    over = pool(dv.NOALLOC_MAX_BLOCKS + 1)
    assert dv.dv_stream_in_noalloc(over, 0, 0, 1, z, t1, FAKE + (1 << 38), 1 << 20,
                                   check=False) == dv.DV_ERR_UNSUPPORTED
    at = pool(dv.NOALLOC_MAX_BLOCKS, owner=FAKE + (1 << 37) + 2)
    assert dv.dv_stream_in_noalloc(at, 0, 0, 1, z, t1, None, 1 << 20,
                                   check=False) == dv.DV_ERR_INVALID  # null source
    assert dv.dv_stream_in_noalloc(at, 0, 0, 1, z, t1, FAKE + (1 << 38), 16,
                                   check=False) == dv.DV_ERR_SPACE
    # the same descriptor through dv_stream_in: the misaligned workspace counts
    assert dv.dv_stream_in(at, 0, 0, 1, z, t1, FAKE + (1 << 38), 1 << 20,
                           check=False) == dv.DV_ERR_INVALID
    dense = dv.Cache(dv.DV_DENSE, 1, 1, 64, 1, [FAKE], max_seq=8)
    assert dv.dv_stream_in_noalloc(dense, 0, 0, 1, z, np.array([9], np.int32),
                                   FAKE + (1 << 38), 1 << 20,
                                   check=False) == dv.DV_ERR_RANGE


def test_block_table_must_not_overlap_what_a_call_writes():
    """The kernels read the block table while the call writes the stream's
    destination (pack), the pool (unpack), the owner map or the claim
    counts; a table overlapping any of them is refused on the host."""
    L, H, D, B, NB, MB = 2, 4, 64, 3, 12, 4
    pool = FAKE
    pool_bytes = L * 2 * NB * H * 16 * D * 2
    table_bytes = B * MB * 4
    wire = FAKE + (1 << 34)
    owner = FAKE + (1 << 36)
    t1 = np.array([16, 33, 0], np.int32)

    def paged(table, own=None):
        return dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=16, num_blocks=NB,
                        max_blocks=MB, block_tables=[table], block_owners=[own])

    need = dv.dv_packed_bytes(paged(FAKE + (1 << 35)), 0, L, None, t1)
    bad = dv.DV_ERR_INVALID
    # pack: the table inside the destination (its first or last bytes)
    for table in (wire + need - 16, wire - table_bytes + 4):
        rc, _ = dv.dv_stream_out_prompt(paged(table), 0, 0, L, None, t1, wire, need,
                                        check=False)
        assert rc == bad, hex(table)
    # unpack: the table inside the pool, or inside the owner map
    assert dv.dv_stream_in(paged(pool + pool_bytes - 8), 0, 0, L, None, t1, wire, need,
                           check=False) == bad
    assert dv.dv_stream_in(paged(owner + 16, owner), 0, 0, L, None, t1, wire, need,
                           check=False) == bad
    # claim counts over the table
    counts = FAKE + (1 << 37)
    assert dv.dv_block_claims(paged(counts + 4 * NB - 4), 0, None, t1, counts,
                              check=False) == bad
    # sizing does not look at addresses
    assert dv.dv_packed_bytes(paged(pool), 0, L, None, t1) == need


def test_range_errors():
    c = dense()
    z = np.zeros(4, np.int32)
    full = np.full(4, 50, np.int32)
    assert dv.dv_packed_bytes(c, 0, 2, z, full, check=False)[0] == dv.DV_OK
    assert dv.dv_packed_bytes(c, 0, 3, z, full, check=False)[0] == dv.DV_ERR_RANGE
    assert dv.dv_packed_bytes(c, 2, 1, z, full, check=False)[0] == dv.DV_ERR_RANGE
    assert dv.dv_packed_bytes(c, -1, 1, z, full, check=False)[0] == dv.DV_ERR_RANGE
    assert dv.dv_packed_bytes(c, 0, 2, z, full + 1, check=False)[0] == dv.DV_ERR_RANGE
    assert dv.dv_packed_bytes(c, 0, 2, full, z, check=False)[0] == dv.DV_ERR_RANGE
    assert dv.dv_packed_bytes(c, 0, 2, z - 1, full, check=False)[0] == dv.DV_ERR_RANGE
    # empty layer range and empty token ranges are valid, zero bytes
    assert dv.dv_packed_bytes(c, 1, 1, z, full) == 0
    assert dv.dv_packed_bytes(c, 0, 2, full, full) == 0


def test_invalid_descriptors():
    z = np.zeros(4, np.int32)
    one = np.ones(4, np.int32)
    for bad in (dense(D=36), dense(L=0), dense(H=0), dense(B=0), dense(S=0), dense(E=0),
                dense(kind=7), dense(mem=5)):
        assert dv.dv_packed_bytes(bad, 0, 1, z, one, check=False)[0] == dv.DV_ERR_INVALID
    paged_no_table = dv.Cache(dv.DV_PAGED, 1, 1, 64, 4, [FAKE], block_size=16, num_blocks=4,
                              max_blocks=2)
    assert dv.dv_packed_bytes(paged_no_table, 0, 1, z, one, check=False)[0] == dv.DV_ERR_INVALID


def test_stream_calls_reject_before_enqueue():
    """Errors return before any HIP call, so they work without a GPU."""
    c = dense()
    z = np.zeros(4, np.int32)
    t1 = np.array([10, 0, 3, 50], np.int32)
    need = dv.dv_packed_bytes(c, 0, 2, z, t1)
    rc, n = dv.dv_stream_out_prompt(c, 0, 0, 2, z, t1, FAKE + (1 << 30), need - 16, check=False)
    assert rc == dv.DV_ERR_SPACE and n == need
    rc, _ = dv.dv_stream_out_prompt(c, 1, 0, 2, z, t1, FAKE + (1 << 30), need, check=False)
    assert rc == dv.DV_ERR_RANGE  # microbatch 1 of 1
    rc, _ = dv.dv_stream_out_prompt(c, 0, 0, 2, z, t1, FAKE + (1 << 30) + 8, need, check=False)
    assert rc == dv.DV_ERR_INVALID  # misaligned destination
    rc, _ = dv.dv_stream_out_prompt(c, 0, 0, 2, z, t1, FAKE + 64, need, check=False)
    assert rc == dv.DV_ERR_INVALID  # destination overlaps the cache
    rc, _ = dv.dv_stream_out_prompt(c, 0, 0, 2, z, t1, 0, need, check=False)
    assert rc == dv.DV_ERR_INVALID  # null destination
    misaligned = dense(bases=(FAKE + 4,))
    rc, _ = dv.dv_stream_out_prompt(misaligned, 0, 0, 2, z, t1, FAKE + (1 << 30), need,
                                    check=False)
    assert rc == dv.DV_ERR_INVALID
    assert dv.dv_stream_in(c, 0, 0, 2, z, t1, FAKE + (1 << 30), need - 1, check=False) == \
        dv.DV_ERR_SPACE
    assert dv.dv_stream_in(c, 0, 0, 2, z, t1 + 50, FAKE + (1 << 30), need,
                           check=False) == dv.DV_ERR_RANGE
    pos = np.array([49, -1, 3, 50], np.int32)  # 50 is past capacity
    rc, _ = dv.dv_stream_out_token(c, 0, 0, 2, pos, FAKE + (1 << 30), 1 << 20, check=False)
    assert rc == dv.DV_ERR_RANGE
    # zero-byte streams succeed without touching anything
    assert dv.dv_stream_out_prompt(c, 0, 0, 2, z, z, 0, 0) == 0
    assert dv.dv_stream_out_token(c, 0, 0, 2, np.full(4, -1, np.int32), 0, 0) == 0
    assert dv.dv_stream_in(c, 0, 1, 1, z, t1, 0, 0) == dv.DV_OK


def test_ksplit_limits():
    z = np.zeros(4, np.int32)
    one = np.ones(4, np.int32) * 2
    big = dense(D=512, kind=dv.DV_DENSE_KSPLIT)  # 64 groups of 16 bytes per token
    rc, _ = dv.dv_stream_out_prompt(big, 0, 0, 1, z, one, FAKE + (1 << 34), 1 << 30,
                                    check=False)
    assert rc == dv.DV_ERR_UNSUPPORTED


def test_swap_rejections():
    z = np.zeros(4, np.int32)
    t1 = np.full(4, 10, np.int32)
    d = dense()
    h = dense(bases=(FAKE + (1 << 33),), mem=dv.DV_MEM_HOST_PINNED, S=20)
    # direction must match the memory kinds
    assert dv.dv_swap_out(h, 0, d, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_INVALID
    assert dv.dv_swap_in(d, 0, h, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_INVALID
    # shapes must agree
    h2 = dense(H=4, bases=(FAKE + (1 << 33),), mem=dv.DV_MEM_HOST_PINNED)
    assert dv.dv_swap_out(d, 0, h2, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_INVALID
    # the host mirror must hold the range
    hs = dense(S=8, bases=(FAKE + (1 << 33),), mem=dv.DV_MEM_HOST_PINNED)
    assert dv.dv_swap_out(d, 0, hs, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_RANGE
    # paged caches are not swapped
    p = dv.Cache(dv.DV_PAGED, 2, 3, 64, 4, [FAKE], block_size=16, num_blocks=8, max_blocks=4,
                 block_tables=[FAKE])
    assert dv.dv_swap_out(p, 0, h, 0, 0, 2, z, t1, check=False) == dv.DV_ERR_UNSUPPORTED
    # empty ranges are a no-op
    assert dv.dv_swap_out(d, 0, h, 0, 0, 2, z, z) == dv.DV_OK


def test_swapper_create_rejections():
    """Bad scheduler arguments are rejected before any stream is created."""
    import ctypes as C
    dev = dense(bases=(FAKE, FAKE + (1 << 32)))
    host = dense(bases=(FAKE + (1 << 34),) * 4, mem=dv.DV_MEM_HOST_PINNED, S=64)
    h = C.c_void_p(0)
    one_slot = dense(bases=(FAKE,))
    assert dv.lib.dv_swapper_create(one_slot.ref, host.ref, C.byref(h)) == dv.DV_ERR_INVALID
    assert dv.lib.dv_swapper_create(host.ref, dev.ref, C.byref(h)) == dv.DV_ERR_INVALID
    other = dense(H=4, bases=(FAKE + (1 << 34),) * 4, mem=dv.DV_MEM_HOST_PINNED)
    assert dv.lib.dv_swapper_create(dev.ref, other.ref, C.byref(h)) == dv.DV_ERR_INVALID
    paged = dv.Cache(dv.DV_PAGED, 2, 3, 64, 4, [FAKE, FAKE], block_size=16, num_blocks=8,
                     max_blocks=4, block_tables=[FAKE, FAKE])
    assert dv.lib.dv_swapper_create(paged.ref, host.ref, C.byref(h)) == dv.DV_ERR_UNSUPPORTED
    assert dv.lib.dv_swapper_create(dev.ref, host.ref, None) == dv.DV_ERR_INVALID
    # the two slots must be disjoint, and so must the host mirrors (which
    # hold 2*2*4*3*64*64*2 bytes each here)
    mirror = 2 * 2 * 4 * 3 * 64 * 64 * 2
    mirrors = [FAKE + (1 << 34) + i * mirror for i in range(4)]
    apart = dense(bases=mirrors, mem=dv.DV_MEM_HOST_PINNED, S=64)
    for slots in ((FAKE, FAKE), (FAKE, FAKE + 2 * 2 * 4 * 3 * 50 * 64 * 2 - 16), (FAKE, 0)):
        assert dv.lib.dv_swapper_create(dense(bases=slots).ref, apart.ref, C.byref(h)) == \
            dv.DV_ERR_INVALID, slots
    for bases in (mirrors[:3] + [mirrors[1] + 16], mirrors[:3] + [mirrors[3] + 8]):
        hosts = dense(bases=bases, mem=dv.DV_MEM_HOST_PINNED, S=64)
        assert dv.lib.dv_swapper_create(dev.ref, hosts.ref, C.byref(h)) == dv.DV_ERR_INVALID
    assert h.value is None
    for f in ("dv_swapper_sync", "dv_swapper_destroy"):
        assert getattr(dv.lib, f)(None) == dv.DV_ERR_INVALID


def test_streamer_create_rejections():
    import ctypes as C
    c = dense()
    h = C.c_void_p(0)
    st = FAKE + (1 << 33)
    assert dv.lib.dv_streamer_create(None, 0, st, 1 << 20, st, 1 << 20, C.byref(h)) == \
        dv.DV_ERR_INVALID
    assert dv.lib.dv_streamer_create(c.ref, 1, st, 1 << 20, st, 1 << 20, C.byref(h)) == \
        dv.DV_ERR_RANGE
    assert dv.lib.dv_streamer_create(c.ref, 0, st + 8, 1 << 20, st, 1 << 20, C.byref(h)) == \
        dv.DV_ERR_INVALID
    assert dv.lib.dv_streamer_create(c.ref, 0, None, 1 << 20, st, 1 << 20, C.byref(h)) == \
        dv.DV_ERR_INVALID
    assert dv.lib.dv_streamer_create(dense(D=36).ref, 0, st, 1 << 20, st, 1 << 20,
                                     C.byref(h)) == dv.DV_ERR_INVALID
    # staging, destination and the source microbatch must not overlap
    other = FAKE + (1 << 34)
    assert dv.lib.dv_streamer_create(c.ref, 0, st, 1 << 20, st + (1 << 19), 1 << 20,
                                     C.byref(h)) == dv.DV_ERR_INVALID
    assert dv.lib.dv_streamer_create(c.ref, 0, FAKE + 4096, 1 << 20, other, 1 << 20,
                                     C.byref(h)) == dv.DV_ERR_INVALID
    assert dv.lib.dv_streamer_create(c.ref, 0, st, 1 << 20, FAKE + 4096, 1 << 20,
                                     C.byref(h)) == dv.DV_ERR_INVALID
    # nor may staging or destination cover a paged source's block table
    table = FAKE + (1 << 35)
    pg = dv.Cache(dv.DV_PAGED, 2, 4, 64, 3, [FAKE], block_size=16, num_blocks=12,
                  max_blocks=4, block_tables=[table])
    for stg, dst in ((table - 64, other), (st, table + 40)):
        assert dv.lib.dv_streamer_create(pg.ref, 0, stg, 1 << 10, dst, 1 << 10,
                                         C.byref(h)) == dv.DV_ERR_INVALID, (hex(stg), hex(dst))
    assert h.value is None
    for f in ("dv_streamer_flush", "dv_streamer_destroy"):
        assert getattr(dv.lib, f)(None) == dv.DV_ERR_INVALID


def test_plain_copy_baseline_rejections():
    """The copy-ceiling baseline checks its arguments before launching."""
    from paper_2403_01876_amd import baseline
    lib = baseline._load()
    bad = dv.DV_ERR_INVALID
    for dst, src, n in ((FAKE + 8, FAKE + (1 << 30), 64),      # misaligned destination
                        (FAKE, FAKE + (1 << 30) + 4, 64),      # misaligned source
                        (FAKE, FAKE + (1 << 30), 60),          # not whole 16-byte units
                        (FAKE, FAKE + 32, 64),                 # overlapping regions
                        (None, FAKE, 64)):
        assert lib.dvb_plain_copy(dst, src, n, None) == bad, (dst, src, n)
    assert lib.dvb_plain_copy(FAKE, FAKE + 16, 0, None) == dv.DV_OK  # nothing to copy


def test_block_copy_baseline_rejections():
    """The paged kernels' block-order ceiling checks its arguments first."""
    from paper_2403_01876_amd import baseline
    lib = baseline._load()
    bad = dv.DV_ERR_INVALID
    far, order = FAKE + (1 << 34), FAKE + (1 << 36)
    for dst, src, o, nb, bb in ((FAKE + 8, far, order, 4, 8192),   # misaligned destination
                                (FAKE, far + 4, order, 4, 8192),   # misaligned source
                                (FAKE, far, order + 2, 4, 8192),   # misaligned order
                                (FAKE, far, None, 4, 8192),        # no order
                                (FAKE, far, order, 4, 4096),       # block not whole pieces
                                (FAKE, far, order, 4, 0),
                                (FAKE, FAKE + 8192, order, 4, 8192)):  # overlapping
        assert lib.dvb_block_copy(dst, src, o, nb, bb, 0, None) == bad, (dst, src, o, nb, bb)
    assert lib.dvb_block_copy(FAKE, far, order, 0, 8192, 1, None) == dv.DV_OK  # nothing
    assert lib.dvb_block_copy(FAKE, FAKE + (1 << 45), order, 1 << 31, 8192, 0,
                              None) == dv.DV_ERR_UNSUPPORTED  # 2^31 pieces


def test_binding_fails_loudly_without_the_library(tmp_path):
    """No fallback: a copy of the package without libdv.so refuses to import."""
    import shutil
    import subprocess
    import sys
    pkg = os.path.join(ROOT, "paper_2403_01876_amd")
    dst = tmp_path / "paper_2403_01876_amd"
    shutil.copytree(pkg, dst, ignore=shutil.ignore_patterns("*.so", "__pycache__", "csrc"))
    code = ("import sys; sys.path.insert(0, %r)\n"
            "try:\n    import paper_2403_01876_amd\nexcept ImportError as e:\n"
            "    print('refused:', e); sys.exit(3)\nsys.exit(0)\n") % str(tmp_path)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 3, r.stdout + r.stderr
    assert "libdv.so is missing" in r.stdout


C_PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "dv.h"

int main(void) {
  void* bases[1] = {(void*)(unsigned long long)(1ull << 40)};
  dv_cache c;
  memset(&c, 0, sizeof c);
  c.kind = DV_DENSE; c.mem = DV_MEM_DEVICE; c.elem_bytes = 2;
  c.num_layers = 10; c.num_heads = 40; c.head_dim = 128; c.batch = 8; c.max_seq = 2048;
  c.num_mb = 1; c.mb_base = bases;
  int32_t t1[8] = {512, 600, 700, 800, 900, 1000, 1024, 0};
  uint64_t bytes = 0, cache = 0;
  if (dv_packed_bytes(&c, 0, 10, NULL, t1, &bytes) != DV_OK) return 1;
  if (dv_cache_bytes(&c, &cache) != DV_OK) return 2;
  /* validation errors come back before anything reaches the runtime */
  int rc = dv_stream_out_prompt(&c, -1, 0, 10, NULL, t1, NULL, 0, NULL, NULL);
  printf("%llu %llu %d %s %d\n", (unsigned long long)bytes, (unsigned long long)cache, rc,
         dv_status_string(rc), dv_api_version());
  return 0;
}
"""


def test_header_and_library_from_c(tmp_path):
    """The boundary from plain C: include/dv.h compiles as C99 with warnings
    as errors, and a program linked against libdv.so sizes a stream and gets
    validation errors back (no GPU needed)."""
    import subprocess
    src = tmp_path / "use_dv.c"
    src.write_text(C_PROGRAM)
    exe = tmp_path / "use_dv"
    libdir = os.path.dirname(dv.LIB_PATH)
    cc = subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                         "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                         "-L", libdir, "-ldv", "-Wl,-rpath," + libdir],
                        capture_output=True, text=True, timeout=120)
    assert cc.returncode == 0, cc.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    n, cache, rc, *rest = run.stdout.split()
    assert int(n) == 10 * 2 * 40 * 128 * 2 * (512 + 600 + 700 + 800 + 900 + 1000 + 1024)
    assert int(cache) == 10 * 2 * 8 * 40 * 2048 * 128 * 2
    assert int(rc) == dv.DV_ERR_RANGE and rest[-1] == str(dv.API_VERSION)


def test_descriptor_keeps_its_buffers_alive():
    """A descriptor built from temporaries keeps them referenced, so their
    memory cannot be reused while the descriptor holds their addresses."""
    import gc
    import weakref

    class Buf:
        def __init__(self):
            self.a = np.zeros(64, np.uint8)

        def data_ptr(self):
            return self.a.ctypes.data

    b = Buf()
    ref = weakref.ref(b)
    c = dv.Cache(dv.DV_DENSE, 1, 1, 16, 1, [b], max_seq=1)
    del b
    gc.collect()
    assert ref() is not None
    del c
    gc.collect()
    assert ref() is None


def test_extent_limits_at_and_past_the_boundary():
    """Each extent limit the header lists: the largest accepted value sizes
    its stream, one step past it is DV_ERR_UNSUPPORTED (sizing calls only)."""
    z1 = np.zeros(1, np.int32)
    U = dv.DV_ERR_UNSUPPORTED

    def sized(c, t1):
        return dv.dv_packed_bytes(c, 0, 1, z1, np.array([t1], np.int32), check=False)

    # 2^24 layers (a launch's first slab index, 2 * layer + 1, is an int32)
    assert sized(dense(L=1 << 24, H=1, D=8, B=1, S=1), 1) == (0, 2 * 16)
    assert sized(dense(L=(1 << 24) + 1, H=1, D=8, B=1, S=1), 1)[0] == U
    assert dv.dv_cache_bytes(dense(L=(1 << 24) + 1, H=1, D=8, B=1, S=1), check=False)[0] == U
    # token capacity 2^24 (dense max_seq)
    assert sized(dense(L=1, H=1, D=8, B=1, S=1 << 24), 1 << 24) == (0, 2 * 16 << 24)
    assert sized(dense(L=1, H=1, D=8, B=1, S=(1 << 24) + 1), 1)[0] == U
    # token capacity of a paged table: max_blocks * block_size
    paged = lambda maxb: dv.Cache(dv.DV_PAGED, 1, 1, 8, 1, [FAKE], block_size=16,  # noqa: E731
                                  num_blocks=4, max_blocks=maxb, block_tables=[FAKE])
    assert sized(paged(1 << 20), 1 << 24) == (0, 2 * 16 << 24)
    assert sized(paged((1 << 20) + 1), 1)[0] == U
    # one head of a paged block: block_size * head_dim * elem_bytes = 2^33
    # bytes (2^29 units; the paged kernel counts two heads' units in int32)
    # (within the capacity limits above only for head_dim * elem_bytes >= 2^9)
    blk = lambda bs: dv.Cache(dv.DV_PAGED, 1, 1, 512, 1, [FAKE], block_size=bs,  # noqa: E731
                              num_blocks=4, max_blocks=1, block_tables=[FAKE])
    assert sized(blk(1 << 23), 1) == (0, 2 * 1024)
    assert sized(blk((1 << 23) + 1), 1)[0] == U
    assert dv.dv_cache_bytes(blk((1 << 23) + 1), check=False)[0] == U
    # head_dim * elem_bytes = 2^20 bytes (2^16 units)
    assert sized(dense(L=1, H=1, D=1 << 19, B=1, S=2), 1) == (0, 2 << 20)
    assert sized(dense(L=1, H=1, D=(1 << 19) + 8, B=1, S=2), 1)[0] == U
    # heads * head_dim * elem_bytes = 2^24 bytes
    assert sized(dense(L=1, H=1 << 16, D=128, B=1, S=2), 1) == (0, 2 << 24)
    assert sized(dense(L=1, H=(1 << 16) + 1, D=128, B=1, S=2), 1)[0] == U
    # capacity * head_dim * elem_bytes = 2^34 bytes
    assert sized(dense(L=1, H=1, D=512, B=1, S=1 << 24), 1) == (0, 2 * 1024)
    assert sized(dense(L=1, H=1, D=520, B=1, S=1 << 24), 1)[0] == U
    # storage below 2^48 bytes: 2^13 layers x 2 x 2^10 sequences x 2^24 bytes
    assert dv.dv_cache_bytes(dense(L=1 << 13, H=1, D=8, B=(1 << 10) - 1, S=1 << 20)) \
        == (1 << 13) * 2 * ((1 << 10) - 1) * (1 << 24)
    assert dv.dv_cache_bytes(dense(L=1 << 13, H=1, D=8, B=1 << 10, S=1 << 20), check=False)[0] == U
    # a paged table can address more tokens than the pool holds: its longest
    # stream (every sequence at capacity) is bounded the same way
    def sized_b(c):
        B = c.c.batch
        return dv.dv_packed_bytes(c, 0, 1, np.zeros(B, np.int32), np.ones(B, np.int32),
                                  check=False)

    pg = lambda B: dv.Cache(dv.DV_PAGED, 1 << 13, 1, 8, B, [FAKE], block_size=16,  # noqa: E731
                            num_blocks=4, max_blocks=1 << 16, block_tables=[FAKE])
    assert sized_b(pg((1 << 10) - 1)) == (0, 2 * 16 * ((1 << 10) - 1))
    assert sized_b(pg(1 << 10))[0] == U
    # products that would wrap 64 bits are refused, not wrapped
    assert sized(dense(L=1 << 24, H=1 << 4, D=128, B=1, S=1 << 24), 1)[0] == U
    assert dv.dv_cache_bytes(dense(L=1 << 24, H=1 << 16, D=128, B=1 << 30, S=1 << 24),
                             check=False)[0] == U


def test_binding_refuses_per_microbatch_arrays_of_another_length():
    """The library reads block_table[mb] and block_owner[mb] for every
    microbatch index below num_mb = len(bases); the binding refuses table
    and owner arrays whose length differs from the bases'."""
    kw = dict(block_size=16, num_blocks=4, max_blocks=2)
    with pytest.raises(ValueError):
        dv.Cache(dv.DV_PAGED, 1, 1, 8, 1, [FAKE, FAKE + (1 << 30)], block_tables=[FAKE], **kw)
    with pytest.raises(ValueError):
        dv.Cache(dv.DV_PAGED, 1, 1, 8, 1, [FAKE], block_tables=[FAKE],
                 block_owners=[FAKE, FAKE], **kw)
    c = dv.Cache(dv.DV_PAGED, 1, 1, 8, 1, [FAKE, FAKE + (1 << 30)],
                 block_tables=[FAKE + (1 << 40), FAKE + (1 << 41)], block_owners=[None, None],
                 **kw)
    assert c.c.num_mb == 2


def test_binding_refuses_range_arrays_shorter_than_the_batch():
    """The library reads one range entry per sequence and cannot see an
    array's length: the binding refuses a short one before the call."""
    c = dense(B=4)
    with pytest.raises(ValueError):
        dv.dv_packed_bytes(c, 0, 2, None, np.array([1, 2, 3], np.int32))
    with pytest.raises(ValueError):
        dv.dv_stream_out_prompt(c, 0, 0, 2, [0, 0], np.ones(4, np.int32), FAKE + (1 << 30), 1)
    with pytest.raises(ValueError):
        dv.dv_stream_out_token(c, 0, 0, 2, [1, 2, 3], FAKE + (1 << 30), 1 << 20)
    with pytest.raises(ValueError):
        dv.dv_stream_in(c, 0, 0, 2, None, [5], FAKE + (1 << 30), 1 << 20)
    assert dv.dv_packed_bytes(c, 0, 2, None, np.ones(4, np.int32)) == 2 * 2 * 3 * 64 * 2 * 4


def test_oversized_later_launch_group_is_refused_before_any_launch():
    """With more than 64 sequences a call runs in launch groups.  When only a
    later group's grid passes 2^31 units or tiles the call must still refuse
    before enqueuing the earlier groups: here it returns
    DV_ERR_UNSUPPORTED, where a launch attempt (no GPU in this process)
    would have returned DV_ERR_HIP."""
    U = dv.DV_ERR_UNSUPPORTED
    H, B = 1 << 20, 128
    z = np.zeros(B, np.int32)
    wire = 1 << 48  # far from every fake cache below

    def lens(small, large):
        return np.array([small] * 64 + [large] * 64, np.int32)

    def both_directions(c, t1):
        n = dv.dv_packed_bytes(c, 0, 1, z, t1)
        assert dv.dv_stream_out_prompt(c, 0, 0, 1, z, t1, wire, n, check=False)[0] == U
        assert dv.dv_stream_in(c, 0, 0, 1, z, t1, wire, n, check=False) == U

    # short runs: 64 sequences x 32 tokens x 2^20 heads = 2^31 units
    both_directions(dense(L=1, H=H, D=8, B=B, S=64), lens(1, 32))
    # dense tiles: 64 x 2^20 heads x 32 tiles of 512 units
    both_directions(dense(L=1, H=H, D=8, B=B, S=1 << 14), lens(1, 1 << 14))
    # split key: the key slabs' 64-token tiles pass 2^31 (the value slabs'
    # 512-unit tiles do not)
    both_directions(dense(L=1, H=H, D=8, B=B, S=2048, kind=dv.DV_DENSE_KSPLIT),
                    lens(1, 2048))
    # paged: 64 x 64 blocks x 2^19 head pairs
    pg = dv.Cache(dv.DV_PAGED, 1, H, 8, B, [FAKE], block_size=16, num_blocks=B * 64,
                  max_blocks=64, block_tables=[FAKE + (1 << 46)])
    both_directions(pg, lens(1, 1024))
    # swap of narrow rows through the copy kernel: 64 x 32 x 2^20 units
    dev_c = dense(L=1, H=H, D=8, B=B, S=64)
    host_c = dense(L=1, H=H, D=8, B=B, S=64, bases=(1 << 44,), mem=dv.DV_MEM_HOST_PINNED)
    assert dv.dv_swap_out(dev_c, 0, host_c, 0, 0, 1, z, lens(1, 32), check=False) == U
    assert dv.dv_swap_in(host_c, 0, dev_c, 0, 0, 1, z, lens(1, 32), check=False) == U
    # just below the limit the sizing still works: 31 tokens in the later group
    assert dv.dv_packed_bytes(dense(L=1, H=H, D=8, B=B, S=64), 0, 1, z, lens(1, 31)) > 0

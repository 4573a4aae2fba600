"""Pins of the CPU oracle against numpy primitives and invariants (no GPU).

The oracle copies bytes, so its results are exact; what can be wrong is an
address: a dropped term, a swapped index, K and V exchanged, the ragged
prefix ignored, the block table or the split key not followed.  Each test
below fixes the oracle to something other than its own formulas:

* numpy boolean-mask selection in C order (the wire is the selected elements
  sorted by layer, K|V, sequence, head, token, dim), for dense, paged (via
  fancy indexing) and split-key (via reshape/transpose) layouts;
* address decode by brute force: with every element holding its own storage
  index, each wire element names its source;
* the streaming invariants: stream-out then stream-in reproduces the cache;
  N increments after the prompt equal one full stream; a paged cache with an
  identity table gathers to the dense bytes; layer ranges concatenate;
* all 65536 16-bit codes (NaN payloads, infinities, subnormals, -0) survive;
* the swap copy equals numpy slice assignment.

``test_planted_mistakes_are_caught`` builds the oracle with known mistakes
planted and checks that these pins fail for every one of them.
"""

import numpy as np
import pytest

import oracle
import synth
from tests import refs


def rng(seed):
    return np.random.default_rng(seed)


def rand_shape(r, paged=False):
    L = int(r.integers(1, 4))
    H = int(r.integers(1, 5))
    E = int(r.choice([1, 2, 4]))
    D = int(r.choice([16, 32, 48, 64])) // E * E if E < 4 else int(r.choice([4, 8, 12]))
    D = max(D, 16 // E)
    D = D - D % (16 // E)
    B = int(r.integers(1, 6))
    S = int(r.integers(1, 40))
    return L, H, D, B, S, E


def rand_ranges(r, B, cap):
    t0 = np.zeros(B, np.int32)
    t1 = np.zeros(B, np.int32)
    for b in range(B):
        a, c = sorted(int(v) for v in r.integers(0, cap + 1, size=2))
        if r.random() < 0.2:
            c = a  # empty range
        t0[b], t1[b] = a, c
    return t0, t1


def dense_case(seed):
    r = rng(seed)
    L, H, D, B, S, E = rand_shape(r)
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    buf = synth.fill_bytes(lay.storage_bytes(), seed)
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0, L + 1))
    t0, t1 = rand_ranges(r, B, S)
    return lay, buf, (L, B, H, S, D, E), l0, l1, t0, t1


def paged_case(seed, identity=False):
    r = rng(seed)
    L, H, D, B, _, E = rand_shape(r)
    bs = int(r.choice([1, 2, 4, 8]))
    cap_tok = [int(r.integers(0, 30)) for _ in range(B)]
    maxb = max(1, max((c + bs - 1) // bs for c in cap_tok) + int(r.integers(0, 3)))
    if identity:
        bt = np.arange(B * maxb, dtype=np.int32).reshape(B, maxb)
        nb = B * maxb
    else:
        bt, nb = synth.make_paged_tables(seed, cap_tok, bs, maxb)
        nb = max(nb, 1)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    t0 = np.zeros(B, np.int32)
    t1 = np.zeros(B, np.int32)
    for b in range(B):
        hi = cap_tok[b] if not identity else maxb * bs
        a, c = sorted(int(v) for v in r.integers(0, hi + 1, size=2))
        t0[b], t1[b] = a, c
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0, L + 1))
    return lay, bt, nb, bs, maxb, (L, B, H, D, E), l0, l1, t0, t1


# ---------------------------------------------------------------------------
# dense layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(40))
def test_dense_pack_is_mask_selection(oracle_lib, seed):
    lay, buf, shp, l0, l1, t0, t1 = dense_case(seed)
    got = oracle_lib.pack(lay, buf, l0, l1, t0, t1)
    exp = refs.pack_dense(buf, *shp, l0, l1, t0, t1)
    assert got.tobytes() == exp.tobytes()


@pytest.mark.parametrize("seed", range(12))
def test_address_decode_brute_force(oracle_lib, seed):
    """Every element holds its own storage index; the wire names its sources."""
    r = rng(1000 + seed)
    L, H, B, S = (int(r.integers(1, 4)), int(r.integers(1, 5)), int(r.integers(1, 5)),
                  int(r.integers(1, 24)))
    D = int(r.choice([4, 8, 12]))
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=4)
    idx = np.arange(lay.storage_elems(), dtype=np.uint32)
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0, L + 1))
    t0, t1 = rand_ranges(r, B, S)
    wire = oracle_lib.pack(lay, idx.view(np.uint8), l0, l1, t0, t1).view(np.uint32)
    mask = refs.range_mask(L, B, H, S, D, l0, l1, t0, t1)
    # the wire is exactly the selected storage indices, ascending
    assert np.array_equal(wire, np.flatnonzero(mask.reshape(-1)))
    # and the oracle's inverse map agrees element by element
    back = oracle_lib.wire_to_storage(lay, l0, l1, t0, t1, np.arange(wire.size))
    assert np.array_equal(back, wire.astype(np.int64))
    # coordinates decoded from a wire value are inside the requested ranges
    for w in wire[:: max(1, wire.size // 50)]:
        l, kv, b, h, s, d = np.unravel_index(int(w), (L, 2, B, H, S, D))
        assert l0 <= l < l1 and t0[b] <= s < t1[b]


@pytest.mark.parametrize("kind", [oracle.DENSE, oracle.PAGED, oracle.KSPLIT])
@pytest.mark.parametrize("seed", range(6))
def test_inverse_map_names_each_wire_source(oracle_lib, kind, seed):
    """The inverse map the full-size GPU tests sample with, for every layout:
    pack a cache whose every 4-byte element holds its own storage index and
    the wire lists the sources; wire_to_storage must return the same list.
    Sources are distinct and each lies in the (layer, sequence) ranges."""
    r = rng(1300 + seed)
    L, H, B = int(r.integers(1, 4)), int(r.integers(1, 5)), int(r.integers(1, 6))
    D = int(r.choice([4, 8, 12]))  # 4-byte elements: 16-byte groups of 4
    if kind == oracle.PAGED:
        bs = int(r.choice([1, 3, 4]))
        lens = [int(r.integers(0, 20)) for _ in range(B)]
        maxb = max(1, max((n + bs - 1) // bs for n in lens)) + 1
        bt, nb = synth.make_paged_tables(seed, lens, bs, maxb)
        lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=4, block_size=bs,
                            num_blocks=max(nb, 1), block_table=bt)
        cap = lens
    else:
        S = int(r.integers(1, 24))
        lay = oracle.Layout(kind, L, H, D, B, seq_cap=S, elem_bytes=4)
        cap = [S] * B
    t0 = np.zeros(B, np.int32)
    t1 = np.zeros(B, np.int32)
    for b in range(B):
        a, e = sorted(int(v) for v in r.integers(0, cap[b] + 1, size=2))
        t0[b], t1[b] = a, e
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0, L + 1))
    idx = np.arange(lay.storage_elems(), dtype=np.uint32)
    wire = oracle_lib.pack(lay, idx.view(np.uint8), l0, l1, t0, t1).view(np.uint32)
    back = oracle_lib.wire_to_storage(lay, l0, l1, t0, t1, np.arange(wire.size))
    assert np.array_equal(back, wire.astype(np.int64))
    assert np.unique(wire).size == wire.size
    assert wire.size == (l1 - l0) * 2 * H * D * int((t1 - t0).sum())


@pytest.mark.parametrize("seed", range(20))
def test_unpack_writes_only_the_ranges(oracle_lib, seed):
    lay, buf, shp, l0, l1, t0, t1 = dense_case(100 + seed)
    n = oracle_lib.wire_elems(lay, l0, l1, t0, t1) * lay.elem_bytes
    wire = synth.fill_bytes(n, 7 + seed)
    sentinel = np.full(lay.storage_bytes(), 0xA5, dtype=np.uint8)
    got = sentinel.copy()
    oracle_lib.unpack(lay, got, l0, l1, t0, t1, wire)
    exp = refs.unpack_dense(sentinel, *shp, l0, l1, t0, t1, wire)
    assert got.tobytes() == exp.tobytes()


@pytest.mark.parametrize("seed", range(20))
def test_round_trip_reproduces_cache(oracle_lib, seed):
    """Invariant 1: stream-out then stream-in into an empty cache."""
    lay, buf, shp, l0, l1, t0, t1 = dense_case(200 + seed)
    wire = oracle_lib.pack(lay, buf, l0, l1, t0, t1)
    recv = np.zeros_like(buf)
    oracle_lib.unpack(lay, recv, l0, l1, t0, t1, wire)
    L, B, H, S, D, E = shp
    m = refs.range_mask(L, B, H, S, D, l0, l1, t0, t1)
    x = refs.dense_view(buf, *shp)
    y = refs.dense_view(recv, *shp)
    assert np.array_equal(y[m], x[m])
    assert not y[~m].any()


def test_tiny_workload_round_trip_and_increments(oracle_lib):
    """Workload 0: prompt 100 for both sequences, 16 increments, empty receiver."""
    w = synth.make_workload(0)
    lay = oracle.Layout(oracle.DENSE, w.layers, w.heads, w.head_dim, w.batch,
                        seq_cap=w.max_seq, elem_bytes=w.elem_bytes)
    full_hi = (w.lens + w.steps).astype(np.int32)
    zero = np.zeros(w.batch, np.int32)
    # sender: zero cache with the positions [0, len + steps) filled
    sender = np.zeros(lay.storage_bytes(), np.uint8)
    src = synth.fill_bytes(lay.storage_bytes(), w.data_seed)
    oracle_lib.unpack(lay, sender, 0, w.layers, zero, full_hi,
                      oracle_lib.pack(lay, src, 0, w.layers, zero, full_hi))
    recv = np.zeros_like(sender)
    t0, t1 = w.prompt_ranges()
    wire = oracle_lib.pack(lay, sender, 0, w.layers, t0, t1)
    assert wire.nbytes == 409600
    oracle_lib.unpack(lay, recv, 0, w.layers, t0, t1, wire)
    for i in range(w.steps):
        p = w.step_positions(i)
        inc = oracle_lib.pack(lay, sender, 0, w.layers, p, p + 1)
        assert inc.nbytes == 4096
        oracle_lib.unpack(lay, recv, 0, w.layers, p, p + 1, inc)
    assert recv.tobytes() == sender.tobytes()


@pytest.mark.parametrize("seed", range(10))
def test_increments_equal_full_stream(oracle_lib, seed):
    """Invariant 2: prompt + N single-token increments == one stream of len+N."""
    r = rng(300 + seed)
    L, H, D, B, S, E = rand_shape(r)
    S = max(S, 8)
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    buf = synth.fill_bytes(lay.storage_bytes(), seed)
    nsteps = int(r.integers(1, 6))
    lens = r.integers(0, S - nsteps + 1, size=B).astype(np.int32)
    zero = np.zeros(B, np.int32)
    a = np.zeros_like(buf)
    oracle_lib.unpack(lay, a, 0, L, zero, lens, oracle_lib.pack(lay, buf, 0, L, zero, lens))
    for i in range(nsteps):
        p = lens + i
        oracle_lib.unpack(lay, a, 0, L, p, p + 1, oracle_lib.pack(lay, buf, 0, L, p, p + 1))
    b = np.zeros_like(buf)
    hi = lens + nsteps
    oracle_lib.unpack(lay, b, 0, L, zero, hi, oracle_lib.pack(lay, buf, 0, L, zero, hi))
    assert a.tobytes() == b.tobytes()


@pytest.mark.parametrize("seed", range(10))
def test_layer_ranges_concatenate(oracle_lib, seed):
    lay, buf, shp, _, _, t0, t1 = dense_case(400 + seed)
    L = shp[0]
    m = int(rng(seed).integers(0, L + 1))
    whole = oracle_lib.pack(lay, buf, 0, L, t0, t1)
    parts = np.concatenate([oracle_lib.pack(lay, buf, 0, m, t0, t1),
                            oracle_lib.pack(lay, buf, m, L, t0, t1)])
    assert whole.tobytes() == parts.tobytes()


@pytest.mark.parametrize("seed", range(10))
def test_sequences_concatenate_inside_each_slab(oracle_lib, seed):
    """Within one (layer, K|V) slab, sequence b's tokens follow sequence b-1's."""
    lay, buf, shp, l0, l1, t0, t1 = dense_case(450 + seed)
    L, B, H, S, D, E = shp
    whole = oracle_lib.pack(lay, buf, l0, l1, t0, t1)
    pieces = []
    for b in range(B):
        z0, z1 = np.zeros(B, np.int32), np.zeros(B, np.int32)
        z0[b], z1[b] = t0[b], t1[b]
        pieces.append(oracle_lib.pack(lay, buf, l0, l1, z0, z1).reshape(max(l1 - l0, 0) * 2, -1)
                      if l1 > l0 else np.zeros((0, 0), np.uint8))
    if l1 > l0:
        slabs = np.concatenate(pieces, axis=1).reshape(-1)
        assert whole.tobytes() == slabs.tobytes()
    else:
        assert whole.size == 0


@pytest.mark.parametrize("seed", range(10))
def test_size_formula(oracle_lib, seed):
    lay, buf, shp, l0, l1, t0, t1 = dense_case(500 + seed)
    L, B, H, S, D, E = shp
    n = oracle_lib.wire_elems(lay, l0, l1, t0, t1)
    assert n == (l1 - l0) * 2 * H * D * int(np.sum(t1 - t0))
    assert n == int(refs.range_mask(L, B, H, S, D, l0, l1, t0, t1).sum())


def test_all_16bit_codes_round_trip(oracle_lib):
    """Element i holds code i mod 65536: NaN payloads, Inf, subnormal, -0."""
    L, H, D, B, S = 2, 4, 64, 2, 128
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=2)
    codes = (np.arange(lay.storage_elems()) % 65536).astype(np.uint16)
    t0 = np.zeros(B, np.int32)
    t1 = np.full(B, S, np.int32)
    wire = oracle_lib.pack(lay, codes.view(np.uint8), 0, L, t0, t1)
    assert np.array_equal(np.sort(np.unique(wire.view(np.uint16))), np.arange(65536))
    back = np.zeros(lay.storage_bytes(), np.uint8)
    oracle_lib.unpack(lay, back, 0, L, t0, t1, wire)
    assert back.tobytes() == codes.view(np.uint8).tobytes()


# ---------------------------------------------------------------------------
# paged layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(30))
def test_paged_pack_is_mask_selection(oracle_lib, seed):
    lay, bt, nb, bs, maxb, (L, B, H, D, E), l0, l1, t0, t1 = paged_case(600 + seed)
    pool = synth.fill_bytes(lay.storage_bytes(), seed)
    scap = maxb * bs
    x = refs.paged_logical(pool, L, nb, H, bs, D, E, bt, scap)
    m = refs.range_mask(L, B, H, scap, D, l0, l1, t0, t1)
    got = oracle_lib.pack(lay, pool, l0, l1, t0, t1)
    assert got.tobytes() == x[m].view(np.uint8).tobytes()


@pytest.mark.parametrize("seed", range(10))
def test_paged_identity_table_matches_dense(oracle_lib, seed):
    """Invariant 3: identity block table gathers the dense bytes."""
    lay, bt, nb, bs, maxb, (L, B, H, D, E), l0, l1, t0, t1 = paged_case(700 + seed, True)
    S = maxb * bs
    dense = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    dbuf = synth.fill_bytes(dense.storage_bytes(), seed)
    x = refs.dense_view(dbuf, L, B, H, S, D, E)
    pool = refs.pool_from_logical(x, (L, nb, H, D), bt, bs, E)
    got = oracle_lib.pack(lay, pool, l0, l1, t0, t1)
    exp = oracle_lib.pack(dense, dbuf, l0, l1, t0, t1)
    assert got.tobytes() == exp.tobytes()


@pytest.mark.parametrize("seed", range(10))
def test_paged_scatter_to_fresh_permutation(oracle_lib, seed):
    """Gather with table A, scatter into table B, gather again: same wire;
    pool bytes outside the ranges keep their sentinel."""
    lay, bt, nb, bs, maxb, (L, B, H, D, E), l0, l1, t0, t1 = paged_case(800 + seed)
    pool = synth.fill_bytes(lay.storage_bytes(), seed)
    wire = oracle_lib.pack(lay, pool, l0, l1, t0, t1)
    bt_b = bt.copy()
    valid = bt >= 0
    bt_b[valid] = np.random.default_rng(seed).permutation(bt[valid])
    lay_b = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                          num_blocks=nb, block_table=bt_b)
    recv = np.full(lay_b.storage_bytes(), 0x3C, np.uint8)
    oracle_lib.unpack(lay_b, recv, l0, l1, t0, t1, wire)
    assert oracle_lib.pack(lay_b, recv, l0, l1, t0, t1).tobytes() == wire.tobytes()
    scap = maxb * bs
    m = refs.range_mask(L, B, H, scap, D, l0, l1, t0, t1)
    sent = np.full(lay_b.storage_bytes(), 0x3C, np.uint8)
    exp_logical = refs.paged_logical(sent, L, nb, H, bs, D, E, bt_b, scap)
    exp_logical[m] = wire.view(refs.DT[E])
    # expected pool: sentinel, with each streamed token written through table B
    p = sent.view(refs.DT[E]).reshape(L, 2, nb, H, bs, D)
    for b in range(B):
        sel = np.arange(t0[b], t1[b])
        if sel.size == 0 or l1 == l0:
            continue
        p[l0:l1, :, bt_b[b, sel // bs], :, sel % bs, :] = exp_logical[l0:l1, :, b, :, sel, :]
    assert recv.tobytes() == sent.tobytes()


def test_paged_rejects_invalid_table_entries(oracle_lib):
    bt = np.array([[0, -1], [1, 5]], np.int32)
    lay = oracle.Layout(oracle.PAGED, 1, 1, 8, 2, elem_bytes=2, block_size=4, num_blocks=2,
                        block_table=bt)
    assert oracle_lib.check(lay, 0, 1, [0, 0], [4, 4]) == oracle.OK
    assert oracle_lib.check(lay, 0, 1, [0, 0], [5, 4]) == oracle.RANGE
    assert oracle_lib.check(lay, 0, 1, [0, 4], [4, 5]) == oracle.RANGE
    assert oracle_lib.check(lay, 0, 1, [0, 0], [4, 9]) == oracle.RANGE


# ---------------------------------------------------------------------------
# split-key layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(20))
def test_ksplit_pack_matches_dense(oracle_lib, seed):
    lay, buf, shp, l0, l1, t0, t1 = dense_case(900 + seed)
    L, B, H, S, D, E = shp
    ks = oracle.Layout(oracle.KSPLIT, L, H, D, B, seq_cap=S, elem_bytes=E)
    kbuf = refs.ksplit_from_dense(buf, *shp)
    assert oracle_lib.pack(ks, kbuf, l0, l1, t0, t1).tobytes() == \
        refs.pack_dense(buf, *shp, l0, l1, t0, t1).tobytes()
    # and unpack into a split-key receiver equals the dense unpack, re-split
    wire = synth.fill_bytes(oracle_lib.wire_elems(ks, l0, l1, t0, t1) * E, seed)
    recv = np.zeros(ks.storage_bytes(), np.uint8)
    oracle_lib.unpack(ks, recv, l0, l1, t0, t1, wire)
    exp = refs.unpack_dense(np.zeros_like(buf), *shp, l0, l1, t0, t1, wire)
    assert refs.ksplit_to_dense(recv, *shp).tobytes() == exp.tobytes()


# ---------------------------------------------------------------------------
# swap copy and validation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(15))
def test_copy_ranges_is_slice_assignment(oracle_lib, seed):
    r = rng(1100 + seed)
    L, H, D, B, S, E = rand_shape(r)
    S2 = S + int(r.integers(0, 5))
    a = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S, elem_bytes=E)
    c = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S2, elem_bytes=E)
    src = synth.fill_bytes(a.storage_bytes(), seed)
    dst = np.full(c.storage_bytes(), 0x77, np.uint8)
    exp = dst.copy()
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0, L + 1))
    t0, t1 = rand_ranges(r, B, S)
    oracle_lib.copy_ranges(a, src, c, dst, l0, l1, t0, t1)
    xs = refs.dense_view(src, L, B, H, S, D, E)
    xd = refs.dense_view(exp, L, B, H, S2, D, E)
    for b in range(B):
        xd[l0:l1, :, b, :, t0[b]:t1[b], :] = xs[l0:l1, :, b, :, t0[b]:t1[b], :]
    assert dst.tobytes() == exp.tobytes()
    # swap-in after swap-out is the identity on the ranges
    back = np.zeros_like(src)
    oracle_lib.copy_ranges(c, dst, a, back, l0, l1, t0, t1)
    m = refs.range_mask(L, B, H, S, D, l0, l1, t0, t1)
    assert np.array_equal(refs.dense_view(back, L, B, H, S, D, E)[m], xs[m])


def test_check_rejects_bad_ranges(oracle_lib):
    lay = oracle.Layout(oracle.DENSE, 2, 2, 8, 2, seq_cap=10, elem_bytes=2)
    assert oracle_lib.check(lay, 0, 2, [0, 0], [10, 10]) == oracle.OK
    assert oracle_lib.check(lay, 0, 2, [0, 0], [11, 10]) == oracle.RANGE
    assert oracle_lib.check(lay, 0, 2, [3, 0], [2, 10]) == oracle.RANGE
    assert oracle_lib.check(lay, 0, 2, [-1, 0], [2, 10]) == oracle.RANGE
    assert oracle_lib.check(lay, 1, 0, [0, 0], [1, 1]) == oracle.RANGE
    assert oracle_lib.check(lay, 0, 3, [0, 0], [1, 1]) == oracle.RANGE
    bad = oracle.Layout(oracle.KSPLIT, 2, 2, 12, 2, seq_cap=10, elem_bytes=2)
    assert oracle_lib.check(bad, 0, 2, [0, 0], [1, 1]) == oracle.INVALID


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

def _pins_pass(orc) -> bool:
    """The mask-selection pins over dense, ragged, paged and split-key cases."""
    try:
        # a fixed case with every extent above one, then random ones
        fixed = oracle.Layout(oracle.DENSE, 2, 3, 8, 4, seq_cap=9, elem_bytes=2)
        fbuf = synth.fill_bytes(fixed.storage_bytes(), 99)
        ft0 = np.array([0, 2, 1, 0], np.int32)
        ft1 = np.array([9, 5, 7, 3], np.int32)
        cases = [(fixed, fbuf, (2, 4, 3, 9, 8, 2), 0, 2, ft0, ft1)]
        cases += [dense_case(seed) for seed in range(6)]
        for lay, buf, shp, l0, l1, t0, t1 in cases:
            if orc.pack(lay, buf, l0, l1, t0, t1).tobytes() != \
                    refs.pack_dense(buf, *shp, l0, l1, t0, t1).tobytes():
                return False
            L, B, H, S, D, E = shp
            ks = oracle.Layout(oracle.KSPLIT, L, H, D, B, seq_cap=S, elem_bytes=E)
            if orc.pack(ks, refs.ksplit_from_dense(buf, *shp), l0, l1, t0, t1).tobytes() != \
                    refs.pack_dense(buf, *shp, l0, l1, t0, t1).tobytes():
                return False
        for seed in range(6):
            lay, bt, nb, bs, maxb, (L, B, H, D, E), l0, l1, t0, t1 = paged_case(600 + seed)
            pool = synth.fill_bytes(lay.storage_bytes(), seed)
            x = refs.paged_logical(pool, L, nb, H, bs, D, E, bt, maxb * bs)
            m = refs.range_mask(L, B, H, maxb * bs, D, l0, l1, t0, t1)
            if orc.pack(lay, pool, l0, l1, t0, t1).tobytes() != x[m].view(np.uint8).tobytes():
                return False
    except (ValueError, AssertionError):
        return False
    return True


@pytest.mark.parametrize("mutant", [1, 2, 3, 4, 5, 6])
def test_planted_mistakes_are_caught(tmp_path, mutant, oracle_lib):
    assert _pins_pass(oracle_lib)
    path = oracle.build(str(tmp_path / f"libdvoracle_m{mutant}.so"), mutant=mutant)
    assert not _pins_pass(oracle.Oracle(path)), f"planted mistake {mutant} not caught"

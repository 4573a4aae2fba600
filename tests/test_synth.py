"""The seeded input generators (host side)."""
import numpy as np

import synth


def test_splitmix64_known_answers():
    # First outputs of SplitMix64 started at state 0, as published with the
    # xoshiro/xoroshiro reference seeding code.
    g = synth.SplitMix64(0)
    assert [g.next() for _ in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                            0x06C45D188009454F]


def test_counter_mode_equals_stream():
    seed = 0x1234_5678_9ABC_DEF0
    g = synth.SplitMix64(seed)
    stream = np.array([g.next() for _ in range(64)], dtype=np.uint64)
    assert np.array_equal(synth.words_u64(seed, 0, 64), stream)
    assert np.array_equal(synth.words_u64(seed, 10, 5), stream[10:15])
    raw = synth.fill_bytes(64 * 8, seed)
    assert np.array_equal(raw.view(np.uint64), stream)
    assert np.array_equal(synth.fill_bytes(40, seed, first_byte=24), raw[24:64])


def test_bytes_at_matches_fill():
    seed = 77
    raw = synth.fill_bytes(4096, seed)
    for width, dt in [(1, np.uint8), (2, np.uint16), (4, np.uint32), (8, np.uint64)]:
        idx = np.arange(0, 4096, width * 3)
        got = synth.bytes_at(seed, idx, width).astype(dt)
        assert np.array_equal(got, raw.view(dt)[idx // width])


def test_workloads_shapes_and_lengths():
    w0 = synth.make_workload(0)
    assert (w0.layers, w0.heads, w0.head_dim, w0.batch, w0.max_seq) == (2, 4, 64, 2, 128)
    assert list(w0.lens) == [100, 100] and w0.steps == 16
    w1 = synth.make_workload(1)
    assert w1.lens.min() >= 512 and w1.lens.max() <= 1024 and len(w1.lens) == 8
    w3 = synth.make_workload(3)
    assert w3.lens.min() >= 64 and w3.lens.max() <= 2048 and len(w3.lens) == 16
    w4 = synth.make_workload(4)
    assert w4.paged and w4.block_size == 16 and len(w4.lens) == 32
    for bt in (w4.block_table_a, w4.block_table_b):
        used = bt[bt >= 0]
        # each table is a permutation of the whole pool
        assert np.array_equal(np.sort(used), np.arange(w4.num_blocks))
        for b in range(w4.batch):
            nb = (int(w4.lens[b]) + w4.steps + 15) // 16
            assert (bt[b, :nb] >= 0).all() and (bt[b, nb:] == -1).all()
    assert not np.array_equal(w4.block_table_a, w4.block_table_b)
    # deterministic from the seed
    assert np.array_equal(synth.make_workload(4).block_table_a, w4.block_table_a)


def test_host_c_fill_equals_numpy_definition():
    synth.build_host()
    for n, first in [(1, 0), (7, 3), (4096, 0), (1000, 13), (65536 + 5, 1 << 35)]:
        assert synth.fill_bytes(n, 99, first).tobytes() == \
            synth.fill_bytes_numpy(n, 99, first).tobytes()

"""The background streamer: layer-by-layer prompt streaming and token
streaming overlapped with the compute stream (checked against the oracle)."""
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


@pytest.mark.parametrize("case", ["ragged", "uniform", "short"])
def test_layer_by_layer_prompt_to_host(oracle_lib, case):
    """Each layer is written by the compute stream just before it is pushed;
    the host buffer ends up holding the whole prompt's contiguous buffer.
    Runs of 64 KB or more go by the DMA engines straight from the cache (one
    pitched copy per layer slab and sequence, or one per layer when every
    sequence has the same range); shorter ones through the pack kernel and
    the staging buffer."""
    L, H, D, B, S = 6, 3, 128, 4, 300
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    cache = G.dev_const(lay.storage_bytes(), 0xA5)  # not yet computed
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    lens = {"ragged": np.array([300, 17, 0, 129], np.int32),
            "uniform": np.full(B, 280, np.int32),
            "short": np.array([100, 17, 0, 129], np.int32)}[case]
    zero = np.zeros(B, np.int32)
    total = dv.dv_packed_bytes(c, 0, L, zero, lens)
    staging = G.dev_const(total, 0)
    host = torch.full((total,), 0x11, dtype=torch.uint8, pin_memory=True)
    layer_wires = [synth.fill_bytes(dv.dv_packed_bytes(c, l, l + 1, zero, lens), 10 + l)
                   for l in range(L)]
    if case == "ragged":
        # through staging a host destination is written in 256 KiB rows plus
        # a remainder; these layers would be two whole rows and a tail
        assert all(w.size // (256 << 10) == 2 and w.size % (256 << 10) for w in layer_wires)
    dev_wires = [G.to_dev(wl) for wl in layer_wires]
    torch.cuda.synchronize()
    compute = torch.cuda.Stream()
    s = dv.Streamer(c, 0, staging, total, host.data_ptr(), total)
    off = 0
    with torch.cuda.stream(compute):
        for l in range(L):
            # "compute" layer l: a long spin, then the layer's K/V land in the cache
            torch.cuda._sleep(2_000_000)
            dv.dv_stream_in(c, 0, l, l + 1, zero, lens, dev_wires[l], dev_wires[l].numel(),
                            compute)
            off += s.push(l, l + 1, zero, lens, off, stream=compute)
    assert off == total
    s.flush()
    s.close()
    torch.cuda.synchronize()
    # expected: the cache after all layers, packed whole
    exp_cache = np.full(lay.storage_bytes(), 0xA5, np.uint8)
    for l in range(L):
        oracle_lib.unpack(lay, exp_cache, l, l + 1, zero, lens, layer_wires[l])
    exp = oracle_lib.pack(lay, exp_cache, 0, L, zero, lens)
    assert host.numpy().tobytes() == exp.tobytes()


def test_token_streaming_many_steps(oracle_lib):
    """100 decode steps (more than the streamer's 64 events), each token
    written by the compute stream and pushed to its own slot."""
    L, H, D, B, S = 2, 2, 64, 3, 160
    lay = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S)
    host_cache = synth.fill_bytes(lay.storage_bytes(), 3)
    cache = G.to_dev(host_cache)
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    steps = 100
    base = np.array([10, 30, 50], np.int32)
    inc = dv.dv_packed_bytes(c, 0, L, base, base + 1)
    staging = G.dev_const(inc * 4, 0)  # 4 slots, reused
    host = torch.zeros(inc * steps, dtype=torch.uint8, pin_memory=True)
    tok_wires = [synth.fill_bytes(inc, 100 + i) for i in range(steps)]
    dev_tok = [G.to_dev(t) for t in tok_wires]
    torch.cuda.synchronize()
    compute = torch.cuda.Stream()
    s = dv.Streamer(c, 0, staging, inc * 4, host.data_ptr(), inc * steps)
    with torch.cuda.stream(compute):
        for i in range(steps):
            p = base + i
            dv.dv_stream_in(c, 0, 0, L, p, p + 1, dev_tok[i], inc, compute)
            # staging slot i % 4, destination slot i
            assert s.push(0, L, p, p + 1, (i % 4) * inc, i * inc, stream=compute) == inc
    s.flush()
    s.close()
    torch.cuda.synchronize()
    h = host.numpy()
    for i in range(steps):
        assert h[i * inc:(i + 1) * inc].tobytes() == tok_wires[i].tobytes(), i


def test_paged_source_layer_by_layer_and_from_two_threads(oracle_lib):
    """A paged source cache (random block table) streamed layer by layer into
    device memory, the layers pushed from two host threads at once (each
    layer to its own offset), then each sequence's next token; every byte
    equals the oracle's pack."""
    import threading
    L, H, D, B, bs = 6, 4, 128, 5, 16
    lens = [70, 3, 0, 48, 129]
    maxb = max((n + 1 + bs - 1) // bs for n in lens) + 1
    bt, nb = synth.make_paged_tables(61, [n + 1 for n in lens], bs, maxb)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, block_size=bs, num_blocks=nb, block_table=bt)
    host_pool = synth.fill_bytes(lay.storage_bytes(), 62)
    pool = G.to_dev(host_pool)
    btd = G.to_dev(bt)
    c = dv.Cache(dv.DV_PAGED, L, H, D, B, [pool], block_size=bs, num_blocks=nb,
                 max_blocks=maxb, block_tables=[btd])
    zero = np.zeros(B, np.int32)
    t1 = np.array(lens, np.int32)
    per_layer = [dv.dv_packed_bytes(c, l, l + 1, zero, t1) for l in range(L)]
    offs = np.concatenate([[0], np.cumsum(per_layer)]).astype(np.int64)
    inc = dv.dv_packed_bytes(c, 0, L, t1, t1 + 1)
    total = int(offs[-1]) + inc
    staging = G.dev_const(total, 0)
    dst = G.dev_const(total, 0x11)
    s = dv.Streamer(c, 0, staging, total, dst, total)
    errors = []

    def push_layers(layers):
        try:
            for l in layers:
                s.push(l, l + 1, zero, t1, int(offs[l]))
        except Exception as e:  # surfaced below
            errors.append(e)

    threads = [threading.Thread(target=push_layers, args=(range(k, L, 2),)) for k in (0, 1)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    assert s.push(0, L, t1, t1 + 1, int(offs[-1])) == inc
    assert s.flush() == dv.DV_OK
    s.close()
    torch.cuda.synchronize()
    got = G.host(dst)
    for l in range(L):
        exp = oracle_lib.pack(lay, host_pool, l, l + 1, zero, t1)
        assert got[offs[l]:offs[l + 1]].tobytes() == exp.tobytes(), l
    exp = oracle_lib.pack(lay, host_pool, 0, L, t1, t1 + 1)
    assert got[offs[-1]:].tobytes() == exp.tobytes()


def test_streamer_errors_surface():
    L, H, D, B, S = 1, 1, 64, 2, 16
    cache = G.dev_const(L * 2 * B * H * S * D * 2, 0)
    c = dv.Cache(dv.DV_DENSE, L, H, D, B, [cache], max_seq=S)
    staging = G.dev_const(4096, 0)
    dst = G.dev_const(4096, 0)
    s = dv.Streamer(c, 0, staging, 4096, dst, 4096)
    rc, n = s.push(0, 1, [0, 0], [17, 0], 0, check=False)
    assert rc == dv.DV_ERR_RANGE
    rc, n = s.push(0, 1, [0, 0], [16, 16], 0, check=False)
    assert rc == dv.DV_ERR_SPACE and n == 2 * 2 * 16 * 64 * 2
    rc, n = s.push(0, 1, [0, 0], [1, 1], 8, check=False)
    assert rc == dv.DV_ERR_INVALID  # unaligned offset
    rc, n = s.push(0, 1, [0, 0], [1, 1], 0, 4096, check=False)
    assert rc == dv.DV_ERR_SPACE  # destination offset past the end
    # a compute stream under graph capture is refused and the capture goes on
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            cache.add_(1)
            rc, n = s.push(0, 1, [0, 0], [1, 1], 0, stream=torch.cuda.current_stream(),
                           check=False)
            cache.add_(1)
    assert rc == dv.DV_ERR_INVALID
    g.replay()
    torch.cuda.synchronize()
    assert int(cache[0]) == 2  # the capture holds both adds
    assert s.flush() == dv.DV_OK
    # after the refusals the streamer still works
    assert s.push(0, 1, [0, 0], [1, 1], 0) == 2 * 2 * 64 * 2
    assert s.flush() == dv.DV_OK
    torch.cuda.synchronize()
    exp = torch.cat([cache[0:128], cache[16 * 128:17 * 128], cache[2 * 16 * 128:2 * 16 * 128 + 128],
                     cache[3 * 16 * 128:3 * 16 * 128 + 128]])
    assert torch.equal(dst[:512], exp)
    s.close()

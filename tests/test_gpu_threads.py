"""Calls from several host threads at once, each thread on a stream of its own.

The header allows calls from several host threads; calls on different
streams that touch different bytes must not disturb each other.  Each thread
repeats a pack and an unpack of its own cache into its own wire and
receiver -- a dense cache, a paged pool scattered through an owner-map
workspace, a split-key cache, decode-step increments of a paged pool -- all
threads released together by a barrier, so their launches interleave on the
GPU (ctypes drops the GIL for the duration of each call).  Afterwards every
wire and every receiver equals the oracle's.
"""
import threading

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

ITERS = 12


def dense_job(seed, kind):
    """A dense or split-key cache with ragged prompt ranges."""
    r = np.random.default_rng(seed)
    L, H, D, B, S, E = 3, 8, 128, 12, 600, 2
    okind, dkind = (oracle.DENSE, dv.DV_DENSE) if kind == "dense" else \
        (oracle.KSPLIT, dv.DV_DENSE_KSPLIT)
    lay = oracle.Layout(okind, L, H, D, B, seq_cap=S, elem_bytes=E)
    host_cache = synth.fill_bytes(lay.storage_bytes(), seed)
    t0 = r.integers(0, 100, size=B).astype(np.int32)
    t1 = np.minimum(t0 + r.integers(0, 500, size=B), S).astype(np.int32)
    src = dv.Cache(dkind, L, H, D, B, [G.to_dev(host_cache)], max_seq=S, elem_bytes=E)
    recv = G.dev_const(lay.storage_bytes(), 0xA5)
    dst = dv.Cache(dkind, L, H, D, B, [recv], max_seq=S, elem_bytes=E)
    return dict(lay=lay, host=host_cache, src=src, dst=dst, recv=recv, l0=0, l1=L,
                t0=t0, t1=t1, token=False)


def paged_job(seed, token):
    """A paged pool: whole prompts scattered through a workspace (pool
    order), or one decode-step token per sequence."""
    r = np.random.default_rng(seed)
    L, H, D, B, E, bs = 2, 8, 128, 16, 2, 16
    lens = [int(r.integers(200, 700)) for _ in range(B)]
    maxb = max((n + bs - 1) // bs for n in lens) + 1
    bt, nb = synth.make_paged_tables(seed, lens, bs, maxb)
    lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                        block_table=bt)
    host_pool = synth.fill_bytes(lay.storage_bytes(), seed)
    valid = bt >= 0
    bt_b = bt.copy()
    bt_b[valid] = r.permutation(bt[valid])
    lay_b = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs, num_blocks=nb,
                          block_table=bt_b)
    kw = dict(elem_bytes=E, block_size=bs, num_blocks=nb, max_blocks=maxb)
    src = dv.Cache(dv.DV_PAGED, L, H, D, B, [G.to_dev(host_pool)], block_tables=[G.to_dev(bt)],
                   **kw)
    recv = G.dev_const(lay_b.storage_bytes(), 0xA5)
    ws = G.dev_const(nb * 4, 0)
    dst = dv.Cache(dv.DV_PAGED, L, H, D, B, [recv], block_tables=[G.to_dev(bt_b)],
                   block_owners=[ws], **kw)
    if token:
        t0 = np.array([n - 1 for n in lens], np.int32)
        t0[r.random(B) < 0.25] = -1  # inactive sequences
        t1 = np.where(t0 >= 0, t0 + 1, 0).astype(np.int32)
        t0 = np.maximum(t0, 0).astype(np.int32)
    else:
        t0 = np.zeros(B, np.int32)
        t1 = np.array(lens, np.int32)
    return dict(lay=lay, host=host_pool, src=src, dst=dst, recv=recv, l0=0, l1=L, t0=t0,
                t1=t1, token=token, lay_b=lay_b, ws=ws)


def test_concurrent_host_threads(oracle_lib):
    jobs = [dense_job(11, "dense"), paged_job(12, False), dense_job(13, "ksplit"),
            paged_job(14, True)]
    for j in jobs:
        lay_b = j.get("lay_b", j["lay"])
        j["exp_wire"] = oracle_lib.pack(j["lay"], j["host"], j["l0"], j["l1"], j["t0"], j["t1"])
        j["exp_recv"] = np.full(lay_b.storage_bytes(), 0xA5, np.uint8)
        oracle_lib.unpack(lay_b, j["exp_recv"], j["l0"], j["l1"], j["t0"], j["t1"],
                          j["exp_wire"])
        n = j["exp_wire"].nbytes
        assert n > 0
        j["wire"] = G.dev_const(n, 0x5C)
        if j["token"]:  # increments: pos = t0 for active sequences, -1 otherwise
            j["pos"] = np.where(j["t1"] > j["t0"], j["t0"], -1).astype(np.int32)
    torch.cuda.synchronize()
    start = threading.Barrier(len(jobs))
    errors = []

    def work(j):
        try:
            s = torch.cuda.Stream()
            n = j["exp_wire"].nbytes
            start.wait()
            for _ in range(ITERS):
                if j["token"]:
                    m = dv.dv_stream_out_token(j["src"], 0, j["l0"], j["l1"], j["pos"],
                                               j["wire"], n, s)
                else:
                    m = dv.dv_stream_out_prompt(j["src"], 0, j["l0"], j["l1"], j["t0"],
                                                j["t1"], j["wire"], n, s)
                assert m == n
                dv.dv_stream_in(j["dst"], 0, j["l0"], j["l1"], j["t0"], j["t1"], j["wire"], n,
                                s)
            s.synchronize()
        except Exception as e:  # noqa: BLE001 -- reported by the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=work, args=(j,)) for j in jobs]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i, j in enumerate(jobs):
        assert G.host(j["wire"]).tobytes() == j["exp_wire"].tobytes(), f"job {i}: wire"
        assert G.host(j["recv"]).tobytes() == j["exp_recv"].tobytes(), f"job {i}: receiver"

"""Randomized streams between layouts, byte for byte against the oracle.

Each case draws a sender and a receiver layout independently (dense, paged
or split key, each with its own capacity, block size and table), shared
layer / head / head_dim / batch / element-size extents, a layer sub-range
and per-sequence ranges (prompt prefixes, arbitrary spans, runs of a few
tokens, empty ranges, single tokens with inactive sequences), then packs the sender, compares the
stream with the oracle's pack, streams it into a sentinel-filled receiver
(paged receivers sometimes with an owner-map workspace) and compares the
whole receiver with the oracle's unpack.  Every case prints its seed first,
so a failure names it.
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

KINDS = (dv.DV_DENSE, dv.DV_PAGED, dv.DV_DENSE_KSPLIT)
OKIND = {dv.DV_DENSE: oracle.DENSE, dv.DV_PAGED: oracle.PAGED,
         dv.DV_DENSE_KSPLIT: oracle.KSPLIT}


class Side:
    """One layout with its host mirror, device buffers and descriptor."""

    def __init__(self, r, kind, L, H, D, B, E, cap, seed, fill=None):
        self.kind = kind
        owners = None
        if kind == dv.DV_PAGED:
            bs = int(r.choice([1, 2, 4, 8, 16, 32]))
            maxb = max(1, -(-cap // bs)) + int(r.integers(0, 3))
            used = [maxb] * B  # every logical block mapped, so any range is valid
            bt, nb = synth.make_paged_tables(seed, [u * bs for u in used], bs, maxb)
            extra = int(r.integers(0, 4))  # pool blocks no table entry maps
            nb += extra
            self.lay = oracle.Layout(oracle.PAGED, L, H, D, B, elem_bytes=E, block_size=bs,
                                     num_blocks=nb, block_table=bt)
            self.bt_dev = G.to_dev(bt)
            if r.random() < 0.5:
                owners = [torch.full((nb,), 3, dtype=torch.int32, device=G.DEV)]
            tables = [self.bt_dev]
            extents = dict(block_size=bs, num_blocks=nb, max_blocks=maxb,
                           block_tables=tables, block_owners=owners)
        else:
            S = cap + int(r.integers(0, 20))
            self.lay = oracle.Layout(OKIND[kind], L, H, D, B, seq_cap=S, elem_bytes=E)
            extents = dict(max_seq=S)
        n = self.lay.storage_bytes()
        self.host = synth.fill_bytes(n, seed) if fill is None else np.full(n, fill, np.uint8)
        self.dev = G.to_dev(self.host)
        self.desc = dv.Cache(kind, L, H, D, B, [self.dev], elem_bytes=E, **extents)


def one_case(orc, seed):
    r = np.random.default_rng(seed)
    E = int(r.choice([2, 2, 2, 1, 4, 8]))
    # 1..32 16-byte groups per token (split key holds at most 32)
    D = int(r.choice([1, 2, 4, 8, 16, 32])) * (16 // E)
    L = int(r.integers(1, 4))
    H = int(r.integers(1, 9))
    B = int(r.integers(65, 90)) if r.random() < 0.1 else int(r.integers(1, 10))
    kinds = [int(k) for k in r.choice(KINDS, size=2)]
    tmax = int(r.integers(1, 160))
    style = r.choice(["prompt", "spans", "tokens", "short"])
    if style == "tokens":
        pos = r.integers(0, tmax, size=B).astype(np.int32)
        pos[r.random(B) < 0.3] = -1
        t0 = np.maximum(pos, 0).astype(np.int32)
        t1 = np.where(pos >= 0, pos + 1, 0).astype(np.int32)
    else:
        t0 = np.zeros(B, np.int32)
        t1 = np.zeros(B, np.int32)
        for b in range(B):
            if style == "prompt":
                a, c = 0, int(r.integers(0, tmax + 1))
            elif style == "short":  # a few tokens, as a multi-token decode step
                a = int(r.integers(0, tmax + 1))
                c = min(tmax, a + int(r.integers(0, 13)))
            else:
                a, c = sorted(int(v) for v in r.integers(0, tmax + 1, size=2))
            if r.random() < 0.15:
                c = a
            t0[b], t1[b] = a, c
    l0 = int(r.integers(0, L))
    l1 = int(r.integers(l0 + 1, L + 1))
    cap = tmax + 1
    snd = Side(r, kinds[0], L, H, D, B, E, cap, seed)
    rcv = Side(r, kinds[1], L, H, D, B, E, cap, seed + 7, fill=0xA5)

    exp = orc.pack(snd.lay, snd.host, l0, l1, t0, t1)
    n = exp.nbytes
    wire = G.dev_const(n + 32, 0x5C)
    st = torch.cuda.current_stream()
    if style == "tokens" and r.random() < 0.5:
        got_n = dv.dv_stream_out_token(snd.desc, 0, l0, l1, pos, wire, n, st)
    else:
        got_n = dv.dv_stream_out_prompt(snd.desc, 0, l0, l1, t0, t1, wire, n, st)
    assert got_n == n
    torch.cuda.synchronize()
    w = G.host(wire)
    assert w[:n].tobytes() == exp.tobytes(), "stream-out differs from the oracle"
    assert (w[n:] == 0x5C).all(), "stream-out wrote past its end"

    if n:
        dv.dv_stream_in(rcv.desc, 0, l0, l1, t0, t1, wire, n, st)
    torch.cuda.synchronize()
    exp_recv = rcv.host.copy()
    orc.unpack(rcv.lay, exp_recv, l0, l1, t0, t1, exp)
    assert G.host(rcv.dev).tobytes() == exp_recv.tobytes(), "stream-in differs from the oracle"


@pytest.mark.parametrize("block", range(10))
def test_random_streams_between_layouts(oracle_lib, block):
    """1000 cases in blocks of 100."""
    for seed in range(block * 100, (block + 1) * 100):
        print(f"fuzz case seed {seed}", flush=True)
        one_case(oracle_lib, 5000 + seed)

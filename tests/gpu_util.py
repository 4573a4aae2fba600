"""Helpers for the GPU tests: device buffers, sampled oracle checks."""
from __future__ import annotations

import numpy as np
import torch

import synth

DEV = torch.device("cuda:0")
TDT = {1: torch.uint8, 2: torch.int16, 4: torch.int32, 8: torch.int64}
NDT = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


def dev_filled(nbytes: int, seed: int) -> torch.Tensor:
    """Device buffer holding the counter-mode stream (device fill kernel)."""
    t = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    synth.device_fill(t.data_ptr(), (nbytes + 15) // 16 * 16, seed,
                      stream=torch.cuda.current_stream().cuda_stream)
    return t


def dev_const(nbytes: int, byte: int) -> torch.Tensor:
    return torch.full((max(nbytes, 16),), byte, dtype=torch.uint8, device=DEV)


def assert_same_bytes(dev: torch.Tensor, exp: np.ndarray, what: str,
                      chunk: int = 1 << 30) -> int:
    """Every byte of the host array ``exp`` equals the byte at the same offset
    of the device buffer ``dev`` (compared on the device, ``chunk`` bytes at
    a time).  Returns the number of bytes compared."""
    e8 = np.ascontiguousarray(exp).view(np.uint8).reshape(-1)
    d8 = dev.view(torch.uint8).reshape(-1)
    n = e8.size
    assert d8.numel() >= n, f"{what}: device buffer of {d8.numel()} B, expected {n} B"
    for off in range(0, n, chunk):
        m = min(chunk, n - off)
        e = torch.from_numpy(e8[off:off + m]).to(DEV)
        g = d8[off:off + m]
        if not torch.equal(g, e):
            bad = (g != e).nonzero().reshape(-1)
            raise AssertionError(f"{what}: {bad.numel()} of {m} bytes differ in "
                                 f"[{off}, {off + m}); first at byte {off + int(bad[0])}")
        del e
    return n


def gather(t: torch.Tensor, idx: np.ndarray, E: int) -> np.ndarray:
    """Elements idx of device buffer t (E-byte items), to the host."""
    v = t.view(TDT[E])
    i = torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int64)).to(DEV)
    return v[i].cpu().numpy().view(NDT[E])


def check_pack_sampled(orc, lay, data_seed: int, wire: torch.Tensor, l0, l1, t0, t1,
                       nsamp: int, seed: int) -> int:
    """Wire elements at random indices equal the generated source elements the
    oracle says they hold.  Returns the number of samples checked."""
    E = lay.elem_bytes
    nel = orc.wire_elems(lay, l0, l1, t0, t1)
    if nel == 0:
        return 0
    rng = np.random.default_rng(seed)
    w = rng.integers(0, nel, size=nsamp)
    w = np.concatenate([w, [0, nel - 1]])
    src = orc.wire_to_storage(lay, l0, l1, t0, t1, w)
    assert (src >= 0).all()
    exp = synth.bytes_at(data_seed, src.astype(np.uint64) * np.uint64(E), E).astype(NDT[E])
    got = gather(wire, w, E)
    bad = np.flatnonzero(got != exp)
    assert bad.size == 0, f"{bad.size} of {w.size} sampled wire elements differ; first at {w[bad[0]]}"
    return w.size


def check_unpack_sampled(orc, lay, wire_seed: int, cache: torch.Tensor, l0, l1, t0, t1,
                         nsamp: int, seed: int) -> int:
    """Cache elements the oracle maps sampled wire indices to hold those wire
    elements (the wire was filled from ``wire_seed``)."""
    E = lay.elem_bytes
    nel = orc.wire_elems(lay, l0, l1, t0, t1)
    if nel == 0:
        return 0
    rng = np.random.default_rng(seed)
    w = np.concatenate([rng.integers(0, nel, size=nsamp), [0, nel - 1]])
    dst = orc.wire_to_storage(lay, l0, l1, t0, t1, w)
    assert (dst >= 0).all()
    exp = synth.bytes_at(wire_seed, w.astype(np.uint64) * np.uint64(E), E).astype(NDT[E])
    got = gather(cache, dst, E)
    bad = np.flatnonzero(got != exp)
    assert bad.size == 0, f"{bad.size} of {w.size} sampled cache elements differ"
    return w.size


def dense6(t: torch.Tensor, L, B, H, S, D, E) -> torch.Tensor:
    return t[: L * 2 * B * H * S * D * E].view(TDT[E]).view(L, 2, B, H, S, D)


def assert_dense_ranges_equal(recv, src, L, B, H, S, D, E, l0, l1, t0, t1, sentinel=None):
    """recv equals src on the ranges; elsewhere recv holds `sentinel` bytes
    (if given).  Runs on the device."""
    r = dense6(recv, L, B, H, S, D, E)
    s = dense6(src, L, B, H, S, D, E)
    for b in range(B):
        a, e = int(t0[b]), int(t1[b])
        assert torch.equal(r[l0:l1, :, b, :, a:e, :], s[l0:l1, :, b, :, a:e, :]), f"seq {b}"
    if sentinel is not None:
        m = torch.ones((L, 2, B, H, S), dtype=torch.bool, device=DEV)
        for b in range(B):
            m[l0:l1, :, b, :, int(t0[b]):int(t1[b])] = False
        sv = torch.full((E,), sentinel, dtype=torch.uint8, device=DEV).view(TDT[E])[0]
        outside = r[m]
        assert bool((outside == sv).all()), "bytes outside the ranges changed"


def owner_map_expected(bt, nb, bs, t0, t1):
    """Inverse of a block table over the ranges, as the header defines it:
    pool block -> b * max_blocks + j, -1 for blocks no streamed token uses."""
    maxb = bt.shape[1]
    own = np.full(nb, -1, np.int32)
    for b in range(bt.shape[0]):
        if t1[b] <= t0[b]:
            continue
        for j in range(t0[b] // bs, (t1[b] - 1) // bs + 1):
            if 0 <= bt[b, j] < nb:
                own[bt[b, j]] = b * maxb + j
    return own

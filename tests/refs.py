"""Expected values from numpy primitives, independent of the oracle's C code.

Every helper here states a streaming result through a library routine rather
than through the oracle's address formulas:

* a dense cache is a C-ordered array ``[L][2][B][H][S][D]``; the selected
  region of a stream is a boolean mask over it, and the contiguous buffer is
  that mask's selection in C order (numpy boolean indexing), i.e. the
  selected elements sorted by (layer, K|V, sequence, head, token, dim);
* a paged pool or a split-key cache is mapped to the same logical array by
  numpy fancy indexing / reshape / transpose and then selected the same way.
"""
from __future__ import annotations

import numpy as np

DT = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


def range_mask(L, B, H, S, D, l0, l1, t0, t1) -> np.ndarray:
    m = np.zeros((L, 2, B, H, S, D), dtype=bool)
    for b in range(B):
        m[l0:l1, :, b, :, t0[b]:t1[b], :] = True
    return m


def dense_view(buf: np.ndarray, L, B, H, S, D, E) -> np.ndarray:
    return buf.view(DT[E])[: L * 2 * B * H * S * D].reshape(L, 2, B, H, S, D)


def pack_dense(buf, L, B, H, S, D, E, l0, l1, t0, t1) -> np.ndarray:
    x = dense_view(buf, L, B, H, S, D, E)
    return x[range_mask(L, B, H, S, D, l0, l1, t0, t1)].view(np.uint8)


def unpack_dense(buf, L, B, H, S, D, E, l0, l1, t0, t1, wire) -> np.ndarray:
    out = buf.copy()
    x = dense_view(out, L, B, H, S, D, E)
    x[range_mask(L, B, H, S, D, l0, l1, t0, t1)] = wire.view(DT[E])
    return out


def paged_logical(pool, L, NB, H, bs, D, E, bt, scap) -> np.ndarray:
    """Logical [L][2][B][H][scap][D] array read through the block table.

    Positions whose table entry is -1 read block 0 (they are never selected).
    """
    p = pool.view(DT[E]).reshape(L, 2, NB, H, bs, D).transpose(0, 1, 3, 2, 4, 5)
    s = np.arange(scap)
    blk = np.maximum(bt[:, s // bs], 0)               # [B, scap]
    slot = np.broadcast_to(s % bs, blk.shape)         # [B, scap]
    x = p[:, :, :, blk, slot, :]                      # [L, 2, H, B, scap, D]
    return np.ascontiguousarray(x.transpose(0, 1, 3, 2, 4, 5))


def pool_from_logical(x, pool_shape, bt, bs, E, base=None) -> np.ndarray:
    """Pool bytes holding logical array x [L][2][B][H][S][D] through table bt.

    Every (sequence, logical block) with a valid entry is written; pool
    blocks no table names keep ``base`` (zeros by default).
    """
    L, NB, H, D = pool_shape
    pool = (np.zeros(L * 2 * NB * H * bs * D, dtype=DT[E]) if base is None
            else base.view(DT[E]).copy())
    p = pool.reshape(L, 2, NB, H, bs, D)
    B, S = x.shape[2], x.shape[4]
    for b in range(B):
        for j in range(bt.shape[1]):
            if bt[b, j] < 0 or j * bs >= S:
                continue
            p[:, :, bt[b, j], :, :, :] = x[:, :, b, :, j * bs:(j + 1) * bs, :]
    return pool.view(np.uint8)


def ksplit_from_dense(buf, L, B, H, S, D, E) -> np.ndarray:
    """Same content with the key slab stored as [..][D/x][S][x], x = 16/E."""
    x = 16 // E
    d = dense_view(buf, L, B, H, S, D, E)
    out = d.copy()
    k = d[:, 0].reshape(L, B, H, S, D // x, x).transpose(0, 1, 2, 4, 3, 5)
    out[:, 0] = np.ascontiguousarray(k).reshape(L, B, H, S, D)
    return out.reshape(-1).view(np.uint8)


def ksplit_to_dense(buf, L, B, H, S, D, E) -> np.ndarray:
    x = 16 // E
    v = buf.view(DT[E])[: L * 2 * B * H * S * D].reshape(L, 2, B, H, S, D).copy()
    k = v[:, 0].reshape(L, B, H, D // x, S, x).transpose(0, 1, 2, 4, 3, 5)
    v[:, 0] = np.ascontiguousarray(k).reshape(L, B, H, S, D)
    return v.reshape(-1).view(np.uint8)

"""The oracle run layer by layer on host threads (full-size parity tests and
the benchmark's CPU-baseline leg).  TEST INFRASTRUCTURE ONLY, like the rest
of this package.

The oracle moves one element at a time on one thread; the full-size
workloads stream up to 11 GB per call.  Layer ranges concatenate: the stream
of layers [l0, l1) is the stream of [l0, m) followed by that of [m, l1)
(pinned in the CPU tests).  So a call over [l0, l1) is split here into one
oracle call per layer [l, l+1), each on a host thread of its own, writing
its own slab of the contiguous buffer (pack) or its own layer of the cache
(unpack, copy).  The oracle's code is unchanged: this module only slices
buffers and hands them to it, and ctypes releases the GIL during each call.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np


def host_threads() -> int:
    """The process's CPU affinity count."""
    return max(1, len(os.sched_getaffinity(0)))


def _run(fn, items, threads: Optional[int]):
    with ThreadPoolExecutor(threads or host_threads()) as ex:
        list(ex.map(fn, items))


def layer_bytes(orc, lay, t0, t1) -> int:
    """Bytes of one layer's stream for these token ranges."""
    return orc.wire_elems(lay, 0, 1, t0, t1) * lay.elem_bytes


def pack(orc, lay, cache: np.ndarray, l0: int, l1: int, t0, t1,
         threads: Optional[int] = None) -> np.ndarray:
    """The oracle's stream of layers [l0, l1), one layer per call."""
    per = layer_bytes(orc, lay, t0, t1)
    out = np.empty(per * (l1 - l0), dtype=np.uint8)
    if per == 0:
        return out

    def one(l):
        k = l - l0
        orc.pack_into(lay, cache, l, l + 1, t0, t1, out[k * per:(k + 1) * per])

    _run(one, range(l0, l1), threads)
    return out


def unpack(orc, lay, cache: np.ndarray, l0: int, l1: int, t0, t1, wire: np.ndarray,
           threads: Optional[int] = None) -> None:
    """The oracle's stream-in of layers [l0, l1) into ``cache`` (in place)."""
    per = layer_bytes(orc, lay, t0, t1)
    if per == 0:
        return
    assert wire.nbytes >= per * (l1 - l0)

    def one(l):
        k = l - l0
        orc.unpack(lay, cache, l, l + 1, t0, t1, wire[k * per:(k + 1) * per])

    _run(one, range(l0, l1), threads)


def copy_ranges(orc, src_lay, src: np.ndarray, dst_lay, dst: np.ndarray, l0: int, l1: int,
                t0, t1, threads: Optional[int] = None) -> None:
    """The oracle's copy of the ranges of layers [l0, l1), one layer per call."""
    _run(lambda l: orc.copy_ranges(src_lay, src, dst_lay, dst, l, l + 1, t0, t1),
         range(l0, l1), threads)

"""ctypes binding of the comparison baselines (``libdv_baseline.so``).

``per_region_copy``: one copy call per contiguous region (the comparison
baseline of the paper's evaluation, Sec. 5.1).  ``plain_copy``: a contiguous
16-byte copy with the pack kernel's launch shape, the ceiling the streaming
kernels are set against.  ``block_copy``: a copy of whole blocks in a block
table's order, the ceiling of the paged kernels.  Used by the benchmark and
its tests only.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import dv

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdv_baseline.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        lib.dvb_per_region_copy.argtypes = [ctypes.POINTER(dv.dv_cache), i32, i32, i32, vp, vp,
                                            vp, ctypes.c_uint64, vp]
        lib.dvb_per_region_copy.restype = ctypes.c_int64
        lib.dvb_plain_copy.argtypes = [vp, vp, ctypes.c_uint64, vp]
        lib.dvb_plain_copy.restype = ctypes.c_int
        lib.dvb_block_copy.argtypes = [vp, vp, vp, ctypes.c_uint32, ctypes.c_uint32,
                                       ctypes.c_int, vp]
        lib.dvb_block_copy.restype = ctypes.c_int
        _lib = lib
    return _lib


def per_region_copy(cache: dv.Cache, mb: int, l0: int, l1: int, t0, t1, dst, dst_cap: int,
                    stream=None) -> int:
    """Returns the number of copy calls issued."""
    a0, p0 = dv._i32(np.zeros(cache.c.batch, np.int32) if t0 is None else t0, cache.c.batch)
    a1, p1 = dv._i32(t1, cache.c.batch)
    n = _load().dvb_per_region_copy(cache.ref, mb, l0, l1, p0, p1, dv._addr(dst), dst_cap,
                                    dv._stream(stream))
    if n < 0:
        raise dv.DvError(int(n), "dvb_per_region_copy")
    return int(n)


def plain_copy(dst, src, nbytes: int, stream=None) -> None:
    rc = _load().dvb_plain_copy(dv._addr(dst), dv._addr(src), nbytes, dv._stream(stream))
    if rc != dv.DV_OK:
        raise dv.DvError(int(rc), "dvb_plain_copy")


def block_copy(dst, src, order, nblocks: int, block_bytes: int, scatter: bool = False,
               stream=None) -> None:
    """Block ``order[c]`` of ``src`` to block c of ``dst`` (or, with
    ``scatter``, block c of ``src`` to block ``order[c]`` of ``dst``)."""
    rc = _load().dvb_block_copy(dv._addr(dst), dv._addr(src), dv._addr(order), nblocks,
                                block_bytes, 1 if scatter else 0, dv._stream(stream))
    if rc != dv.DV_OK:
        raise dv.DvError(int(rc), "dvb_block_copy")

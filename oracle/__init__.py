"""CPU oracle for the KV-cache streaming path (ctypes over ``dv_oracle.c``).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package; the HIP library
never does, and the two share no code.  The arithmetic is in ``dv_oracle.c``
(plain C, one element at a time); this file only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "dv_oracle.c")
LIB_PATH = os.path.join(HERE, "libdvoracle.so")

DENSE, PAGED, KSPLIT = 0, 1, 2
OK, INVALID, RANGE = 0, -1, -2


def build(out_path: str = LIB_PATH, mutant: int = 0) -> str:
    """Compile the oracle with gcc (``mutant`` > 0 plants a known mistake)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared", SRC,
           "-o", out_path]
    if mutant:
        cmd.insert(1, f"-DDVO_MUTANT={mutant}")
    subprocess.run(cmd, check=True)
    return out_path


class _Layout(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("elem_bytes", ctypes.c_int64),
        ("layers", ctypes.c_int64),
        ("heads", ctypes.c_int64),
        ("head_dim", ctypes.c_int64),
        ("batch", ctypes.c_int64),
        ("seq_cap", ctypes.c_int64),
        ("block_size", ctypes.c_int64),
        ("num_blocks", ctypes.c_int64),
        ("max_blocks", ctypes.c_int64),
        ("block_table", ctypes.POINTER(ctypes.c_int32)),
    ]


class Layout:
    """A cache layout as the oracle sees it (host memory only)."""

    def __init__(self, kind: int, layers: int, heads: int, head_dim: int, batch: int,
                 seq_cap: int = 0, elem_bytes: int = 2, block_size: int = 0,
                 num_blocks: int = 0, block_table: Optional[np.ndarray] = None):
        self.kind, self.layers, self.heads = kind, layers, heads
        self.head_dim, self.batch, self.elem_bytes = head_dim, batch, elem_bytes
        self.seq_cap, self.block_size, self.num_blocks = seq_cap, block_size, num_blocks
        self.block_table = None
        max_blocks = 0
        if block_table is not None:
            self.block_table = np.ascontiguousarray(block_table, dtype=np.int32)
            max_blocks = self.block_table.shape[1]
        self.max_blocks = max_blocks
        self._c = _Layout(kind, elem_bytes, layers, heads, head_dim, batch, seq_cap,
                          block_size, num_blocks, max_blocks,
                          None if self.block_table is None else
                          self.block_table.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))

    def storage_elems(self) -> int:
        if self.kind == PAGED:
            return (self.layers * 2 * self.num_blocks * self.heads * self.block_size
                    * self.head_dim)
        return self.layers * 2 * self.batch * self.heads * self.seq_cap * self.head_dim

    def storage_bytes(self) -> int:
        return self.storage_elems() * self.elem_bytes


class Oracle:
    def __init__(self, lib_path: str = LIB_PATH):
        if not os.path.exists(lib_path):
            raise RuntimeError(f"{lib_path} is not built; run oracle.build()")
        lib = ctypes.CDLL(lib_path)
        P = ctypes.POINTER(_Layout)
        i64, vp, i32p = ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p
        lib.dvo_elem_index.argtypes = [P, i64, i64, i64, i64, i64, i64]
        lib.dvo_elem_index.restype = i64
        lib.dvo_check.argtypes = [P, i64, i64, i32p, i32p]
        lib.dvo_check.restype = ctypes.c_int
        lib.dvo_wire_elems.argtypes = [P, i64, i64, i32p, i32p]
        lib.dvo_wire_elems.restype = i64
        lib.dvo_pack.argtypes = [P, vp, i64, i64, i32p, i32p, vp]
        lib.dvo_pack.restype = ctypes.c_int
        lib.dvo_unpack.argtypes = [P, vp, i64, i64, i32p, i32p, vp]
        lib.dvo_unpack.restype = ctypes.c_int
        lib.dvo_copy_ranges.argtypes = [P, vp, P, vp, i64, i64, i32p, i32p]
        lib.dvo_copy_ranges.restype = ctypes.c_int
        lib.dvo_wire_to_storage.argtypes = [P, i64, i64, i32p, i32p, vp, i64, vp]
        lib.dvo_wire_to_storage.restype = ctypes.c_int
        self.lib = lib

    @staticmethod
    def _r(t):
        a = np.ascontiguousarray(t, dtype=np.int32)
        return a, a.ctypes.data

    def check(self, lay: Layout, l0: int, l1: int, t0, t1) -> int:
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        return self.lib.dvo_check(ctypes.byref(lay._c), l0, l1, p0, p1)

    def elem_index(self, lay: Layout, l, kv, b, h, s, d) -> int:
        return self.lib.dvo_elem_index(ctypes.byref(lay._c), l, kv, b, h, s, d)

    def wire_elems(self, lay: Layout, l0, l1, t0, t1) -> int:
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        return self.lib.dvo_wire_elems(ctypes.byref(lay._c), l0, l1, p0, p1)

    def pack(self, lay: Layout, cache: np.ndarray, l0, l1, t0, t1) -> np.ndarray:
        """Contiguous wire bytes (uint8) for the ranges."""
        cache = np.ascontiguousarray(cache)
        assert cache.nbytes >= lay.storage_bytes()
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        rc = self.lib.dvo_check(ctypes.byref(lay._c), l0, l1, p0, p1)
        if rc != OK:
            raise ValueError(f"oracle rejects ranges ({rc})")
        n = self.lib.dvo_wire_elems(ctypes.byref(lay._c), l0, l1, p0, p1)
        wire = np.empty(n * lay.elem_bytes, dtype=np.uint8)
        rc = self.lib.dvo_pack(ctypes.byref(lay._c), cache.ctypes.data, l0, l1, p0, p1,
                               wire.ctypes.data)
        assert rc == OK
        return wire

    def pack_into(self, lay: Layout, cache: np.ndarray, l0, l1, t0, t1,
                  out: np.ndarray) -> None:
        """As ``pack``, into the first wire bytes of the contiguous uint8
        array ``out``."""
        cache = np.ascontiguousarray(cache)
        assert cache.nbytes >= lay.storage_bytes()
        assert out.dtype == np.uint8 and out.flags.c_contiguous
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        rc = self.lib.dvo_check(ctypes.byref(lay._c), l0, l1, p0, p1)
        if rc != OK:
            raise ValueError(f"oracle rejects ranges ({rc})")
        n = self.lib.dvo_wire_elems(ctypes.byref(lay._c), l0, l1, p0, p1)
        assert out.nbytes >= n * lay.elem_bytes
        rc = self.lib.dvo_pack(ctypes.byref(lay._c), cache.ctypes.data, l0, l1, p0, p1,
                               out.ctypes.data)
        assert rc == OK

    def unpack(self, lay: Layout, cache: np.ndarray, l0, l1, t0, t1, wire: np.ndarray) -> None:
        """Writes the ranges of ``cache`` (in place) from ``wire``."""
        assert cache.flags.c_contiguous and cache.nbytes >= lay.storage_bytes()
        wire = np.ascontiguousarray(wire)
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        n = self.lib.dvo_wire_elems(ctypes.byref(lay._c), l0, l1, p0, p1)
        assert wire.nbytes >= n * lay.elem_bytes
        rc = self.lib.dvo_unpack(ctypes.byref(lay._c), cache.ctypes.data, l0, l1, p0, p1,
                                 wire.ctypes.data)
        if rc != OK:
            raise ValueError(f"oracle rejects ranges ({rc})")

    def copy_ranges(self, src_lay: Layout, src: np.ndarray, dst_lay: Layout, dst: np.ndarray,
                    l0, l1, t0, t1) -> None:
        assert dst.flags.c_contiguous
        src = np.ascontiguousarray(src)
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        rc = self.lib.dvo_copy_ranges(ctypes.byref(src_lay._c), src.ctypes.data,
                                      ctypes.byref(dst_lay._c), dst.ctypes.data, l0, l1, p0, p1)
        if rc != OK:
            raise ValueError(f"oracle rejects copy ({rc})")

    def wire_to_storage(self, lay: Layout, l0, l1, t0, t1, widx) -> np.ndarray:
        w = np.ascontiguousarray(widx, dtype=np.int64)
        out = np.empty_like(w)
        a0, p0 = self._r(t0)
        a1, p1 = self._r(t1)
        rc = self.lib.dvo_wire_to_storage(ctypes.byref(lay._c), l0, l1, p0, p1, w.ctypes.data,
                                          w.size, out.ctypes.data)
        if rc != OK:
            raise ValueError(f"oracle rejects ranges ({rc})")
        return out


_default: Optional[Oracle] = None


def get() -> Oracle:
    """The oracle built from source (builds it if the library is missing)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB_PATH):
            build()
        _default = Oracle()
    return _default

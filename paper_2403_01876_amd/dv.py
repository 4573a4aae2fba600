"""Python binding of ``libdv.so`` (ctypes): argument marshalling only.

The functions carry the C names (``dv_stream_out_prompt`` ...) and take the
same arguments; buffers may be given as raw addresses or as tensors (their
``data_ptr()`` is passed), streams as raw ``hipStream_t`` values or
``torch.cuda.Stream`` objects.  Every byte is moved by the library's HIP
kernels or DMA calls; there is no Python or CPU fallback, and importing this
module fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdv.so")

DV_OK, DV_ERR_INVALID, DV_ERR_RANGE, DV_ERR_SPACE, DV_ERR_UNSUPPORTED, DV_ERR_HIP = \
    0, -1, -2, -3, -4, -5
DV_DENSE, DV_PAGED, DV_DENSE_KSPLIT = 0, 1, 2
DV_MEM_DEVICE, DV_MEM_HOST_PINNED = 0, 1


class DvError(RuntimeError):
    def __init__(self, status: int, call: str):
        super().__init__(f"{call}: {status_string(status)} ({status})")
        self.status = status


class dv_cache(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("mem", ctypes.c_int32),
        ("elem_bytes", ctypes.c_int32),
        ("num_layers", ctypes.c_int32),
        ("num_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("max_seq", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("num_blocks", ctypes.c_int32),
        ("max_blocks", ctypes.c_int32),
        ("num_mb", ctypes.c_int32),
        ("mb_base", ctypes.POINTER(ctypes.c_void_p)),
        ("block_table", ctypes.POINTER(ctypes.c_void_p)),
        ("block_owner", ctypes.POINTER(ctypes.c_void_p)),
    ]


API_VERSION = 3  # DV_API_VERSION the dv_cache layout and calls here match


def _load():
    # torch's libraries need the HIP runtime by file name (libamdhip64.so)
    # while libdv.so needs it by SONAME (libamdhip64.so.7): importing torch
    # first makes libdv.so bind to the runtime torch already loaded, so both
    # share one runtime (a second copy in the process sees no device).
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(dv_cache)
    i32, u64, vp = ctypes.c_int32, ctypes.c_uint64, ctypes.c_void_p
    u64p = ctypes.POINTER(ctypes.c_uint64)
    sig = {
        "dv_cache_bytes": [P, u64p],
        "dv_packed_bytes": [P, i32, i32, vp, vp, u64p],
        "dv_stream_out_prompt": [P, i32, i32, i32, vp, vp, vp, u64, u64p, vp],
        "dv_stream_out_token": [P, i32, i32, i32, vp, vp, u64, u64p, vp],
        "dv_stream_in": [P, i32, i32, i32, vp, vp, vp, u64, vp],
        "dv_stream_in_noalloc": [P, i32, i32, i32, vp, vp, vp, u64, vp],
        "dv_swap_out": [P, i32, P, i32, i32, i32, vp, vp, vp],
        "dv_swap_in": [P, i32, P, i32, i32, i32, vp, vp, vp],
        "dv_block_claims": [P, i32, vp, vp, vp, vp],
        "dv_api_version": [],
        "dv_swapper_create": [P, P, ctypes.POINTER(vp)],
        "dv_swapper_prefetch": [vp, i32, vp],
        "dv_swapper_begin_step": [vp, i32, vp, ctypes.POINTER(i32)],
        "dv_swapper_end_step": [vp, i32, vp, vp, vp],
        "dv_swapper_sync": [vp],
        "dv_swapper_destroy": [vp],
        "dv_streamer_create": [P, i32, vp, u64, vp, u64, ctypes.POINTER(vp)],
        "dv_streamer_push": [vp, vp, i32, i32, vp, vp, u64, u64, u64p],
        "dv_streamer_flush": [vp],
        "dv_streamer_destroy": [vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.dv_status_string.argtypes = [ctypes.c_int]
    lib.dv_status_string.restype = ctypes.c_char_p
    if lib.dv_api_version() != API_VERSION:
        raise ImportError(f"{LIB_PATH} is API version {lib.dv_api_version()}, this binding "
                          f"expects {API_VERSION}: rebuild with __graft_entry__.build()")
    return lib


lib = _load()

# Symbols include/dv.h declares (checked by the tests against the library).
EXPORTS = ("dv_cache_bytes", "dv_packed_bytes", "dv_stream_out_prompt", "dv_stream_out_token",
           "dv_stream_in", "dv_swap_out", "dv_swap_in", "dv_status_string", "dv_api_version",
           "dv_swapper_create", "dv_swapper_prefetch", "dv_swapper_begin_step",
           "dv_swapper_end_step", "dv_swapper_sync", "dv_swapper_destroy",
           "dv_streamer_create", "dv_streamer_push", "dv_streamer_flush", "dv_streamer_destroy",
           "dv_block_claims", "dv_stream_in_noalloc")
NOALLOC_MAX_BLOCKS = 1 << 20  # DV_NOALLOC_MAX_BLOCKS


def status_string(status: int) -> str:
    return lib.dv_status_string(status).decode()


def _addr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)}")


def _stream(s) -> int:
    """A hipStream_t: an int passes through, a torch stream gives its handle,
    None means torch's current stream (as for torch's own operations)."""
    if s is None:
        import torch
        try:
            return torch.cuda.current_stream().cuda_stream
        except RuntimeError:  # no device: the null stream (the runtime reports the rest)
            return 0
    if isinstance(s, int):
        return s
    return s.cuda_stream


class Cache:
    """A ``dv_cache`` descriptor plus the host arrays it points to."""

    def __init__(self, kind: int, layers: int, heads: int, head_dim: int, batch: int,
                 bases: Sequence, max_seq: int = 0, elem_bytes: int = 2,
                 mem: int = DV_MEM_DEVICE, block_size: int = 0, num_blocks: int = 0,
                 max_blocks: int = 0, block_tables: Optional[Sequence] = None,
                 block_owners: Optional[Sequence] = None):
        """``block_owners``: optional per-microbatch int32 [num_blocks] device
        workspaces (None entries allowed) that let bulk paged stream-ins
        scatter in pool order."""
        # The library reads block_table[mb] and block_owner[mb] for every
        # microbatch index it accepts (below num_mb = len(bases)) and cannot
        # see the arrays' lengths, so shorter arrays are refused here.
        for name, arr in (("block_tables", block_tables), ("block_owners", block_owners)):
            if arr is not None and len(arr) != len(bases):
                raise ValueError(f"{name} has {len(arr)} entries, bases has {len(bases)}")
        # Tensors and arrays given here stay referenced for the descriptor's
        # life, so a temporary cannot be freed while its address is in use.
        self._keep = [x for x in list(bases) + list(block_tables or []) +
                      list(block_owners or []) if not isinstance(x, int) and x is not None]
        self.bases = (ctypes.c_void_p * len(bases))(*[_addr(b) for b in bases])
        self.tables = self.owners = None
        if block_tables is not None:
            self.tables = (ctypes.c_void_p * len(block_tables))(*[_addr(t) for t in block_tables])
        if block_owners is not None:
            self.owners = (ctypes.c_void_p * len(block_owners))(
                *[_addr(o) for o in block_owners])
        ptr = ctypes.POINTER(ctypes.c_void_p)
        self.c = dv_cache(kind, mem, elem_bytes, layers, heads, head_dim, batch, max_seq,
                          block_size, num_blocks, max_blocks, len(bases),
                          ctypes.cast(self.bases, ptr),
                          None if self.tables is None else ctypes.cast(self.tables, ptr),
                          None if self.owners is None else ctypes.cast(self.owners, ptr))

    @property
    def ref(self):
        return ctypes.byref(self.c)


def _i32(a, n: int):
    """An int32 array the library reads ``n`` entries of (one per sequence):
    shorter arrays are refused here, since the C side cannot see their length."""
    if a is None:
        return None, 0
    arr = np.ascontiguousarray(a, dtype=np.int32).reshape(-1)
    if arr.size < n:
        raise ValueError(f"range array has {arr.size} entries, the cache has {n} sequences")
    return arr, arr.ctypes.data


def _check(rc: int, name: str, check: bool):
    if check and rc != DV_OK:
        raise DvError(rc, name)
    return rc


def dv_cache_bytes(cache: Cache, check: bool = True):
    out = ctypes.c_uint64(0)
    rc = lib.dv_cache_bytes(cache.ref, ctypes.byref(out))
    _check(rc, "dv_cache_bytes", check)
    return out.value if check else (rc, out.value)


def dv_packed_bytes(cache: Cache, l0: int, l1: int, t0, t1, check: bool = True):
    a0, p0 = _i32(t0, cache.c.batch)
    a1, p1 = _i32(t1, cache.c.batch)
    out = ctypes.c_uint64(0)
    rc = lib.dv_packed_bytes(cache.ref, l0, l1, p0, p1, ctypes.byref(out))
    _check(rc, "dv_packed_bytes", check)
    return out.value if check else (rc, out.value)


def dv_stream_out_prompt(src: Cache, mb: int, l0: int, l1: int, t0, t1, dst, dst_cap: int,
                         stream=None, check: bool = True):
    """Returns the stream size in bytes (or ``(status, bytes)`` with check=False)."""
    a0, p0 = _i32(t0, src.c.batch)
    a1, p1 = _i32(t1, src.c.batch)
    out = ctypes.c_uint64(0)
    rc = lib.dv_stream_out_prompt(src.ref, mb, l0, l1, p0, p1, _addr(dst), dst_cap,
                                  ctypes.byref(out), _stream(stream))
    _check(rc, "dv_stream_out_prompt", check)
    return out.value if check else (rc, out.value)


def dv_stream_out_token(src: Cache, mb: int, l0: int, l1: int, pos, dst, dst_cap: int,
                        stream=None, check: bool = True):
    ap, pp = _i32(pos, src.c.batch)
    out = ctypes.c_uint64(0)
    rc = lib.dv_stream_out_token(src.ref, mb, l0, l1, pp, _addr(dst), dst_cap,
                                 ctypes.byref(out), _stream(stream))
    _check(rc, "dv_stream_out_token", check)
    return out.value if check else (rc, out.value)


def dv_stream_in(dst: Cache, mb: int, l0: int, l1: int, t0, t1, src, src_bytes: int,
                 stream=None, check: bool = True) -> int:
    a0, p0 = _i32(t0, dst.c.batch)
    a1, p1 = _i32(t1, dst.c.batch)
    rc = lib.dv_stream_in(dst.ref, mb, l0, l1, p0, p1, _addr(src), src_bytes, _stream(stream))
    return _check(rc, "dv_stream_in", check)


def dv_stream_in_noalloc(dst: Cache, mb: int, l0: int, l1: int, t0, t1, src, src_bytes: int,
                         stream=None, check: bool = True) -> int:
    a0, p0 = _i32(t0, dst.c.batch)
    a1, p1 = _i32(t1, dst.c.batch)
    rc = lib.dv_stream_in_noalloc(dst.ref, mb, l0, l1, p0, p1, _addr(src), src_bytes,
                                  _stream(stream))
    return _check(rc, "dv_stream_in_noalloc", check)


def dv_block_claims(cache: Cache, mb: int, t0, t1, counts, stream=None,
                    check: bool = True) -> int:
    """Per-block claim counts of a paged table over the ranges, into the
    device int32 buffer `counts` (read it after synchronising)."""
    a0, p0 = _i32(t0, cache.c.batch)
    a1, p1 = _i32(t1, cache.c.batch)
    rc = lib.dv_block_claims(cache.ref, mb, p0, p1, _addr(counts), _stream(stream))
    return _check(rc, "dv_block_claims", check)


def dv_swap_out(dev: Cache, slot: int, host: Cache, host_mb: int, l0: int, l1: int, t0, t1,
                stream=None, check: bool = True) -> int:
    a0, p0 = _i32(t0, dev.c.batch)
    a1, p1 = _i32(t1, dev.c.batch)
    rc = lib.dv_swap_out(dev.ref, slot, host.ref, host_mb, l0, l1, p0, p1, _stream(stream))
    return _check(rc, "dv_swap_out", check)


def dv_swap_in(host: Cache, host_mb: int, dev: Cache, slot: int, l0: int, l1: int, t0, t1,
               stream=None, check: bool = True) -> int:
    a0, p0 = _i32(t0, host.c.batch)
    a1, p1 = _i32(t1, host.c.batch)
    rc = lib.dv_swap_in(host.ref, host_mb, dev.ref, slot, l0, l1, p0, p1, _stream(stream))
    return _check(rc, "dv_swap_in", check)


def dv_api_version() -> int:
    return lib.dv_api_version()


class Swapper:
    """The microbatch swap scheduler (dv_swapper_*); keeps its descriptors."""

    def __init__(self, dev_slots: Cache, host: Cache):
        self.dev, self.host = dev_slots, host
        h = ctypes.c_void_p(0)
        _check(lib.dv_swapper_create(dev_slots.ref, host.ref, ctypes.byref(h)),
               "dv_swapper_create", True)
        self.h = h

    def prefetch(self, mb: int, lens, check: bool = True) -> int:
        a, p = _i32(lens, self.host.c.batch)
        return _check(lib.dv_swapper_prefetch(self.h, mb, p), "dv_swapper_prefetch", check)

    def begin_step(self, mb: int, stream=None) -> int:
        slot = ctypes.c_int32(-1)
        _check(lib.dv_swapper_begin_step(self.h, mb, _stream(stream), ctypes.byref(slot)),
               "dv_swapper_begin_step", True)
        return slot.value

    def end_step(self, mb: int, t0, t1, stream=None, check: bool = True) -> int:
        a0, p0 = _i32(t0, self.host.c.batch)
        a1, p1 = _i32(t1, self.host.c.batch)
        return _check(lib.dv_swapper_end_step(self.h, mb, _stream(stream), p0, p1),
                      "dv_swapper_end_step", check)

    def sync(self) -> None:
        _check(lib.dv_swapper_sync(self.h), "dv_swapper_sync", True)

    def close(self) -> None:
        if self.h:
            _check(lib.dv_swapper_destroy(self.h), "dv_swapper_destroy", True)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def dv_swapper_create(dev_slots: Cache, host: Cache) -> Swapper:
    return Swapper(dev_slots, host)


class Streamer:
    """The background streamer (dv_streamer_*); keeps its descriptor and its
    staging and destination buffers alive while it exists."""

    def __init__(self, src: Cache, mb: int, staging, staging_cap: int, dst, dst_cap: int):
        self.src = src
        self._keep = [x for x in (staging, dst) if not isinstance(x, int)]
        h = ctypes.c_void_p(0)
        _check(lib.dv_streamer_create(src.ref, mb, _addr(staging), staging_cap, _addr(dst),
                                      dst_cap, ctypes.byref(h)), "dv_streamer_create", True)
        self.h = h

    def push(self, l0: int, l1: int, t0, t1, staging_offset: int, dst_offset=None,
             stream=None, check: bool = True):
        """Returns the region's size in bytes (or (status, bytes) with check=False).
        ``dst_offset`` defaults to ``staging_offset``."""
        a0, p0 = _i32(t0, self.src.c.batch)
        a1, p1 = _i32(t1, self.src.c.batch)
        out = ctypes.c_uint64(0)
        if dst_offset is None:
            dst_offset = staging_offset
        rc = lib.dv_streamer_push(self.h, _stream(stream), l0, l1, p0, p1, staging_offset,
                                  dst_offset, ctypes.byref(out))
        _check(rc, "dv_streamer_push", check)
        return out.value if check else (rc, out.value)

    def flush(self, check: bool = True) -> int:
        return _check(lib.dv_streamer_flush(self.h), "dv_streamer_flush", check)

    def close(self) -> None:
        if self.h:
            _check(lib.dv_streamer_destroy(self.h), "dv_streamer_destroy", True)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

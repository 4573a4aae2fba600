"""Seeded synthetic workloads for the KV-cache streaming path.

This module generates inputs only: cache contents, sequence lengths, decode
positions and paged block tables.  It holds none of the streaming arithmetic
(no address maps, no wire offsets); the oracle and the HIP library both take
their inputs from here and nothing else is shared between them.

Random numbers come from SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014), used two ways:

* counter mode for bulk bytes: 64-bit word k of a buffer filled with seed s is
  ``mix(s + (k + 1) * GOLDEN)``, i.e. the (k+1)-th output of a SplitMix64
  stream started at state s.  Byte j of the buffer is byte (j mod 8),
  little-endian, of word j div 8.  ``synth/csrc/gen_fill.hip`` implements the
  same definition on the GPU so multi-GB caches fill in milliseconds; the two
  are checked against each other in the tests.
* stream mode for lengths and permutations (``SplitMix64`` below).

Workload shapes follow the model-shaped caches of the paper's evaluation
(OPT-13B/66B, BLOOM-176B and a LLaMA-2-70B GQA paged cache, Sec. 5); the
lengths are drawn uniformly in the ranges each workload states.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import List, Optional

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1

# Stream tags: each purpose draws from its own stream so that adding a draw
# to one never shifts another.
TAG_DATA = 0xD474
TAG_LEN = 0x1E45
TAG_PERM_A = 0xB7A0
TAG_PERM_B = 0xB7B0
TAG_SAMPLE = 0x5A3B


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def mix64(z: int) -> int:
    """The SplitMix64 output function applied to one 64-bit value."""
    return _mix(z & MASK64)


class SplitMix64:
    """Sequential SplitMix64 stream: state += GOLDEN, output mix(state)."""

    def __init__(self, seed: int):
        self.state = seed & MASK64

    def next(self) -> int:
        self.state = (self.state + GOLDEN) & MASK64
        return _mix(self.state)

    def below(self, n: int) -> int:
        """Integer in [0, n) as next() mod n (the bias is below 2**-40 here)."""
        return self.next() % n

    def uniform_int(self, lo: int, hi: int) -> int:
        """Integer in [lo, hi], inclusive."""
        return lo + self.next() % (hi - lo + 1)

    def permutation(self, n: int) -> np.ndarray:
        """Fisher-Yates shuffle of range(n), j = next() mod (i + 1)."""
        p = np.arange(n, dtype=np.int64)
        for i in range(n - 1, 0, -1):
            j = self.next() % (i + 1)
            p[i], p[j] = p[j], p[i]
        return p


def derived_seed(seed: int, tag: int) -> int:
    """Seed of the stream for one purpose (data, lengths, permutations)."""
    return mix64((seed ^ tag) & MASK64)


def words_u64(seed: int, first_word: int, count: int) -> np.ndarray:
    """Counter-mode words ``first_word .. first_word+count-1`` as uint64."""
    k = np.arange(first_word + 1, first_word + 1 + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & MASK64) + k * np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def fill_bytes(nbytes: int, seed: int, first_byte: int = 0) -> np.ndarray:
    """Host fill: ``nbytes`` bytes of the counter-mode stream from ``first_byte``.

    Uses the C twin (``csrc/gen_host.c``) when it is built, else numpy."""
    lib = _host_lib()
    if lib is not None:
        out = np.empty(nbytes, dtype=np.uint8)
        lib.dvsynth_host_fill(out.ctypes.data, nbytes, seed & MASK64, first_byte)
        return out
    return fill_bytes_numpy(nbytes, seed, first_byte)


def host_threads() -> int:
    """Host threads for the parallel helpers: the process's CPU affinity."""
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def fill_into(out: np.ndarray, seed: int, first_byte: int = 0,
              threads: Optional[int] = None) -> np.ndarray:
    """Fill the contiguous uint8 array ``out`` with stream bytes
    ``first_byte .. first_byte + out.size``, split into chunks filled on
    ``threads`` host threads (the C twin releases the GIL)."""
    from concurrent.futures import ThreadPoolExecutor

    assert out.dtype == np.uint8 and out.flags.c_contiguous
    lib = _host_lib()
    n = out.size
    if lib is None:
        out[:] = fill_bytes_numpy(n, seed, first_byte)
        return out
    chunk = 1 << 26
    base = out.ctypes.data

    def one(off):
        lib.dvsynth_host_fill(base + off, min(chunk, n - off), seed & MASK64, first_byte + off)

    with ThreadPoolExecutor(threads or host_threads()) as ex:
        list(ex.map(one, range(0, n, chunk)))
    return out


def fill_bytes_parallel(nbytes: int, seed: int, threads: Optional[int] = None) -> np.ndarray:
    """``fill_bytes(nbytes, seed)`` on several host threads."""
    return fill_into(np.empty(nbytes, dtype=np.uint8), seed, 0, threads)


def fill_bytes_numpy(nbytes: int, seed: int, first_byte: int = 0) -> np.ndarray:
    """The numpy statement of the same definition (reference for the C twin)."""
    w0 = first_byte // 8
    w1 = (first_byte + nbytes + 7) // 8
    words = words_u64(seed, w0, w1 - w0)
    raw = words.view(np.uint8)
    off = first_byte - w0 * 8
    return raw[off:off + nbytes].copy()


def bytes_at(seed: int, byte_index: np.ndarray, width: int) -> np.ndarray:
    """Values of ``width``-byte little-endian items starting at each byte index.

    Used to compute single generated values (for sampled checks) without
    materialising the buffer.  ``byte_index`` must be ``width``-aligned and
    ``width`` must divide 8.
    """
    byte_index = np.asarray(byte_index, dtype=np.uint64)
    k = byte_index // np.uint64(8)
    shift = (byte_index % np.uint64(8)) * np.uint64(8)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & MASK64) + (k + np.uint64(1)) * np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    mask = np.uint64((1 << (8 * width)) - 1) if width < 8 else np.uint64(MASK64)
    return (z >> shift) & mask


_HOST_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdvsynth_host.so")
_host = None


def build_host(out: str = _HOST_LIB_PATH) -> str:
    """Compile the host fill with gcc."""
    import subprocess
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "gen_host.c")
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", src, "-o", out], check=True)
    return out


def _host_lib():
    global _host
    if _host is None:
        if not os.path.exists(_HOST_LIB_PATH):
            try:
                build_host()
            except Exception:  # no compiler: numpy path
                _host = False
                return None
        lib = ctypes.CDLL(_HOST_LIB_PATH)
        lib.dvsynth_host_fill.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                          ctypes.c_uint64]
        lib.dvsynth_host_fill.restype = None
        _host = lib
    return _host or None


# ---------------------------------------------------------------------------
# Workloads
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    """One synthetic KV-cache workload.

    Shapes are one pipeline stage's (or one tensor-parallel shard's) share of
    a model's KV cache.  ``lens`` are prompt lengths per sequence; decode step
    i writes position ``lens[b] + i`` of every active sequence.
    """
    name: str
    layers: int
    heads: int
    head_dim: int
    batch: int
    max_seq: int
    lens: np.ndarray
    steps: int
    elem_bytes: int = 2
    paged: bool = False
    block_size: int = 0
    num_blocks: int = 0
    max_blocks: int = 0
    block_table_a: Optional[np.ndarray] = None
    block_table_b: Optional[np.ndarray] = None
    microbatches: int = 1
    device_slots: int = 1
    seed: int = 0

    @property
    def data_seed(self) -> int:
        return derived_seed(self.seed, TAG_DATA)

    def dense_bytes(self, max_seq: Optional[int] = None) -> int:
        s = self.max_seq if max_seq is None else max_seq
        return self.layers * 2 * self.batch * self.heads * s * self.head_dim * self.elem_bytes

    def pool_bytes(self) -> int:
        return (self.layers * 2 * self.num_blocks * self.heads * self.block_size
                * self.head_dim * self.elem_bytes)

    def payload_bytes(self, ntok: int) -> int:
        """Bytes of a stream of ``ntok`` tokens summed over sequences."""
        return self.layers * 2 * self.heads * self.head_dim * self.elem_bytes * ntok

    def prompt_ranges(self):
        t0 = np.zeros(self.batch, dtype=np.int32)
        t1 = self.lens.astype(np.int32)
        return t0, t1

    def step_positions(self, i: int) -> np.ndarray:
        return (self.lens + i).astype(np.int32)


def _block_tables(rng: SplitMix64, blocks_per_seq: List[int], num_blocks: int,
                  max_blocks: int) -> np.ndarray:
    """Assign a random permutation of the pool to the sequences in order.

    Sequence b owns pool blocks perm[off_b : off_b + blocks_per_seq[b]];
    unused table entries are -1.
    """
    perm = rng.permutation(num_blocks)
    bt = np.full((len(blocks_per_seq), max_blocks), -1, dtype=np.int32)
    off = 0
    for b, nb in enumerate(blocks_per_seq):
        bt[b, :nb] = perm[off:off + nb]
        off += nb
    assert off == num_blocks
    return bt


def make_workload(index: int, seed: Optional[int] = None) -> Workload:
    """The five synthetic workloads, 0 (tiny) to 4 (paged GQA)."""
    seed = index if seed is None else seed
    lr = SplitMix64(derived_seed(seed, TAG_LEN))
    if index == 0:
        # tiny dense cache: 2 layers, 4 heads, head_dim 64, batch 2, capacity
        # 128; a 100-token prompt for both sequences, then 16 increments
        return Workload("tiny-dense", 2, 4, 64, 2, 128,
                        np.array([100, 100], dtype=np.int64), 16, seed=seed)
    if index == 1:
        # OPT-13B stage: 10 of 40 layers, 40 heads x 128; batch 8, capacity
        # 2048; prompts uniform 512..1024; 128 decode steps
        lens = np.array([lr.uniform_int(512, 1024) for _ in range(8)], dtype=np.int64)
        return Workload("opt13b-stage", 10, 40, 128, 8, 2048, lens, 128, seed=seed)
    if index == 2:
        # OPT-66B stage: 16 of 64 layers, 72 heads x 128; batch 8, capacity
        # 2048; fixed prompt 1000; 4 host microbatches through 2 device slots
        lens = np.full(8, 1000, dtype=np.int64)
        return Workload("opt66b-stage-swap", 16, 72, 128, 8, 2048, lens, 8,
                        microbatches=4, device_slots=2, seed=seed)
    if index == 3:
        # BLOOM-176B shard: 10 of 70 layers, 14 of 112 heads x 128; batch 16,
        # capacity 2048; ragged lengths uniform 64..2048
        lens = np.array([lr.uniform_int(64, 2048) for _ in range(16)], dtype=np.int64)
        return Workload("bloom176b-shard", 10, 14, 128, 16, 2048, lens, 0, seed=seed)
    if index == 4:
        # LLaMA-2-70B paged GQA: 20 of 80 layers, 8 KV heads x 128, block 16,
        # 32 sequences uniform 128..4096; 128 increments into tail blocks
        steps, bs = 128, 16
        lens = np.array([lr.uniform_int(128, 4096) for _ in range(32)], dtype=np.int64)
        per_seq = [int((n + steps + bs - 1) // bs) for n in lens]
        nb = int(sum(per_seq))
        max_blocks = (4096 + steps + bs - 1) // bs
        bta = _block_tables(SplitMix64(derived_seed(seed, TAG_PERM_A)), per_seq, nb, max_blocks)
        btb = _block_tables(SplitMix64(derived_seed(seed, TAG_PERM_B)), per_seq, nb, max_blocks)
        return Workload("llama2-70b-paged", 20, 8, 128, 32, max_blocks * bs, lens, steps,
                        paged=True, block_size=bs, num_blocks=nb, max_blocks=max_blocks,
                        block_table_a=bta, block_table_b=btb, seed=seed)
    raise ValueError(f"no workload {index}")


def make_paged_tables(seed: int, lens_plus: List[int], block_size: int,
                      max_blocks: int, tag: int = TAG_PERM_A):
    """Block tables for arbitrary small paged test shapes."""
    per_seq = [(int(n) + block_size - 1) // block_size for n in lens_plus]
    nb = int(sum(per_seq))
    return _block_tables(SplitMix64(derived_seed(seed, tag)), per_seq, nb, max_blocks), nb


# ---------------------------------------------------------------------------
# Device fill (GPU twin of fill_bytes)
# ---------------------------------------------------------------------------

_HERE = os.path.dirname(os.path.abspath(__file__))
LIBSYNTH_PATH = os.path.join(_HERE, "libdvsynth.so")
_libsynth = None


def libsynth():
    """Load the device fill library built from ``synth/csrc/gen_fill.hip``."""
    global _libsynth
    if _libsynth is None:
        import torch  # noqa: F401  (bind to the HIP runtime torch loaded)
        if not os.path.exists(LIBSYNTH_PATH):
            raise RuntimeError(f"{LIBSYNTH_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIBSYNTH_PATH)
        lib.dvsynth_fill.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                     ctypes.c_uint64, ctypes.c_void_p]
        lib.dvsynth_fill.restype = ctypes.c_int
        _libsynth = lib
    return _libsynth


def device_fill(ptr: int, nbytes: int, seed: int, first_byte: int = 0, stream: int = 0) -> None:
    """Fill ``nbytes`` of device memory with the counter-mode stream.

    ``ptr``, ``nbytes`` and ``first_byte`` must be multiples of 16.
    """
    rc = libsynth().dvsynth_fill(ptr, nbytes, seed & MASK64, first_byte, stream)
    if rc != 0:
        raise RuntimeError(f"dvsynth_fill failed with {rc}")

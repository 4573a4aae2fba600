"""The layer-by-layer threaded oracle (``oracle/par.py``) used by the
full-size parity tests gives the same bytes as one oracle call over the whole
layer range, for every layout, with more threads than layers and fewer."""
import numpy as np
import pytest

import oracle
import synth
from oracle import par as oracle_par
from tests.test_oracle_pins import dense_case, paged_case, rng


def _ksplit_case(seed):
    r = rng(seed)
    L, H, B, S = int(r.integers(1, 5)), int(r.integers(1, 4)), int(r.integers(1, 5)), 24
    lay = oracle.Layout(oracle.KSPLIT, L, H, 32, B, seq_cap=S, elem_bytes=2)
    buf = synth.fill_bytes(lay.storage_bytes(), seed)
    t0 = r.integers(0, S // 2, size=B).astype(np.int32)
    t1 = (t0 + r.integers(0, S // 2 + 1, size=B)).astype(np.int32)
    l0 = int(r.integers(0, L))
    return lay, buf, l0, L, t0, t1


def _cases():
    for seed in range(6):
        lay, buf, _, l0, l1, t0, t1 = dense_case(700 + seed)
        yield lay, buf, l0, l1, t0, t1
        lay, _, _, _, _, _, l0, l1, t0, t1 = paged_case(720 + seed)
        yield lay, synth.fill_bytes(lay.storage_bytes(), seed), l0, l1, t0, t1
        yield _ksplit_case(740 + seed)


@pytest.mark.parametrize("threads", [1, 3, 16])
def test_threaded_pack_and_unpack_equal_one_call(oracle_lib, threads):
    for lay, buf, l0, l1, t0, t1 in _cases():
        whole = oracle_lib.pack(lay, buf, l0, l1, t0, t1)
        par = oracle_par.pack(oracle_lib, lay, buf, l0, l1, t0, t1, threads)
        assert par.tobytes() == whole.tobytes()
        wire = synth.fill_bytes(whole.nbytes, 99)
        a = np.full(lay.storage_bytes(), 0x5C, np.uint8)
        b = a.copy()
        oracle_lib.unpack(lay, a, l0, l1, t0, t1, wire)
        oracle_par.unpack(oracle_lib, lay, b, l0, l1, t0, t1, wire, threads)
        assert a.tobytes() == b.tobytes()


@pytest.mark.parametrize("threads", [1, 4])
def test_threaded_copy_equals_one_call(oracle_lib, threads):
    for seed in range(6):
        lay, buf, (L, B, H, S, D, E), l0, l1, t0, t1 = dense_case(760 + seed)
        other = oracle.Layout(oracle.DENSE, L, H, D, B, seq_cap=S + 3, elem_bytes=E)
        a = np.full(other.storage_bytes(), 0x33, np.uint8)
        b = a.copy()
        oracle_lib.copy_ranges(lay, buf, other, a, l0, l1, t0, t1)
        oracle_par.copy_ranges(oracle_lib, lay, buf, other, b, l0, l1, t0, t1, threads)
        assert a.tobytes() == b.tobytes()


def test_parallel_host_fill_equals_serial():
    for n, first in ((1 << 20, 0), ((1 << 27) + 13, 5)):
        out = np.empty(n, np.uint8)
        synth.fill_into(out, 1234, first, threads=5)
        step = 4093  # spot positions across every chunk, plus both ends
        idx = np.concatenate([np.arange(0, n, step), [n - 1]])
        exp = synth.bytes_at(1234, (idx + first).astype(np.uint64), 1).astype(np.uint8)
        assert np.array_equal(out[idx], exp)
        assert out[:4096].tobytes() == synth.fill_bytes_numpy(4096, 1234, first).tobytes()

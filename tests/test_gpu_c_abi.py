"""The boundary from plain C on the GPU: ``tests/c/abi_parity.c`` links
libdv.so and the HIP runtime (no Python, no torch in that process), runs
every streaming entry point on its own stream and compares each result byte
for byte with the CPU oracle."""
import importlib.util
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
BIN = os.path.join(HERE, "c", "abi_parity.bin")


def built_binary() -> str:
    if not os.path.exists(BIN):  # build() makes it; build here only if it is missing
        spec = importlib.util.spec_from_file_location("abi_build",
                                                      os.path.join(HERE, "c", "build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()
    return BIN


def test_c_program_streams_bit_exact():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():  # pragma: no cover
        pytest.skip("no GPU")
    exe = built_binary()
    print("running", exe, flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi parity ok: 7 cases" in r.stdout

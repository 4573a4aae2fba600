"""Host-side AddressSanitizer and UndefinedBehaviorSanitizer run of the C
ABI's argument checks (slow; CPU only).

Builds ``libdv.so`` with the sanitizers on its host code only (each
``-fsanitize=`` goes to the host pass through ``-Xarch_host``; the GPU code
objects are built as usual) and ``tests/c/host_fuzz.cpp`` with clang++, then
runs 20 000 random descriptors, ranges and addresses through every entry
point.  Every call must return a ``dv_status`` and the sanitizers must report
nothing.  The fuzz passes made-up device addresses, which only a runtime with
no device refuses before use, so the test runs only where no GPU is visible.
"""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.slow

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2403_01876_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SOURCES = ("dv_kernels.hip", "dv_api.cpp", "dv_swapper.cpp", "dv_streamer.cpp",
           "dv_noalloc.hip")


def gpu_visible() -> bool:
    if os.path.exists("/dev/kfd"):
        return True
    r = subprocess.run([sys.executable, "-c",
                        "import torch; print(torch.cuda.device_count())"],
                       capture_output=True, text=True, timeout=600)
    return r.returncode != 0 or r.stdout.strip() not in ("", "0")


def test_argument_checks_under_host_sanitizers(tmp_path):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANG)):
        pytest.skip("ROCm compilers not installed")
    if gpu_visible():
        pytest.skip("runs only where no GPU is visible (the fuzz passes made-up addresses)")
    lib = tmp_path / "libdv.so"
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=undefined",
                "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                    "-shared", "-pthread", "-fvisibility=hidden", "-Xclang", "-target-feature",
                    "-Xclang", "-packed-fp32-ops", *host_san, "-x", "hip",
                    *[os.path.join(CSRC, s) for s in SOURCES], "-o", str(lib)],
                   check=True, capture_output=True, timeout=900)
    exe = tmp_path / "host_fuzz"
    subprocess.run([CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "tests", "c", "host_fuzz.cpp"), f"-L{tmp_path}", "-ldv",
                    f"-Wl,-rpath,{tmp_path}", "-o", str(exe)],
                   check=True, capture_output=True, timeout=300)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    for seed in ("0x1", "0xD474"):
        r = subprocess.run([str(exe), "10000", seed], capture_output=True, text=True, env=env,
                           timeout=900)
        report = r.stdout + r.stderr
        assert r.returncode == 0, report[-4000:]
        assert "runtime error" not in report and "AddressSanitizer" not in report, report[-4000:]
        assert "10000 iterations, 0 failures" in r.stdout
        tally = {ln.split()[0]: [int(x) for x in ln.split()[2::2]]
                 for ln in r.stdout.splitlines() if ln.startswith("dv_")}
        # the random calls reach every outcome that matters: sizes computed,
        # each kind of refusal, and launches handed to the (device-less)
        # runtime, which refuses them
        assert tally["dv_packed_bytes"][0] > 0 and tally["dv_cache_bytes"][0] > 0
        for name in ("dv_stream_out_prompt", "dv_stream_out_token", "dv_stream_in",
                     "dv_stream_in_noalloc"):
            ok, inv, rng, spc, uns, hip = tally[name]
            assert inv > 0 and rng > 0 and hip > 0, (name, tally[name])
        assert tally["dv_stream_out_prompt"][3] > 0  # destination too small
        assert sum(tally["dv_swap_out"][1:]) > 0 and tally["dv_swapper_create"][1] > 0

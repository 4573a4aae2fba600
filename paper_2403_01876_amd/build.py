"""Builds ``libdv.so`` (the C-ABI streaming library) and ``libdvsynth.so``
(the seeded device fill used by tests and the benchmark) for gfx950."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIBDV = os.path.join(PKG, "libdv.so")
LIBSYNTH = os.path.join(ROOT, "synth", "libdvsynth.so")
LIBBASE = os.path.join(PKG, "libdv_baseline.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# -packed-fp32-ops: keep the compiler from emitting packed fp32 instructions
# (none are needed; the kernels move bits only).
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-pthread",
             "-fvisibility=hidden",
             "-Wall", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build_libdv(out: str = LIBDV) -> str:
    srcs = [os.path.join(PKG, "csrc", f) for f in ("dv_kernels.hip", "dv_api.cpp",
                                                    "dv_swapper.cpp", "dv_streamer.cpp",
                                                    "dv_noalloc.hip")]
    tmp = out + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-x", "hip", *srcs, "-o", tmp])
    os.replace(tmp, out)
    return out


def build_baseline(out: str = LIBBASE) -> str:
    """The per-region copy baseline the benchmark compares against."""
    src = os.path.join(PKG, "csrc", "dv_baseline.cpp")
    tmp = out + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-x", "hip", src, "-L" + PKG, "-ldv",
          "-Wl,-rpath,$ORIGIN", "-o", tmp])
    os.replace(tmp, out)
    return out


def build_libsynth(out: str = LIBSYNTH) -> str:
    src = os.path.join(ROOT, "synth", "csrc", "gen_fill.hip")
    tmp = out + ".tmp"
    _run([HIPCC, *HIP_FLAGS, src, "-o", tmp])
    os.replace(tmp, out)
    return out


def build_all() -> None:
    build_libdv()
    build_baseline()
    build_libsynth()


if __name__ == "__main__":
    build_all()
    sys.exit(0)

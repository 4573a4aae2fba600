"""Builds ``abi_parity.bin``, the plain-C GPU test of the boundary, against
the in-tree libdv.so, the oracle and the host generator (run by
``__graft_entry__.build()``; the test builds it itself if it is missing)."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
OUT = os.path.join(HERE, "abi_parity.bin")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(out: str = OUT) -> str:
    libdirs = [os.path.join(ROOT, d) for d in ("paper_2403_01876_amd", "oracle", "synth")]
    rpath = ":".join(["$ORIGIN/../../paper_2403_01876_amd", "$ORIGIN/../../oracle",
                      "$ORIGIN/../../synth", os.path.join(ROCM, "lib")])
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "oracle"), os.path.join(HERE, "abi_parity.c"),
           "-o", out + ".tmp"]
    for d in libdirs:
        cmd += ["-L", d]
    cmd += ["-ldv", "-ldvoracle", "-ldvsynth_host", "-L", os.path.join(ROCM, "lib"),
            "-lamdhip64", "-Wl,-rpath," + rpath]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build()

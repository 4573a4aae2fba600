"""bench.py's host-side contract without a GPU: it refuses more than one
GPU with a message, and the counted-traffic figure is read only while the
kernel sources hash to the value the committed counter summary records."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_counted_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    for which in ("traffic_bytes_per_launch", "traffic_bytes_per_launch_unpack"):
        t = bench.counted_traffic(bench.DENSE_TRAFFIC, which)
        assert t is None or 2 * 1282252800 <= t <= 1.01 * 2 * 1282252800
    # a summary whose recorded hash does not match the sources gives None
    prof = tmp_path / "profiles"
    prof.mkdir()
    src = open(os.path.join(ROOT, "profiles", "dense_runs_hbm_traffic_opt13b_stage.md")).read()
    lines = [("kernel_source_sha256: " + "0" * 64) if ln.startswith("kernel_source_sha256:")
             else ln for ln in src.splitlines()]
    (prof / "dense_runs_hbm_traffic_opt13b_stage.md").write_text("\n".join(lines) + "\n")
    csrc = tmp_path / "paper_2403_01876_amd" / "csrc"
    csrc.mkdir(parents=True)
    for f in ("dv_kernels.hip", "dv_internal.h"):
        (csrc / f).write_bytes(open(os.path.join(ROOT, "paper_2403_01876_amd", "csrc", f),
                                    "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.counted_traffic(bench.DENSE_TRAFFIC, "traffic_bytes_per_launch") is None
    # and a missing summary gives None too
    (prof / "dense_runs_hbm_traffic_opt13b_stage.md").unlink()
    assert bench.counted_traffic(bench.DENSE_TRAFFIC, "traffic_bytes_per_launch") is None


def test_block_order_is_a_permutation_of_the_pool():
    """The block-order ceiling copies every block of the LLaMA-2-70B pool
    once: table A's order, slab by slab, is a permutation of all blocks."""
    import numpy as np

    import synth
    w = synth.make_workload(4)
    order = bench.block_order(w, w.block_table_a)
    n = 2 * w.layers * w.num_blocks
    assert order.size == n and np.array_equal(np.sort(order), np.arange(n))
    # the first slab visits sequence 0's blocks first, in table order
    k = int((w.block_table_a[0] >= 0).sum())
    assert np.array_equal(order[:k], w.block_table_a[0, :k])

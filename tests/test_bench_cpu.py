"""bench.py's host-side accounting, on the CPU: every node of every workload
bench.py offers gets finite algorithmic bytes and flops (fused nodes count
their inputs and outputs, not the intermediates they keep on chip), and the
GPU-count guard refuses more than one GPU."""
import math
import os
import subprocess
import sys

import pytest

import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("key", sorted(bench.WORKLOADS))
def test_node_work_covers_every_node(key):
    from paper_1907_01989_amd import engine
    net, batch = bench.WORKLOADS[key]
    desc = workloads.WORKLOADS[net](min(batch, 2))
    nodes = engine.Plan(desc, bind=False).nodes()
    shapes = bench.tensor_shapes(desc, nodes)
    for i, n in enumerate(nodes):
        flops, byts, bound = bench.node_work(desc, nodes, shapes, i)
        assert math.isfinite(flops) and math.isfinite(byts) and bound in ("hbm", "mfma"), (i, n["kind"])
        if n["tensor"] >= 0:
            assert byts > 0, (i, n["kind"])


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in (r.stdout + r.stderr)

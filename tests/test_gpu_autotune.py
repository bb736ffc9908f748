"""Kernel configuration candidates and the plan-time autotuner.

Every candidate configuration of a node (GEMM tile shapes and kernels,
depthwise rows per thread) accumulates each output in the same order, so
each must reproduce the default configuration's node output bit for bit; the
default itself is held to the oracle by the operator and network tests.  An
autotuned plan must then reproduce the untuned outputs exactly.
"""
import numpy as np
import pytest

import workloads

from gpu_util import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("net,batch", [("mobilenet_v2", 2), ("deeplab", 1)])
def test_every_candidate_matches_default(net, batch):
    import torch
    from paper_1907_01989_amd import _binding as B
    from paper_1907_01989_amd import engine

    desc = workloads.WORKLOADS[net](batch)
    plan = engine.Plan(desc, materialize_all=True)
    xs = plan.input_tensors()
    outs = plan.run(xs)
    torch.cuda.synchronize()
    nodes = plan.nodes()
    cfgs = plan.node_configs()
    ref = {i: plan.read_node(i)[1].cpu().numpy() for i, (_, k, _) in enumerate(cfgs) if k > 1}
    tried = 0
    for i, (_, k, _) in enumerate(cfgs):
        for c in range(1, k):
            B.mgi_plan_set_node_config(plan.handle, i, c)
            name = plan.node_configs()[i][2]
            log(f"[case] {net} b{batch} node {i} ({nodes[i]['kind']}) config {c} {name} shape {nodes[i]['shape']}")
            plan.run(xs, outs)
            got = plan.read_node(i)[1].cpu().numpy()
            np.testing.assert_array_equal(got, ref[i], err_msg=f"node {i} config {name}")
            tried += 1
        if k > 1:
            B.mgi_plan_set_node_config(plan.handle, i, 0)
    assert tried > 100
    plan.close()


@pytest.mark.parametrize("net,batch", [("mobilenet_v1", 4), ("mobilenet_v2", 2)])
def test_autotuned_plan_reproduces_default(net, batch):
    import torch
    from paper_1907_01989_amd import engine

    desc = workloads.WORKLOADS[net](batch)
    log(f"[case] autotune {net} b{batch}")
    plan = engine.Plan(desc)
    xs = plan.input_tensors()
    ref = [o.cpu().numpy() for o in plan.run(xs)]
    torch.cuda.synchronize()
    plan.autotune(xs, reps=3)
    chosen = [name for _, k, name in plan.node_configs() if k > 1]
    log(f"[case] chosen {chosen}")
    got = [o.cpu().numpy() for o in plan.run(xs)]
    torch.cuda.synchronize()
    for g, r in zip(got, ref):
        np.testing.assert_array_equal(g, r)
    plan.close()

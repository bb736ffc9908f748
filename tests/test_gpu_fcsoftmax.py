"""Fully connected layer fused with the softmax that alone reads its logits.

The FC kernel's workgroups count themselves in per tile of rows and the last
one of a tile runs the softmax of its rows with the standalone softmax
kernel's row routine, so every configuration of the node (16, 32 or 64 rows
per workgroup, 4 or 8 K-steps per load batch; the split form: the FC into the
logits, then the softmax kernel) and the unfused plan agree bit for bit, and
each case is held to the oracle at the chained-layer bound.  The arrival
counters must be back at zero after every run: one plan is run several times,
switching configurations (and so the row tiling of the counters) between runs.
Shapes: v1's and v2's heads at batch 64 and 1, a ragged last row tile,
class counts that end inside a 16-column block, rows longer than 1024 (the
softmax's looped path), a K tail, and bf16 storage.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads import ACT_NONE, NetBuilder

from gpu_util import check_layer, log, run_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # n, K, classes
    (64, 1024, 1000),    # MobileNet-v1 head
    (1, 1280, 1000),     # MobileNet-v2 head, batch 1
    (17, 256, 1001),     # ragged last row tile, partial column block
    (5, 64, 2000),       # rows longer than 1024
    (3, 40, 10),         # K tail, one column block
    (100, 512, 37),      # seven 16-row tiles
]


def head_graph(n, K, classes):
    g = NetBuilder(seed=K + classes + n)
    x = g.activation(g.input(n, 1, 1, K, -1, 1), ACT_NONE)
    y = g.softmax(g.fc(x, classes))
    g.mark_output(y)
    return g.graph(f"fcsoftmax_{n}_k{K}_c{classes}"), y


def fused_index(plan):
    kinds = [k["kind"] for k in plan.nodes()]
    idx = [i for i, k in enumerate(kinds) if k == "fc_softmax"]
    assert len(idx) == 1 and "softmax" not in kinds, kinds
    return idx[0]


@pytest.mark.parametrize("n,K,classes", CASES)
def test_fused_fc_softmax(n, K, classes):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = head_graph(n, K, classes)
    plan = engine.Plan(desc, bind=False)
    idx = fused_index(plan)
    ncfg = plan.node_configs()[idx][1]
    names = []
    for cf in range(ncfg):
        B.mgi_plan_set_node_config(plan.handle, idx, cf)
        names.append(plan.node_configs()[idx][2])
    log(f"[case] {desc['name']} configurations {names}")
    assert any(nm.startswith("split") for nm in names) and any(nm.startswith("fc") for nm in names)
    outs = []
    for cf in range(ncfg):
        _, o, _ = run_gpu(desc, materialize_all=False, configs={idx: cf})
        outs.append(o[0])
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_softmax=False)
    for nm, o in zip(names, outs):
        assert np.array_equal(o, plain[0]), nm
    ref = oracle.run_graph(desc, keep=[y])[y]
    ok, msg = check_layer("probabilities", outs[0], ref.reshape(outs[0].shape))
    assert ok, msg
    np.testing.assert_allclose(outs[0].sum(axis=-1), 1.0, rtol=1e-5)


def test_counters_return_to_zero():
    import torch
    from paper_1907_01989_amd import engine, _binding as B
    desc, _ = head_graph(100, 512, 1000)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_softmax=False)
    plan = engine.Plan(desc)
    idx = fused_index(plan)
    ncfg = plan.node_configs()[idx][1]
    xs = plan.input_tensors()
    log(f"[case] {desc['name']} repeated runs over {ncfg} configurations")
    for rep in range(3):
        for cf in range(ncfg):
            B.mgi_plan_set_node_config(plan.handle, idx, cf)
            out = plan.run(xs)[0]
            torch.cuda.synchronize()
            np.testing.assert_array_equal(out.cpu().numpy(), plain[0], err_msg=f"run {rep} config {cf}")


def test_fused_fc_softmax_bf16():
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = head_graph(20, 1280, 1000)
    bdesc = workloads.as_bf16_graph(desc)
    plan = engine.Plan(bdesc, bind=False, dtype=B.DTYPE_BF16)
    idx = fused_index(plan)
    ncfg = plan.node_configs()[idx][1]
    log(f"[case] {desc['name']} bf16 ({ncfg} configurations)")
    _, plain, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_softmax=False)
    for cf in range(ncfg):
        _, fused, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, configs={idx: cf})
        np.testing.assert_array_equal(fused[0], plain[0], err_msg=f"configuration {cf}")
    ref = oracle.run_graph(bdesc, keep=[y], store_bf16=True)[y]
    ok, msg = check_layer("bf16 probabilities", plain[0], ref.reshape(plain[0].shape))
    assert ok, msg


@pytest.mark.parametrize("net", ["mobilenet_v1", "mobilenet_v2"])
def test_fused_fc_softmax_network(net):
    from paper_1907_01989_amd import engine
    desc = workloads.WORKLOADS[net](64)
    kinds = [k["kind"] for k in engine.Plan(desc, bind=False).nodes()]
    assert kinds[-2:] == ["pw_pool", "fc_softmax"], kinds[-3:]
    log(f"[case] {net} b64 fc->softmax fused vs unfused")
    _, fused, _ = run_gpu(desc, materialize_all=False)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_softmax=False)
    for a, b in zip(fused, plain):
        np.testing.assert_array_equal(a, b)

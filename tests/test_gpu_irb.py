"""MobileNet-v2's inverted residual block as one node: pointwise expansion,
depthwise 3x3 and linear projection (with the residual add where the block
has one) in one kernel, the expanded and depthwise tensors kept in LDS.

Every configuration of the node -- the block kernel's tilings, the fused
pointwise -> depthwise kernel followed by the projection GEMM, and the three
separate kernels -- must agree bit for bit with the unfused plan, since each
form rounds every stored intermediate alike and accumulates the projection
over K in the GEMM kernels' order.  Every case is also held to the oracle at
the chained-layer bound.  Shapes: every MobileNet-v2 block shape at batch 64
on the 14x14 and 7x7 planes, the wider planes at small batches, expansions
that end in half a 16-channel block, a projection with three output blocks,
an odd plane and batch 1.
"""
import numpy as np
import pytest

import oracle
from workloads import ACT_NONE, ACT_RELU6, NetBuilder

from gpu_util import check_layer, log, run_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # n, h, w, cin, expanded channels, cout, stride, residual
    (3, 112, 112, 16, 96, 24, 2, False),     # v2 b2
    (3, 56, 56, 24, 144, 24, 1, True),       # v2 b3
    (3, 56, 56, 24, 144, 32, 2, False),      # v2 b4
    (5, 28, 28, 32, 192, 32, 1, True),       # v2 b5, b6
    (5, 28, 28, 32, 192, 64, 2, False),      # v2 b7
    (64, 14, 14, 64, 384, 64, 1, True),      # v2 b8 .. b10
    (64, 14, 14, 64, 384, 96, 1, False),     # v2 b11
    (64, 14, 14, 96, 576, 96, 1, True),      # v2 b12, b13
    (64, 14, 14, 96, 576, 160, 2, False),    # v2 b14
    (64, 7, 7, 160, 960, 160, 1, True),      # v2 b15, b16
    (64, 7, 7, 160, 960, 320, 1, False),     # v2 b17
    (3, 13, 15, 24, 72, 24, 1, True),        # odd plane, expansion of 4.5 blocks
    (2, 28, 28, 40, 120, 48, 2, False),      # three output blocks, 7.5-block expansion
    (1, 14, 14, 64, 384, 64, 1, True),       # batch 1
]


def block_graph(n, h, w, cin, cexp, cout, s, res):
    g = NetBuilder(seed=cin + cexp + cout + s + h)
    x = g.activation(g.input(n, h, w, cin, -1, 1), ACT_NONE)
    e = g.conv(x, cexp, 1, act=ACT_RELU6)
    d = g.dw(e, 3, s=s, act=ACT_RELU6)
    y = g.conv(d, cout, 1, act=ACT_NONE)
    if res:
        y = g.add(y, x)
    g.mark_output(y)
    return g.graph(f"irb_{n}x{h}x{w}_c{cin}_e{cexp}_o{cout}_s{s}{'_res' if res else ''}"), y


@pytest.mark.parametrize("n,h,w,cin,cexp,cout,s,res", CASES)
def test_block(n, h, w, cin, cexp, cout, s, res):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = block_graph(n, h, w, cin, cexp, cout, s, res)
    plan = engine.Plan(desc, bind=False, fuse_irb=2)
    idx = [i for i, k in enumerate(plan.nodes()) if k["kind"] == "irb"]
    kinds = [k["kind"] for k in plan.nodes()]
    assert len(idx) == 1 and not {"pw_gemm", "pw_dw", "dw_conv"} & set(kinds), kinds
    ncfg = plan.node_configs()[idx[0]][1]
    names = []
    for c in range(ncfg):
        B.mgi_plan_set_node_config(plan.handle, idx[0], c)
        names.append(plan.node_configs()[idx[0]][2])
    log(f"[case] {desc['name']} ({ncfg} configurations: {', '.join(names)})")
    assert any(nm.startswith("irb") for nm in names) and any(nm.startswith("split3") for nm in names)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_irb=False, fuse_pwdw=False)
    for c in range(ncfg):
        _, o, _ = run_gpu(desc, materialize_all=False, configs={idx[0]: c}, fuse_irb=2)
        np.testing.assert_array_equal(o[0], plain[0], err_msg=f"configuration {c} ({names[c]})")
    ref = oracle.run_graph(desc, keep=[y])[y]
    ok, msg = check_layer("block output", plain[0], ref.reshape(plain[0].shape))
    log("  " + msg)
    assert ok, msg


def test_block_bf16():
    import workloads
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = block_graph(16, 14, 14, 64, 384, 64, 1, True)
    bdesc = workloads.as_bf16_graph(desc)
    plan = engine.Plan(bdesc, bind=False, fuse_irb=2, dtype=B.DTYPE_BF16)
    idx = [i for i, k in enumerate(plan.nodes()) if k["kind"] == "irb"]
    ncfg = plan.node_configs()[idx[0]][1]
    log(f"[case] {desc['name']} bf16 ({ncfg} configurations)")
    _, plain, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_irb=False, fuse_pwdw=False)
    for c in range(ncfg):
        _, o, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_irb=2, configs={idx[0]: c})
        np.testing.assert_array_equal(o[0], plain[0], err_msg=f"configuration {c}")
    ref = oracle.run_graph(bdesc, keep=[y], store_bf16=True)[y]
    ok, msg = check_layer("block bf16 output", plain[0], ref.reshape(plain[0].shape))
    assert ok, msg


@pytest.mark.parametrize("batch", [1, 64])
def test_block_network(batch):
    """MobileNet-v2 with the block nodes (fuse_irb = 1) equals the plan
    without them bit for bit."""
    import workloads
    desc = workloads.mobilenet_v2(batch)
    log(f"[case] mobilenet_v2 b{batch} block nodes vs unfused projections")
    _, fused, _ = run_gpu(desc, materialize_all=False, fuse_irb=True)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_irb=False)
    for a, b in zip(fused, plain):
        np.testing.assert_array_equal(a, b)

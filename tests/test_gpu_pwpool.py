"""Pointwise convolution fused with the global average pool that alone reads
its output.

The pooled GEMM rounds every output value to the storage type, as the stored
tensor would be, and sums each image's pixels in the pool kernel's order, so
every configuration of the node (M-tiles of 64 or 128 rows holding whole
images, 64 or 128 channels; the split form: the GEMM, then the pool kernel,
through a scratch tensor) and the unfused plan agree bit for bit; each case
is also held to the oracle at the chained-layer bound.  Planes of 49
(MobileNet's 7x7), 64, 16 and 1 pixels, channel counts with partial blocks
and slices, a linear convolution, K tails, bf16 storage and batch 1.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads import ACT_NONE, ACT_RELU6, NetBuilder

from gpu_util import check_layer, log, run_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # n, h, w, K, C, activation
    (64, 7, 7, 1024, 1024, ACT_RELU6),   # MobileNet-v1 pw13 -> pool
    (9, 7, 7, 320, 1280, ACT_RELU6),     # v2 head shape, odd batch
    (5, 8, 8, 72, 40, ACT_NONE),         # 64-pixel planes, K tail, partial block and slice, linear
    (7, 4, 4, 64, 24, ACT_RELU6),        # 8 images per 128-row tile
    (3, 1, 1, 48, 16, ACT_RELU6),        # 1x1 planes
    (1, 7, 7, 256, 128, ACT_RELU6),      # batch 1
    (2, 8, 8, 264, 40, ACT_NONE),        # weight-slab pooled tiles: K tail, partial block, 64-pixel planes
]


def pair_graph(n, h, w, K, C, act):
    g = NetBuilder(seed=K + C + h)
    x = g.activation(g.input(n, h, w, K, -1, 1), ACT_NONE)
    c = g.conv(x, C, 1, act=act)
    y = g.gap(c)
    g.mark_output(y)
    return g.graph(f"pwpool_{n}x{h}x{w}_k{K}_c{C}"), y


@pytest.mark.parametrize("n,h,w,K,C,act", CASES)
def test_fused_pool_pair(n, h, w, K, C, act):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = pair_graph(n, h, w, K, C, act)
    plan = engine.Plan(desc, bind=False, fuse_pool=2)
    kinds = [k["kind"] for k in plan.nodes()]
    idx = [i for i, k in enumerate(kinds) if k == "pw_pool"]
    assert len(idx) == 1 and "global_avgpool" not in kinds, kinds
    ncfg = plan.node_configs()[idx[0]][1]
    names = []
    for cf in range(ncfg):
        B.mgi_plan_set_node_config(plan.handle, idx[0], cf)
        names.append(plan.node_configs()[idx[0]][2])
    log(f"[case] {desc['name']} configurations {names}")
    assert any(nm.startswith("split") for nm in names) and any(nm.startswith("pool") for nm in names)
    outs = []
    for cf in range(ncfg):
        _, o, _ = run_gpu(desc, materialize_all=False, configs={idx[0]: cf}, fuse_pool=2)
        outs.append(o[0])
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_pool=False)
    for nm, o in zip(names, outs):
        assert np.array_equal(o, plain[0]), nm
    ref = oracle.run_graph(desc, keep=[y])[y]
    ok, msg = check_layer("fused output", outs[0], ref.reshape(outs[0].shape))
    assert ok, msg


@pytest.mark.parametrize("n,c", [(16, 320), (1, 64)])
def test_fused_pool_pair_bf16(n, c):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = pair_graph(n, 7, 7, 256, c, ACT_RELU6)
    bdesc = workloads.as_bf16_graph(desc)
    plan = engine.Plan(bdesc, bind=False, fuse_pool=2, dtype=B.DTYPE_BF16)
    idx = [i for i, k in enumerate(plan.nodes()) if k["kind"] == "pw_pool"]
    assert len(idx) == 1
    ncfg = plan.node_configs()[idx[0]][1]
    log(f"[case] {desc['name']} bf16 ({ncfg} configurations)")
    _, plain, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_pool=False)
    for c in range(ncfg):
        _, fused, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_pool=2, configs={idx[0]: c})
        np.testing.assert_array_equal(fused[0], plain[0], err_msg=f"configuration {c}")
    ref = oracle.run_graph(bdesc, keep=[y], store_bf16=True)[y]
    ok, msg = check_layer("fused bf16 output", plain[0], ref.reshape(plain[0].shape))
    assert ok, msg


@pytest.mark.parametrize("net", ["mobilenet_v1", "mobilenet_v2"])
def test_fused_pool_network(net):
    from paper_1907_01989_amd import engine
    desc = workloads.WORKLOADS[net](64)
    kinds = [k["kind"] for k in engine.Plan(desc, bind=False).nodes()]
    assert kinds[-2:] == ["pw_pool", "fc_softmax"], kinds[-3:]
    log(f"[case] {net} b64 pointwise->pool fused vs unfused")
    _, fused, _ = run_gpu(desc, materialize_all=False)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_pool=False)
    for a, b in zip(fused, plain):
        np.testing.assert_array_equal(a, b)

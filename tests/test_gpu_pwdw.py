"""Pointwise convolution fused with the depthwise 3x3 convolution that reads
its output (whole-image tiles, depthwise step on the matrix cores).

The fused kernel accumulates K in the GEMM kernels' order and each depthwise
output with the depthwise kernel's tap order, rounding and activation, so
every configuration of the node -- both tile widths (64 and 128 channels) and
the split form (the two separate kernels through a scratch tensor) -- and
the unfused plan must agree bit for bit.  Every case is also held to the
oracle at the chained-layer bound.  Shapes cover both strides, TF-SAME and
symmetric padding, whole-image tiles (several images per tile, ragged last
tile) and row bands (every v1 band shape, 2- to 7-row bands, odd planes with a
short last band),
partial channel tiles (v2's 96 and 144 channels), channel counts that end in
half a 16-channel block, K tails and single slices, and batch 1.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads import ACT_NONE, ACT_RELU, ACT_RELU6, NetBuilder

from gpu_util import check_layer, log, run_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # n, h, w, K (pointwise inputs), C (channels), stride, pads (None = TF-SAME), dw activation
    (64, 14, 14, 256, 512, 1, None, ACT_RELU6),     # v1 pw6 -> dw7
    (64, 14, 14, 512, 512, 2, None, ACT_RELU6),     # v1 pw11 -> dw12 (pt 0, pb 1)
    (64, 7, 7, 512, 1024, 1, None, ACT_RELU6),      # v1 pw12 -> dw13, 5 images per tile
    (3, 13, 15, 40, 64, 1, None, ACT_NONE),         # ragged plane, K tail, linear
    (5, 9, 11, 24, 128, 2, None, ACT_RELU),         # odd sizes at stride 2 (pt 1)
    (2, 16, 16, 64, 64, 2, (1, 1, 1, 1), ACT_RELU6),  # symmetric padding at stride 2
    (1, 15, 15, 8, 64, 1, None, ACT_RELU6),         # 15 x 15 (widest row at stride 1), one K slice, batch 1
    (7, 4, 4, 32, 192, 1, None, ACT_RELU6),         # 16 images per tile
    # batch 1 at v1's 14 x 14 and 7 x 7 layers (16- and 32-channel image tiles)
    (1, 14, 14, 512, 512, 1, None, ACT_RELU6),      # v1 pw7 -> dw8
    (1, 14, 14, 512, 512, 2, None, ACT_RELU6),      # v1 pw11 -> dw12
    (1, 7, 7, 512, 1024, 1, None, ACT_RELU6),       # v1 pw12 -> dw13
    (1, 14, 14, 160, 120, 1, None, ACT_NONE),       # 15 slices: last tile one slice short, K tail
    # row bands (a halo row computed by both neighbouring bands)
    (3, 112, 112, 32, 64, 2, None, ACT_RELU6),      # v1 pw1 -> dw2
    (2, 56, 56, 64, 128, 1, None, ACT_RELU6),       # v1 pw2 -> dw3
    (2, 56, 56, 128, 128, 2, None, ACT_RELU6),      # v1 pw3 -> dw4
    (3, 28, 28, 128, 256, 1, None, ACT_RELU6),      # v1 pw4 -> dw5
    (3, 28, 28, 256, 256, 2, None, ACT_RELU6),      # v1 pw5 -> dw6
    (2, 56, 56, 24, 144, 1, None, ACT_RELU6),       # v2 expansion, partial channel tile (9 blocks)
    (2, 112, 112, 16, 96, 2, None, ACT_RELU6),      # v2 expansion at 112, 6 blocks
    (2, 27, 29, 40, 80, 1, None, ACT_NONE),         # odd plane, last band short, K tail
    (2, 55, 53, 24, 64, 2, (1, 1, 1, 1), ACT_RELU6),  # odd plane at stride 2, symmetric padding
    (2, 28, 28, 40, 72, 1, None, ACT_RELU6),        # 9 output slices in bands (channels = 8 mod 16)
    (2, 45, 45, 40, 96, 1, None, ACT_RELU6),        # 7-row bands with a 3-row last band, K tail
]


def pair_graph(n, h, w, K, C, s, pads, dw_act):
    g = NetBuilder(seed=K + C + s + h)
    x = g.activation(g.input(n, h, w, K, -1, 1), ACT_NONE)
    p = g.conv(x, C, 1, act=ACT_RELU6)
    y = g.dw(p, 3, s=s, act=dw_act, pads=pads)
    g.mark_output(y)
    return g.graph(f"pwdw_{n}x{h}x{w}_k{K}_c{C}_s{s}"), y


def fused_nodes(plan):
    return [i for i, k in enumerate(plan.nodes()) if k["kind"] == "pw_dw"]


@pytest.mark.parametrize("n,h,w,K,C,s,pads,act", CASES)
def test_fused_pair(n, h, w, K, C, s, pads, act):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = pair_graph(n, h, w, K, C, s, pads, act)
    plan = engine.Plan(desc, bind=False, fuse_pwdw=2)
    idx = fused_nodes(plan)
    assert len(idx) == 1 and "dw_conv" not in [k["kind"] for k in plan.nodes()]
    ncfg = plan.node_configs()[idx[0]][1]
    log(f"[case] {desc['name']} ({ncfg} configurations)")
    outs = []
    for c in range(ncfg):
        _, o, _ = run_gpu(desc, materialize_all=False, configs={idx[0]: c}, fuse_pwdw=2)
        outs.append(o[0])
    names = []
    for c in range(ncfg):
        B.mgi_plan_set_node_config(plan.handle, idx[0], c)
        names.append(plan.node_configs()[idx[0]][2])
    fused_outs = [o for o, n in zip(outs, names) if n.startswith(("img", "band"))]
    split_outs = [o for o, n in zip(outs, names) if n.startswith("split")]
    assert len(fused_outs) >= 1 and len(split_outs) >= 1, names
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_pwdw=False)
    for o in fused_outs + split_outs:
        np.testing.assert_array_equal(o, plain[0])
    fused = fused_outs[0]
    ref = oracle.run_graph(desc, keep=[y])[y]
    ok, msg = check_layer("fused output", fused, ref.reshape(fused.shape))
    assert ok, msg


@pytest.mark.parametrize("n,h,w,K,C,s", [(16, 14, 14, 128, 256, 1),   # image tiles of 16..128 channels
                                         (1, 56, 56, 64, 128, 1),     # 16..128-channel row bands
                                         (1, 7, 7, 512, 1024, 1),     # batch-1 7x7 tiles
                                         (9, 7, 7, 256, 256, 1),      # 7x7 tiles capped at four images
                                         (16, 14, 14, 128, 256, 2)])  # four fragments per wave at stride 2
def test_fused_pair_bf16(n, h, w, K, C, s):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = pair_graph(n, h, w, K, C, s, None, ACT_RELU6)
    bdesc = workloads.as_bf16_graph(desc)
    plan = engine.Plan(bdesc, bind=False, fuse_pwdw=2, dtype=B.DTYPE_BF16)
    idx = fused_nodes(plan)
    ncfg = plan.node_configs()[idx[0]][1]
    log(f"[case] {desc['name']} bf16 ({ncfg} configurations)")
    _, plain, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_pwdw=False)
    for c in range(ncfg):
        _, fused, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_pwdw=2, configs={idx[0]: c})
        np.testing.assert_array_equal(fused[0], plain[0], err_msg=f"configuration {c}")
    ref = oracle.run_graph(bdesc, keep=[y], store_bf16=True)[y]
    ok, msg = check_layer("fused bf16 output", plain[0], ref.reshape(plain[0].shape))
    assert ok, msg


@pytest.mark.parametrize("net", ["mobilenet_v1", "mobilenet_v2"])
def test_fused_network(net):
    from paper_1907_01989_amd import engine
    desc = workloads.WORKLOADS[net](64)
    kinds = [k["kind"] for k in engine.Plan(desc, bind=False).nodes()]
    assert kinds.count("pw_dw") >= 7
    log(f"[case] {net} b64 pointwise->depthwise fused vs unfused")
    _, fused, _ = run_gpu(desc, materialize_all=False)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_pwdw=False)
    for a, b in zip(fused, plain):
        np.testing.assert_array_equal(a, b)

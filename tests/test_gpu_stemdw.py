"""The stem convolution fused with the stride-1 depthwise 3x3 convolution
that reads its output.

The fused kernel computes the stem rows a band needs with the stem kernel's
MFMA, bias and activation and each depthwise output in the depthwise
kernel's tap order and rounding, so every configuration of the node (4- and
2-row bands, and the split form: the two separate kernels through a scratch
tensor) and the unfused plan agree bit for bit; each case is also held to
the oracle at the chained-layer bound.  Shapes cover the MobileNet stem
(224 -> 112, TF-SAME), odd inputs with a short last band, symmetric padding,
1 to 4 channel blocks with a partial output slice (24 channels), fp16 and
fp32 graph inputs, a linear depthwise, bf16 storage and batch 1.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads import ACT_NONE, ACT_RELU, ACT_RELU6, DTYPE_FP16, NetBuilder

from gpu_util import check_layer, log, run_gpu

pytestmark = pytest.mark.gpu

DTYPE_FP32 = 2

CASES = [
    # n, h, w, c (stem outputs), stem pads (None = TF-SAME), dw pads, dw activation, input dtype
    (3, 224, 224, 32, None, None, ACT_RELU6, DTYPE_FP16),          # MobileNet stem -> dw1
    (2, 224, 224, 32, None, None, ACT_RELU6, DTYPE_FP32),          # fp32 graph input
    (1, 97, 113, 16, None, None, ACT_NONE, DTYPE_FP16),            # odd input, one block, linear, batch 1
    (2, 57, 61, 24, (1, 1, 1, 1), None, ACT_RELU, DTYPE_FP16),     # symmetric stem pads, 3 of 4 slices stored
    (2, 66, 50, 48, None, (0, 2, 2, 0), ACT_RELU6, DTYPE_FP16),    # three blocks, depthwise pads 0/2
    (2, 40, 44, 64, None, None, ACT_RELU6, DTYPE_FP32),            # four blocks
]


def pair_graph(n, h, w, c, spads, dpads, dw_act, dtype):
    g = NetBuilder(seed=c + h + w)
    x = g.input(n, h, w, 3, 0, 1, dtype=dtype)
    s = g.conv(x, c, 3, s=2, act=ACT_RELU6, pads=spads)
    y = g.dw(s, 3, s=1, act=dw_act, pads=dpads)
    g.mark_output(y)
    return g.graph(f"stemdw_{n}x{h}x{w}_c{c}_t{dtype}"), y


def fused_nodes(plan):
    return [i for i, k in enumerate(plan.nodes()) if k["kind"] == "stem_dw"]


@pytest.mark.parametrize("n,h,w,c,spads,dpads,act,dtype", CASES)
def test_fused_stem_pair(n, h, w, c, spads, dpads, act, dtype):
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = pair_graph(n, h, w, c, spads, dpads, act, dtype)
    plan = engine.Plan(desc, bind=False, fuse_stemdw=2)
    idx = fused_nodes(plan)
    kinds = [k["kind"] for k in plan.nodes()]
    assert len(idx) == 1 and "dw_conv" not in kinds and "conv_stem" not in kinds, kinds
    ncfg = plan.node_configs()[idx[0]][1]
    names = []
    for cf in range(ncfg):
        B.mgi_plan_set_node_config(plan.handle, idx[0], cf)
        names.append(plan.node_configs()[idx[0]][2])
    log(f"[case] {desc['name']} configurations {names}")
    assert "split" in names and any(nm.startswith("band") for nm in names), names
    outs = []
    for cf in range(ncfg):
        _, o, _ = run_gpu(desc, materialize_all=False, configs={idx[0]: cf}, fuse_stemdw=2)
        outs.append(o[0])
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_stemdw=False)
    kinds_plain = [k["kind"] for k in engine.Plan(desc, bind=False, fuse_stemdw=False).nodes()]
    assert "conv_stem" in kinds_plain and "dw_conv" in kinds_plain, kinds_plain
    for nm, o in zip(names, outs):
        assert np.array_equal(o, plain[0]), nm
    ref = oracle.run_graph(desc, keep=[y])[y]
    ok, msg = check_layer("fused output", outs[0], ref.reshape(outs[0].shape))
    assert ok, msg


def test_fused_stem_pair_bf16():
    from paper_1907_01989_amd import engine, _binding as B
    desc, y = pair_graph(2, 224, 224, 32, None, None, ACT_RELU6, DTYPE_FP16)
    bdesc = workloads.as_bf16_graph(desc)
    plan = engine.Plan(bdesc, bind=False, fuse_stemdw=2, dtype=B.DTYPE_BF16)
    idx = [i for i, k in enumerate(plan.nodes()) if k["kind"] == "stem_dw"]
    assert len(idx) == 1
    ncfg = plan.node_configs()[idx[0]][1]
    log(f"[case] {desc['name']} bf16 ({ncfg} configurations)")
    _, plain, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_stemdw=False)
    for c in range(ncfg):
        _, fused, _ = run_gpu(bdesc, materialize_all=False, dtype=B.DTYPE_BF16, fuse_stemdw=2, configs={idx[0]: c})
        np.testing.assert_array_equal(fused[0], plain[0], err_msg=f"configuration {c}")
    ref = oracle.run_graph(bdesc, keep=[y], store_bf16=True)[y]
    ok, msg = check_layer("fused bf16 output", plain[0], ref.reshape(plain[0].shape))
    assert ok, msg


@pytest.mark.parametrize("net", ["mobilenet_v1", "mobilenet_v2"])
def test_fused_stem_network(net):
    from paper_1907_01989_amd import engine
    desc = workloads.WORKLOADS[net](64)
    kinds = [k["kind"] for k in engine.Plan(desc, bind=False).nodes()]
    assert kinds[0] == "stem_dw", kinds[:3]
    log(f"[case] {net} b64 stem->depthwise fused vs unfused")
    _, fused, _ = run_gpu(desc, materialize_all=False)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_stemdw=False)
    for a, b in zip(fused, plain):
        np.testing.assert_array_equal(a, b)

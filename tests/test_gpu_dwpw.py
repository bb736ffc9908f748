"""Depthwise 3x3 fused into the consuming pointwise convolution.

The fused kernel computes each depthwise output with the standalone kernel's
tap order, fp32 accumulation, activation and fp16 rounding, and runs the
pointwise GEMM with K in the same order, so fused and unfused plans must
agree bit for bit; the unfused operators are held to the oracle by the
operator tests, and the fused output is also checked against the oracle at
the chained-layer bound.  Shapes cover ragged pixel tails, K not a multiple
of 32, channel counts that are not multiples of 16, both strides, both tile
heights (64 and 128 pixels) and a residual epilogue.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads import ACT_NONE, ACT_RELU6, NetBuilder

from gpu_util import check_layer, log, run_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # n, h, w, c (depthwise channels = K), stride, N (pointwise outputs), residual
    (64, 28, 28, 72, 1, 40, False),      # 64-pixel tiles, K tail
    (48, 56, 56, 32, 2, 24, True),       # stride 2, residual
    (128, 14, 14, 96, 1, 160, False),    # 12 blocks for 10
    (17, 57, 55, 20, 1, 320, True),      # odd sizes, 20 blocks, ragged everything
    (64, 112, 112, 32, 1, 64, False),    # 128-pixel tiles (v1 layer 1 shape)
    (8, 113, 111, 8, 2, 16, False),      # one slice, stride 2 on odd sizes
]


def pair_graph(n, h, w, c, s, N, res):
    g = NetBuilder(seed=c + N + s)
    x = g.activation(g.input(n, h, w, c, -1, 1), ACT_NONE)
    d = g.dw(x, 3, s=s, act=ACT_RELU6)
    y = g.conv(d, N, 1, act=ACT_NONE if res else ACT_RELU6)
    if res:
        oh, ow, _ = g.hwc(y)
        r = g.activation(g.input(n, oh, ow, N, -1, 1, name="skip"), ACT_NONE)
        y = g.add(y, r, act=ACT_NONE)
    g.mark_output(y)
    return g.graph(f"dwpw_{n}x{h}x{w}x{c}_s{s}_to{N}_r{int(res)}"), y


@pytest.mark.parametrize("n,h,w,c,s,N,res", CASES)
def test_fused_pair_matches_unfused(n, h, w, c, s, N, res):
    from paper_1907_01989_amd import engine
    desc, y = pair_graph(n, h, w, c, s, N, res)
    kinds = [k["kind"] for k in engine.Plan(desc, bind=False, fuse_dwpw=True).nodes()]
    assert "dw_pw" in kinds and "dw_conv" not in kinds, kinds
    log(f"[case] {desc['name']}")
    _, fused, _ = run_gpu(desc, materialize_all=False, fuse_dwpw=True)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_dwpw=False)
    np.testing.assert_array_equal(fused[0], plain[0])
    ref = oracle.run_graph(desc, keep=[y])[y]
    ok, msg = check_layer("fused output", fused[0], ref.reshape(fused[0].shape))
    assert ok, msg


@pytest.mark.parametrize("net", ["mobilenet_v1", "mobilenet_v2"])
def test_fused_network_matches_unfused(net):
    from paper_1907_01989_amd import engine
    # (with the pointwise -> depthwise and stem -> depthwise fusions off, which
    # would take the depthwise layers first)
    desc = workloads.WORKLOADS[net](64)
    off = {"fuse_pwdw": False, "fuse_stemdw": False}
    kinds = [k["kind"] for k in engine.Plan(desc, bind=False, fuse_dwpw=True, **off).nodes()]
    assert kinds.count("dw_pw") >= 5
    log(f"[case] {net} b64 fused vs unfused")
    _, fused, _ = run_gpu(desc, materialize_all=False, fuse_dwpw=True, **off)
    _, plain, _ = run_gpu(desc, materialize_all=False, fuse_dwpw=False, **off)
    for a, b in zip(fused, plain):
        np.testing.assert_array_equal(a, b)

"""Padding lanes of the channel-sliced layout stay zero.

Tensors are stored in slices of 8 channels; a tensor whose channel count is
not a multiple of 8 has padding lanes in its last slice, which every kernel
must leave at zero (the paper pads its 4-channel slices with zeros, Sec. 4):
consumers such as a concatenation, an argmax or a channel-summing kernel
would otherwise read them.  Every node output of a network whose channel
counts are all odd -- stem, fused stem + depthwise, pointwise, fused
pointwise + depthwise, residual add, dilated depthwise, projection, global
pool, concatenation, resize -- is read back raw (mgi_plan_read_node_raw, with
every node materialised) and its padding lanes checked, for fp16 and bf16
storage and for every kernel configuration of every node.
"""
import numpy as np
import pytest

from workloads import ACT_NONE, ACT_RELU6, NetBuilder

from gpu_util import log

pytestmark = pytest.mark.gpu


def odd_net():
    g = NetBuilder(seed=7)
    x = g.input(2, 30, 30, 3, 0.0, 1.0)
    t1 = g.conv(x, 13, 3, s=2, name="stem")                 # 15x15x13
    t2 = g.dw(t1, 3, 1, name="dw1")                         # fused with the stem
    t3 = g.conv(t2, 21, 1, name="pw1")
    t4 = g.dw(t3, 3, 2, name="dw2")                         # fused with pw1, 8x8x21
    t5 = g.conv(t4, 21, 1, act=ACT_NONE, name="proj")
    t6 = g.add(t5, t4, name="res")                          # residual epilogue of proj
    t7 = g.conv(t6, 45, 1, name="expand")
    t8 = g.dw(t7, 3, 1, d=2, name="dw_dil")                 # dilated: its own kernel
    t9 = g.conv(t8, 11, 1, act=ACT_NONE, name="proj2")
    p = g.gap(t9, name="pool")
    z = g.fc(p, 10, name="fc")
    s = g.softmax(z, name="softmax")
    c = g.concat([t9, t9], name="cat")                      # 22 channels
    r = g.resize(c, 15, 15, True, name="up")
    a = g.argmax(r, name="labels")
    g.mark_output(z)
    g.mark_output(s)
    g.mark_output(a)
    return g.graph("odd_channels")


@pytest.mark.parametrize("dtype", [0, 1])
def test_padding_lanes_stay_zero(dtype):
    import torch
    from paper_1907_01989_amd import _binding as B, engine
    desc = odd_net()
    plan = engine.Plan(desc, materialize_all=True, dtype=dtype)
    nodes = plan.nodes()
    cfg_runs = [{}] + [{i: c} for i in range(len(nodes)) for c in range(1, plan.node_configs()[i][1])]
    xs = plan.input_tensors()
    checked = set()
    for cfgs in cfg_runs:
        for i in range(len(nodes)):
            B.mgi_plan_set_node_config(plan.handle, i, cfgs.get(i, 0))
        plan.run(xs)
        torch.cuda.synchronize()
        for i, n in enumerate(nodes):
            try:
                nbytes = B.mgi_plan_read_node_raw(plan.handle, i)
            except B.MgiError as e:
                assert e.status == 3      # fp32 / int32 outputs are not sliced
                continue
            nb_, h, w, c = n["shape"]
            S = (c + 7) // 8
            assert nbytes == S * nb_ * h * w * 16, (n, nbytes)
            raw = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda:0")
            B.mgi_plan_read_node_raw(plan.handle, i, raw.data_ptr())
            torch.cuda.synchronize()
            v = raw.cpu().numpy().view(np.uint16).reshape(S, nb_ * h * w, 8)
            pad = v[S - 1, :, c - 8 * (S - 1):]
            # +0 or -0 only (the sign bit may be set; nothing else)
            bad = (pad & 0x7FFF) != 0
            assert not bad.any(), (f"{n['kind']} {desc['ops'][n['tensor']]['name']} config {cfgs}: "
                                   f"{int(bad.sum())} nonzero padding values")
            checked.add(n["kind"])
        log(f"[case] padding lanes dtype {dtype} configs {cfgs}: {sorted(checked)}")
    assert {"stem_dw", "pw_dw", "pw_gemm", "dw_conv", "global_avgpool", "concat"} <= checked, checked

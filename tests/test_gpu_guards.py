"""Guard regions around every device buffer the engine writes.

The workspace (planned arena plus state region) and every graph output are
allocated with a guard region behind them, filled with a byte pattern; after
runs of every network (and of every kernel configuration of each node on a
small odd-channel network) the guards must be unchanged: no kernel writes
past the buffers the plan gives it.
"""
import numpy as np
import pytest

import workloads

from gpu_util import log
from test_gpu_padlanes import odd_net

pytestmark = pytest.mark.gpu

GUARD = 1 << 16
PATTERN = 0xA5


def guarded_plan(desc, **kw):
    import torch
    from paper_1907_01989_amd import _binding as B, engine
    plan = engine.Plan(desc, bind=False, **kw)
    ws = torch.full((plan.workspace_bytes + 256 + GUARD,), PATTERN, dtype=torch.uint8, device="cuda:0")
    wts = torch.empty(plan.weight_bytes + 256, dtype=torch.uint8, device="cuda:0")
    ws_ptr = (ws.data_ptr() + 255) & ~255
    B.mgi_plan_bind(plan.handle, ws_ptr, (wts.data_ptr() + 255) & ~255, 0)
    plan.bound = True
    plan.ws, plan.wts = ws, wts
    lead = ws_ptr - ws.data_ptr()
    outs, raw = [], []
    for o in plan.alloc_outputs():
        nbytes = o.numel() * o.element_size()
        buf = torch.full((nbytes + GUARD,), PATTERN, dtype=torch.uint8, device="cuda:0")
        raw.append((buf, nbytes))
        outs.append(buf[:nbytes].view(o.dtype).view(o.shape))
    return plan, outs, raw, ws, lead


def check_guards(plan, raw, ws, lead, what):
    import torch
    torch.cuda.synchronize()
    tail = ws[lead + plan.workspace_bytes:].cpu().numpy()
    assert (tail == PATTERN).all(), f"{what}: workspace guard written ({int((tail != PATTERN).sum())} bytes)"
    for k, (buf, nbytes) in enumerate(raw):
        g = buf[nbytes:].cpu().numpy()
        assert (g == PATTERN).all(), f"{what}: guard of output {k} written ({int((g != PATTERN).sum())} bytes)"


@pytest.mark.parametrize("net,batch", [("mobilenet_v1", 1), ("mobilenet_v2", 2), ("deeplab", 1),
                                       ("mobilenet_v1", 64)])
def test_networks_write_inside_their_buffers(net, batch):
    desc = workloads.WORKLOADS[net](batch)
    log(f"[case] guards {net} b{batch}")
    plan, outs, raw, ws, lead = guarded_plan(desc)
    xs = plan.input_tensors()
    for _ in range(2):
        plan.run(xs, outs)
    check_guards(plan, raw, ws, lead, f"{net} b{batch}")


def test_every_configuration_writes_inside_its_buffers():
    from paper_1907_01989_amd import _binding as B
    desc = odd_net()
    plan, outs, raw, ws, lead = guarded_plan(desc, materialize_all=True)
    xs = plan.input_tensors()
    n = len(plan.nodes())
    runs = 0
    for i in range(n):
        c0, k, _ = plan.node_configs()[i]
        for c in range(k):
            B.mgi_plan_set_node_config(plan.handle, i, c)
            plan.run(xs, outs)
            runs += 1
        B.mgi_plan_set_node_config(plan.handle, i, c0)
    log(f"[case] guards odd-channel net: {runs} runs")
    check_guards(plan, raw, ws, lead, "odd-channel net, every configuration")
    assert np.isfinite(outs[0].cpu().numpy()).all()

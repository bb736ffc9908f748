"""Captured launch list (mgi_plan_capture / mgi_plan_replay) against eager runs.

The graph replays the same kernels on the same buffers as mgi_plan_run, so
every replay must reproduce the eager outputs bit for bit.  Replays are
interleaved with eager runs and synchronisations, repeated several times, and
rerun after the input buffer's contents change (the pointers are baked into
the graph, the data is not).
"""
import numpy as np
import pytest

import workloads

from gpu_util import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("net,batch", [("mobilenet_v1", 1), ("mobilenet_v2", 2), ("deeplab", 1)])
def test_graph_replay_matches_eager(net, batch):
    import torch
    from paper_1907_01989_amd import engine

    desc = workloads.WORKLOADS[net](batch)
    log(f"[case] graph replay {net} b{batch}")
    plan = engine.Plan(desc)
    xs = plan.input_tensors()
    ref = [o.cpu().numpy() for o in plan.run(xs)]
    torch.cuda.synchronize()
    gouts = plan.capture(xs)
    for rep in range(4):
        for o in gouts:
            o.fill_(-7)
        plan.replay()
        torch.cuda.synchronize()
        for g, r in zip(gouts, ref):
            np.testing.assert_array_equal(g.cpu().numpy(), r, err_msg=f"replay {rep}")
        eager = plan.run(xs)
        torch.cuda.synchronize()
        for e, r in zip(eager, ref):
            np.testing.assert_array_equal(e.cpu().numpy(), r)
    # new contents in the captured input buffer: replay follows them
    g = torch.Generator().manual_seed(5)
    new = torch.rand(xs[0].shape, generator=g).to(xs[0].device, xs[0].dtype)
    xs[0].copy_(new)
    ref2 = [o.cpu().numpy() for o in plan.run([new])]
    plan.replay()
    torch.cuda.synchronize()
    for g_, r in zip(gouts, ref2):
        np.testing.assert_array_equal(g_.cpu().numpy(), r)
    assert any(not np.array_equal(a, b) for a, b in zip(ref, ref2))
    plan.close()


def test_run_rejects_mismatched_device_tensors():
    """Wrong element type, byte size or layout of a device tensor is refused
    on the host, before any kernel is launched."""
    import torch
    from paper_1907_01989_amd import engine

    g = workloads.NetBuilder(seed=0)
    x = g.input(1, 16, 16, 3, 0.0, 1.0)
    t = g.conv(x, 16, 3, 2, name="stem")
    p = g.gap(t, name="pool")
    z = g.fc(p, 10, name="fc")
    g.mark_output(z)
    plan = engine.Plan(g.graph("io_checks_gpu"))
    log("[case] run argument checks")
    xs = plan.input_tensors()
    good = plan.alloc_outputs()
    with pytest.raises(ValueError, match="dtype"):
        plan.run([xs[0].float()], good)
    with pytest.raises(ValueError, match="bytes"):
        plan.run(xs, [torch.empty((1, 9), dtype=torch.float32, device="cuda:0")])
    with pytest.raises(ValueError, match="contiguous"):
        plan.run([xs[0].transpose(1, 2)], good)
    with pytest.raises(ValueError, match="dtype"):
        plan.run(xs, [torch.empty((1, 10), dtype=torch.int32, device="cuda:0")])
    out = plan.run(xs, good)[0]
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()

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

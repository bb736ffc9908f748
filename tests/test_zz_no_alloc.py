"""mgi_plan_run_noalloc: the run whose workspace is the library's static
device array, against mgi_plan_run on the same plan and buffers.

Calls come in a row on one device with shrinking inputs (a 513x513 DeepLab-
style network, MobileNet-v2 at 224, MobileNet-v1 at 128), so each call finds
the previous call's data in the shared array, including where its own state
region (the FC -> softmax arrival counters) lies.  Both entry points run the
same kernels, so outputs must be bit-identical.  A plan whose workspace is
larger than the array is refused before anything is enqueued.
"""
import numpy as np
import pytest

import workloads

from gpu_util import log

pytestmark = pytest.mark.gpu


def _plan_and_reference(desc):
    import torch
    from paper_1907_01989_amd import engine
    plan = engine.Plan(desc)
    xs = plan.input_tensors()
    ref = [o.cpu().numpy() for o in plan.run(xs)]
    torch.cuda.synchronize()
    return plan, xs, ref


def _run_noalloc(plan, xs):
    import torch
    from paper_1907_01989_amd import _binding as B
    outs = plan.alloc_outputs()
    for o in outs:
        o.fill_(-7)                      # nothing stale can pass for a result
    plan.check_io(xs, outs)
    B.mgi_plan_run_noalloc(plan.handle, [x.data_ptr() for x in xs], [o.data_ptr() for o in outs],
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs]


def test_noalloc_matches_run_on_calls_in_a_row():
    from paper_1907_01989_amd import _binding as B
    cases = [("deeplab_513", workloads.deeplab_v2_os16(1)),
             ("mobilenet_v2_224", workloads.mobilenet_v2(1)),
             ("mobilenet_v1_128", workloads.mobilenet_v1(1, res=128))]
    plans = []
    for name, desc in cases:
        plan, xs, ref = _plan_and_reference(desc)
        assert plan.workspace_bytes <= B.NOALLOC_WORKSPACE_BYTES
        plans.append((name, plan, xs, ref))
    sizes = [p.workspace_bytes for _, p, _, _ in plans]
    assert sizes == sorted(sizes, reverse=True)
    for rnd in range(2):
        for name, plan, xs, ref in plans:
            log(f"[case] noalloc {name} call {rnd} (workspace {plan.workspace_bytes} bytes)")
            got = _run_noalloc(plan, xs)
            for a, b in zip(got, ref):
                np.testing.assert_array_equal(a, b)


def test_noalloc_refuses_a_plan_larger_than_its_workspace():
    import torch
    from paper_1907_01989_amd import _binding as B, engine
    plan = engine.Plan(workloads.mobilenet_v1(64))
    log(f"[case] noalloc refusal (workspace {plan.workspace_bytes} bytes)")
    assert plan.workspace_bytes > B.NOALLOC_WORKSPACE_BYTES
    xs = plan.input_tensors()
    outs = plan.alloc_outputs()
    with pytest.raises(B.MgiError) as e:
        B.mgi_plan_run_noalloc(plan.handle, [x.data_ptr() for x in xs], [o.data_ptr() for o in outs],
                               torch.cuda.current_stream().cuda_stream)
    assert e.value.status == 5 and "no-allocation workspace" in str(e.value)

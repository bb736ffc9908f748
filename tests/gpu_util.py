"""Helpers shared by the GPU parity tests: run a network description on the
GPU through the C ABI and on the oracle, and compare."""
from __future__ import annotations

import sys

import numpy as np

import oracle

# Per-layer bound for chained network checks: max |gpu - ref| <= LAYER_TOL * max |ref|
# (fp16 storage of every layer output, fp32 accumulation).
LAYER_TOL = 2e-2
# Logits: relative L2 per image.
LOGITS_RELL2 = 1e-2
# Isolated single operators on exact fp16 inputs: the only rounding is the fp16
# store of the result (half an ulp, 2^-11 relative) and fp32 accumulation;
# the bound leaves a factor of two on the relative part.
ISO_RTOL = 2.0 ** -10
ISO_ATOL_FRAC = 1e-3


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_numpy(t):
    return t.detach().cpu().numpy()


def run_gpu(desc, materialize_all=True, fuse=True, planner=None, fuse_dwpw=False, dtype=0,
            fuse_pwdw=True, configs=None, fuse_stemdw=True, fuse_pool=True, fuse_softmax=True, fuse_irb=False):
    """Run ``desc`` once; returns (plan, outputs as numpy, {tensor id: node output}).
    ``configs``: {node index: kernel configuration} set before the run."""
    import torch
    from paper_1907_01989_amd import engine, _binding as B
    kw = {"fuse_dwpw": fuse_dwpw, "dtype": dtype, "fuse_pwdw": fuse_pwdw, "fuse_stemdw": fuse_stemdw,
          "fuse_pool": fuse_pool, "fuse_softmax": fuse_softmax, "fuse_irb": fuse_irb}
    if planner is not None:
        kw["planner"] = planner
    plan = engine.Plan(desc, fuse=fuse, materialize_all=materialize_all, **kw)
    for i, c in (configs or {}).items():
        B.mgi_plan_set_node_config(plan.handle, i, c)
    xs = plan.input_tensors()
    outs = plan.run(xs)
    nodes = {}
    if materialize_all:
        for i, info in enumerate(plan.nodes()):
            if info["tensor"] < 0:
                continue
            _, t = plan.read_node(i)
            nodes[info["tensor"]] = t
    torch.cuda.synchronize()
    outs_np = [to_numpy(o) for o in outs]
    nodes_np = {k: to_numpy(v) for k, v in nodes.items()}
    return plan, outs_np, nodes_np


def layer_error(g, r):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    denom = float(np.abs(r).max())
    err = float(np.abs(g - r).max())
    return err, denom


def check_layer(name, g, r, tol=LAYER_TOL):
    err, denom = layer_error(g, r)
    ok = err <= tol * max(denom, 1e-30)
    return ok, f"{name}: max|diff|={err:.3e} max|ref|={denom:.3e} ratio={err / max(denom, 1e-30):.3e}"


# bf16 storage: 8 significand bits, half an ulp is 2^-9 relative
ISO_RTOL_BF16 = 2.0 ** -8


def check_isolated(name, g, r, rtol=ISO_RTOL):
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    bound = rtol * np.abs(r) + ISO_ATOL_FRAC * max(float(np.abs(r).max()), 1e-30)
    bad = np.abs(g - r) > bound
    assert not bad.any(), (f"{name}: {int(bad.sum())} of {bad.size} elements out of bound; "
                           f"worst |diff|={float(np.abs(g - r).max()):.3e}")


def logits_check(gl, rl):
    """Per-image relative L2 of the logits and top-1 agreement."""
    gl = np.asarray(gl, np.float64).reshape(gl.shape[0], -1)
    rl = np.asarray(rl, np.float64).reshape(rl.shape[0], -1)
    rel = np.linalg.norm(gl - rl, axis=1) / np.linalg.norm(rl, axis=1)
    top_g = gl.argmax(1)
    top_r = rl.argmax(1)
    srt = np.sort(rl, axis=1)
    gap = srt[:, -1] - srt[:, -2]
    return rel, top_g, top_r, gap


def labels_check(g_labels, r_up, margin=1e-2):
    """Compare argmax labels where the reference's top-2 margin exceeds ``margin``."""
    srt = np.sort(r_up, axis=-1)
    ref = r_up.argmax(-1)
    g = g_labels.reshape(ref.shape)
    mask = (srt[..., -1] - srt[..., -2]) > margin
    mismatches = int(((g != ref) & mask).sum())
    return mismatches, float(mask.mean()), int((g != ref).sum())


def isolated_reference(desc, t, gpu_vals, cache=None):
    """Oracle value of tensor ``t`` computed from the GPU's own materialised
    operands: fused-away producers are recomputed by the oracle from their
    GPU operands, so the result isolates the error of one fused node."""
    cache = {} if cache is None else cache
    if t in cache:
        return cache[t]
    op = desc["ops"][t]
    operands = []
    for u in oracle.op_inputs(op):
        if desc["ops"][u]["op"] == "input":
            operands.append(np.asarray(desc["ops"][u]["data"], np.float64))
        elif u in gpu_vals:
            operands.append(np.asarray(gpu_vals[u], np.float64))
        else:
            operands.append(isolated_reference(desc, u, gpu_vals, cache))
    v = oracle.eval_op(op, operands)
    cache[t] = v
    return v

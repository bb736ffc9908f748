"""Throughput benchmark of the mgi engine on one MI355X.

A step is one forward pass of the whole network over one batch of synthetic,
device-resident input (launch sequence of every fused node on one stream).
Protocol after Sec. 6 of the paper: warm-up runs are skipped, then the mean
over the timed runs is reported.  Prints ONE JSON line on stdout.

  python bench.py [--gpus 1] [--steps 100] [--warmup 10] [--workload v1_b64]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12            # bytes/s, MI355X HBM3E
MFMA_F16_PEAK = 2516.6e12    # flop/s, dense fp16 MFMA
RIDGE = MFMA_F16_PEAK / HBM_PEAK

WORKLOADS = {
    "dw_block": ("dw_block", 1),
    "v1_b1": ("mobilenet_v1", 1),
    "v2_b1": ("mobilenet_v2", 1),
    "v1_b64": ("mobilenet_v1", 64),
    "v2_b64": ("mobilenet_v2", 64),
    "deeplab": ("deeplab", 1),
}


def eprint(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# HIP events through the runtime's C API
# ---------------------------------------------------------------------------
class Hip:
    def __init__(self):
        self.L = ctypes.CDLL("libamdhip64.so")
        self.L.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                               ctypes.c_void_p]
        self.L.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.L.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.L.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        assert self.L.hipEventCreate(ctypes.byref(e)) == 0
        return e.value

    def elapsed_ms(self, a, b):
        f = ctypes.c_float()
        assert self.L.hipEventSynchronize(ctypes.c_void_p(b)) == 0
        assert self.L.hipEventElapsedTime(ctypes.byref(f), ctypes.c_void_p(a), ctypes.c_void_p(b)) == 0
        return f.value

    def destroy(self, e):
        self.L.hipEventDestroy(ctypes.c_void_p(e))

    def record(self, e, stream):
        assert self.L.hipEventRecord(ctypes.c_void_p(e), ctypes.c_void_p(stream)) == 0


def percentiles(xs):
    ys = sorted(xs)
    pick = lambda q: ys[min(len(ys) - 1, int(q * len(ys)))]   # noqa: E731
    return {"mean": sum(ys) / len(ys), "p50": pick(0.5), "p90": pick(0.9)}


# ---------------------------------------------------------------------------
# algorithmic work of each fused node
# ---------------------------------------------------------------------------
def tensor_shapes(desc, nodes):
    """Shape of every graph input and every tensor a node materialises, as
    reported by the engine."""
    shapes = {}
    for t, op in enumerate(desc["ops"]):
        if op["op"] == "input":
            shapes[t] = tuple(op["shape"])
    for n in nodes:
        if n["tensor"] >= 0:
            shapes[n["tensor"]] = tuple(n["shape"])
    return shapes


def op_inputs(op):
    if op["op"] == "input":
        return []
    if op["op"] == "add":
        return [op["a"], op["b"]]
    if op["op"] == "concat":
        return list(op["ins"])
    return [op["in"]]


def node_work(desc, nodes, shapes, i):
    """(flops, bytes, bound) that the method itself must do for node i:
    activations read once and written once in fp16, weights read once."""
    info = nodes[i]
    kind = info["kind"]
    t = info["tensor"]
    materialized = {n["tensor"] for n in nodes if n["tensor"] >= 0}
    ops = desc["ops"]

    def head_of(u):
        op = ops[u]
        if op["op"] == "activation" and op["in"] not in materialized and ops[op["in"]]["op"] != "input":
            return head_of(op["in"])
        if op["op"] == "add":
            for side in ("a", "b"):
                v = op[side]
                if v not in materialized and ops[v]["op"] != "input":
                    return head_of(v)
        return u

    def elems(u):
        n, h, w, c = shapes[u]
        return n * h * w * c

    if t < 0:
        return 0.0, 0.0, "hbm"
    h = head_of(t)
    op = ops[h]
    out_b = elems(t) * 2
    if kind in ("conv_stem", "pw_gemm", "conv_igemm"):
        x = op["in"]
        cin = shapes[x][3]
        n, oh, ow, cout = shapes[t]
        m = n * oh * ow
        flops = 2.0 * m * op["kh"] * op["kw"] * cin * cout
        in_bytes = elems(x) * (4 if (kind == "conv_stem" and ops[x].get("dtype", 2) == 2) else 2)
        byts = in_bytes + out_b + op["w"].size * 2 + op["b"].size * 4
        if h != t:
            byts += out_b          # fused residual operand
    elif kind == "dw_pw":
        # depthwise input in, pointwise output out; the intermediate tensor
        # never reaches memory
        d = head_of(op["in"])
        dop = ops[d]
        n, oh, ow, cout = shapes[t]
        m = n * oh * ow
        cin = op["w"].shape[-1]
        flops = 2.0 * m * cin * cout + 2.0 * m * cin * dop["kh"] * dop["kw"]
        byts = (elems(dop["in"]) * 2 + out_b + op["w"].size * 2 + op["b"].size * 4 +
                dop["w"].size * 2 + dop["b"].size * 4)
        if h != t:
            byts += out_b          # fused residual operand
    elif kind == "pw_dw":
        # pointwise input in, depthwise output out; the pointwise output
        # never reaches memory
        p = head_of(op["in"])
        pop = ops[p]
        n, h_, w_, cin = shapes[pop["in"]]        # 1x1 stride 1: same plane
        cmid = pop["cout"]
        flops = 2.0 * n * h_ * w_ * cin * cmid + 2.0 * elems(t) * op["kh"] * op["kw"]
        byts = (elems(pop["in"]) * 2 + out_b + pop["w"].size * 2 + pop["b"].size * 4 +
                op["w"].size * 2 + op["b"].size * 4)
    elif kind == "irb":
        # inverted residual block: block input in (and the residual), block
        # output out; the expanded and depthwise tensors never reach memory
        dop = ops[head_of(op["in"])]
        pop = ops[head_of(dop["in"])]
        n, h_, w_, cin = shapes[pop["in"]]        # 1x1 stride 1: same plane
        cmid = pop["cout"]
        no, oh, ow, cout = shapes[t]                # 1x1 stride-1 projection: the depthwise plane
        flops = (2.0 * n * h_ * w_ * cin * cmid + 2.0 * no * oh * ow * cmid * dop["kh"] * dop["kw"] +
                 2.0 * no * oh * ow * cmid * cout)
        byts = (elems(pop["in"]) * 2 + out_b + pop["w"].size * 2 + pop["b"].size * 4 +
                dop["w"].size * 2 + dop["b"].size * 4 + op["w"].size * 2 + op["b"].size * 4)
        if h != t:
            byts += out_b          # fused residual operand
    elif kind == "pw_pool":
        # pointwise input in, pooled means out; the pointwise output never
        # reaches memory
        cop = ops[head_of(op["in"])]
        n, h_, w_, cin = shapes[cop["in"]]
        cmid = cop["cout"]
        flops = 2.0 * n * h_ * w_ * cin * cmid + float(n * h_ * w_ * cmid)
        byts = elems(cop["in"]) * 2 + out_b + cop["w"].size * 2 + cop["b"].size * 4
    elif kind == "stem_dw":
        # graph input in, depthwise output out; the stem output never
        # reaches memory
        sop = ops[head_of(op["in"])]
        x = sop["in"]
        cin = shapes[x][3]
        sn, sh_, sw_ = shapes[x][0], (shapes[t][1]), (shapes[t][2])   # stride-1 depthwise: same plane
        cmid = sop["cout"]
        flops = (2.0 * sn * sh_ * sw_ * sop["kh"] * sop["kw"] * cin * cmid +
                 2.0 * elems(t) * op["kh"] * op["kw"])
        in_bytes = elems(x) * (4 if ops[x].get("dtype", 2) == 2 else 2)
        byts = (in_bytes + out_b + sop["w"].size * 2 + sop["b"].size * 4 +
                op["w"].size * 2 + op["b"].size * 4)
    elif kind == "dw_conv":
        flops = 2.0 * elems(t) * op["kh"] * op["kw"]
        byts = elems(op["in"]) * 2 + out_b + op["w"].size * 4 + op["b"].size * 4
    elif kind == "fc_gemm":
        n = shapes[t][0]
        flops = 2.0 * op["w"].size * n
        byts = elems(op["in"]) * 2 + op["w"].size * 2 + op["b"].size * 4 + elems(t) * 4
    elif kind == "global_avgpool":
        flops = float(elems(op["in"]))
        byts = elems(op["in"]) * 2 + out_b
    elif kind == "softmax":
        flops = 3.0 * elems(t)
        byts = elems(t) * 8
    elif kind == "fc_softmax":
        # FC input and weights in, probabilities out (the logits pass between
        # the FC and the softmax inside one launch)
        fop = ops[head_of(op["in"])]
        n = shapes[t][0]
        flops = 2.0 * fop["w"].size * n + 3.0 * elems(t)
        byts = elems(fop["in"]) * 2 + fop["w"].size * 2 + fop["b"].size * 4 + elems(t) * 4
    elif kind == "resize_argmax":
        # the logits in (fp16), int32 labels out; the upsampled logits never
        # reach memory
        src = ops[op["in"]]["in"]
        n, h_, w_, _ = shapes[t]
        c = shapes[src][3]
        flops = float(n * h_ * w_) * c * 8.0
        byts = elems(src) * 2 + n * h_ * w_ * 4
    else:
        ins = op_inputs(op)
        flops = float(elems(t))
        byts = sum(elems(u) * 2 for u in ins) + out_b
    bound = "mfma" if (flops / max(byts, 1.0)) >= RIDGE else "hbm"
    return flops, float(byts), bound


def kernel_sources_hash():
    """Hash of the kernel sources; a counter-based traffic figure is used only
    while the kernels it was measured on are unchanged."""
    import hashlib
    h = hashlib.sha1()
    for f in ("gemm.hip", "ops.hip", "dwpw.hip", "pwdw.hip", "stemdw.hip", "irb.hip", "device.h", "kernels.h"):
        with open(os.path.join(ROOT, "paper_1907_01989_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, layer, config):
    """HBM bytes per launch of (node kind, layer, configuration) from the
    committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary, scaled by the copy
    calibration there; None when absent, measured on other kernel sources or
    on another configuration of the layer."""
    path = os.path.join(ROOT, "profiles", "mobilenet_v1_224_b64_traffic.md")
    if not os.path.exists(path):
        return None
    cur = kernel_sources_hash()
    with open(path) as f:
        for line in f:
            if line.startswith("traffic_bytes_per_launch:"):
                f = line.split()
                if len(f) == 7 and f[1:4] == [kernel, layer, config] and f[6] == cur:
                    return int(f[4])
    return None


# the dominant kernel is timestamped in every DOM_EVERY-th step of the timed region
DOM_EVERY = 5


def roofline_entry(flops, byts, bound, seconds):
    if bound == "mfma":
        ach = flops / seconds / 1e12
        return {"bound": "mfma", "achieved": round(ach, 3), "peak": MFMA_F16_PEAK / 1e12,
                "unit": "TFLOP/s", "frac": round(ach * 1e12 / MFMA_F16_PEAK, 4)}
    ach = byts / seconds / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": round(ach * 1e9 / HBM_PEAK, 4)}


# ---------------------------------------------------------------------------
def run_workload(key, steps, warmup, hip, profile_steps=20, detail=True, tune=True, fuse_dwpw=False,
                 fuse_pwdw=True, fuse_stemdw=True):
    import torch
    import workloads
    from paper_1907_01989_amd import _binding as B
    from paper_1907_01989_amd import engine

    net, batch = WORKLOADS[key]
    desc = workloads.WORKLOADS[net](batch)
    plan = engine.Plan(desc, fuse_dwpw=fuse_dwpw, fuse_pwdw=fuse_pwdw, fuse_stemdw=fuse_stemdw)
    xs = plan.input_tensors()
    outs = plan.alloc_outputs()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    ins = [x.data_ptr() for x in xs]
    ops_ptrs = [o.data_ptr() for o in outs]
    nodes = plan.nodes()
    nn = len(nodes)
    if tune:
        # plan-time tuning of kernel configurations (mgi_plan_autotune), as an
        # application would do once after loading the model
        plan.autotune(xs, outs, reps=10, stream=sh)
    configs = [name for _, _, name in plan.node_configs()]
    for _ in range(warmup):
        B.mgi_plan_run(plan.handle, ins, ops_ptrs, sh)
    torch.cuda.synchronize()

    # per-layer pass (outside the timed region): every node's kernel
    # timestamped at its start and end on the device
    per_node = [0.0] * nn
    if detail:
        evs = [([hip.event() for _ in range(nn)], [hip.event() for _ in range(nn)])
               for _ in range(profile_steps)]
        for k in range(profile_steps):
            B.mgi_plan_run_timed(plan.handle, ins, ops_ptrs, evs[k][0], evs[k][1], sh)
        torch.cuda.synchronize()
        for k in range(profile_steps):
            for i in range(nn):
                per_node[i] += hip.elapsed_ms(evs[k][0][i], evs[k][1][i]) / profile_steps
        for a, b in evs:
            for e in a + b:
                hip.destroy(e)
    dom = max(range(nn), key=lambda i: per_node[i])

    # device time per step, from events between steps of an untimed pass
    marks = [hip.event() for _ in range(21)]
    for k in range(20):
        hip.record(marks[k], sh)
        B.mgi_plan_run(plan.handle, ins, ops_ptrs, sh)
    hip.record(marks[20], sh)
    torch.cuda.synchronize()
    step_ms = percentiles([hip.elapsed_ms(marks[k], marks[k + 1]) for k in range(20)])
    for e in marks:
        hip.destroy(e)

    # timed region: K steps; the dominant node's kernel is timestamped at its
    # start and end in every DOM_EVERY-th step (a timestamped launch costs a
    # few microseconds of its own, so sampling keeps that out of most steps)
    sampled = list(range(0, steps, DOM_EVERY))
    dev = {k: (hip.event(), hip.event()) for k in sampled}
    arrays = {}
    for k, (a, b) in dev.items():
        e0, e1 = [None] * nn, [None] * nn
        e0[dom], e1[dom] = a, b
        arrays[k] = (e0, e1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        if k in arrays:
            B.mgi_plan_run_timed(plan.handle, ins, ops_ptrs, arrays[k][0], arrays[k][1], sh)
        else:
            B.mgi_plan_run(plan.handle, ins, ops_ptrs, sh)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    dom_ms = sum(hip.elapsed_ms(a, b) for a, b in dev.values()) / len(dev)
    for a, b in dev.values():
        hip.destroy(a)
        hip.destroy(b)

    shapes = tensor_shapes(desc, nodes)
    layers = []
    for i, info in enumerate(nodes):
        fl, by, bound = node_work(desc, nodes, shapes, i)
        name = desc["ops"][info["tensor"]]["name"] if info["tensor"] >= 0 else info["kind"]
        entry = {"node": i, "name": name, "kind": info["kind"], "config": configs[i],
                 "us": round(per_node[i] * 1e3, 2)}
        if per_node[i] > 0 and by > 0:
            entry.update({k: v for k, v in roofline_entry(fl, by, bound, per_node[i] * 1e-3).items()
                          if k in ("bound", "frac", "achieved", "unit")})
        layers.append(entry)
    fl, by, bound = node_work(desc, nodes, shapes, dom)
    roof = roofline_entry(fl, by, bound, dom_ms * 1e-3)
    dom_layer = desc["ops"][nodes[dom]["tensor"]]["name"]
    roof.update({"kernel": nodes[dom]["kind"], "layer": dom_layer, "config": configs[dom],
                 "timed_launches": len(dev),
                 "algorithmic_bytes": int(by), "algorithmic_flops": int(fl),
                 "avg_launch_us": round(dom_ms * 1e3, 3),
                 "traffic": measured_traffic(nodes[dom]["kind"], dom_layer, configs[dom])})
    total_s = t1 - t0
    res = {"desc": desc, "batch": batch, "net": net, "ms_per_step": total_s / steps * 1e3,
           "images_per_s": batch * steps / total_s, "roofline": roof, "layers": layers,
           "sum_layer_us": sum(per_node) * 1e3,
           "step_ms_device": {k: round(v, 5) for k, v in step_ms.items()}}
    plan.close()
    return res


def config_sweep(key, reps):
    """Every candidate kernel configuration of every node, one node at a time
    (the others on their finalize-time choice), each run `reps` whole-plan
    times; prints the run order as JSON.  The HBM traffic counters are taken
    over this sequence so that every (layer, configuration) pair the
    autotuner may pick has its own figure."""
    import torch
    import workloads
    from paper_1907_01989_amd import _binding as B
    from paper_1907_01989_amd import engine

    net, batch = WORKLOADS[key]
    desc = workloads.WORKLOADS[net](batch)
    plan = engine.Plan(desc)
    xs = plan.input_tensors()
    outs = plan.alloc_outputs()
    sh = torch.cuda.current_stream().cuda_stream
    ins = [x.data_ptr() for x in xs]
    ops_ptrs = [o.data_ptr() for o in outs]
    nodes = plan.nodes()
    runs = []
    for i in range(len(nodes)):
        c0, n, _ = plan.node_configs()[i]
        for c in range(n):
            B.mgi_plan_set_node_config(plan.handle, i, c)
            for _ in range(reps):
                B.mgi_plan_run(plan.handle, ins, ops_ptrs, sh)
            runs.append({"node": i, "configs": [name for _, _, name in plan.node_configs()]})
        B.mgi_plan_set_node_config(plan.handle, i, c0)
    torch.cuda.synchronize()
    layers = [{"node": i, "kind": nd["kind"],
               "name": desc["ops"][nd["tensor"]]["name"] if nd["tensor"] >= 0 else nd["kind"]}
              for i, nd in enumerate(nodes)]
    print(json.dumps({"config_sweep": runs, "reps": reps, "layers": layers,
                      "kernel_sources": kernel_sources_hash()}), flush=True)
    plan.close()


def run_graph_replay(key, steps, warmup, hip, tune=True):
    """The same workload with the launch list captured once as a HIP graph and
    replayed per step (mgi_plan_capture / mgi_plan_replay)."""
    import torch
    import workloads
    from paper_1907_01989_amd import engine

    net, batch = WORKLOADS[key]
    desc = workloads.WORKLOADS[net](batch)
    plan = engine.Plan(desc)
    xs = plan.input_tensors()
    sh = torch.cuda.current_stream().cuda_stream
    if tune:
        plan.autotune(xs, reps=10, stream=sh)
    plan.capture(xs)
    for _ in range(warmup):
        plan.replay(sh)
    marks = [hip.event() for _ in range(21)]     # per-step device time: untimed pass
    for k in range(20):
        hip.record(marks[k], sh)
        plan.replay(sh)
    hip.record(marks[20], sh)
    torch.cuda.synchronize()
    step_ms = percentiles([hip.elapsed_ms(marks[k], marks[k + 1]) for k in range(20)])
    for e in marks:
        hip.destroy(e)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        plan.replay(sh)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    plan.close()
    total_s = t1 - t0
    return {"images_per_s": batch * steps / total_s, "ms_per_step": total_s / steps * 1e3,
            "step_ms_device": {k: round(v, 5) for k, v in step_ms.items()}}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(net, batch):
    """The oracle, as it stands, timed on this host on bounded samples of the
    workload (about 10-20 s of CPU work in all):
      threads_all  the whole batch in one oracle run with all the process's
                   cores (the reported value, in images/s);
      threads_1    a 4-image slice of the same batch on one thread;
      b1           single-image passes of the network with all cores."""
    import oracle
    import workloads
    cores = len(os.sched_getaffinity(0))
    desc = workloads.WORKLOADS[net](batch)
    oracle.lib()
    prev = oracle.set_threads(cores)

    def timed(d, n_images, threads):
        oracle.set_threads(threads)
        t0 = time.perf_counter()
        oracle.run_graph(d, keep=d["outputs"])
        el = time.perf_counter() - t0
        return n_images / el, el

    try:
        # the batch itself, all cores (a batch of 1 repeats until ~3 s)
        if batch > 1:
            v_all, el_all = timed(desc, batch, cores)
            what = f"the {batch}-image batch of {desc['name']} in one oracle run"
        else:
            n, t0 = 0, time.perf_counter()
            while time.perf_counter() - t0 < 3.0:
                oracle.run_graph(desc, keep=desc["outputs"])
                n += 1
            el_all = time.perf_counter() - t0
            v_all = n / el_all
            what = f"{n} single-image passes of {desc['name']}"
        sub = workloads.subset_batch(desc, list(range(min(4, batch))))
        v_1, el_1 = timed(sub, min(4, batch), 1)
        d1 = workloads.WORKLOADS[net](1)
        n, t0 = 0, time.perf_counter()
        oracle.set_threads(cores)
        while time.perf_counter() - t0 < 2.0:
            oracle.run_graph(d1, keep=d1["outputs"])
            n += 1
        v_b1 = n / (time.perf_counter() - t0)
    finally:
        oracle.set_threads(prev)
    return {"value": round(v_all, 4), "unit": "images/sec", "cores": cores, "kind": "oracle",
            "sample": f"{what} (float64, plain loops, {cores} threads, {el_all:.1f} s); "
                      f"1 thread: 4 images of the same batch, {el_1:.1f} s",
            "threads_all": round(v_all, 4), "threads_1": round(v_1, 4),
            "b1_threads_all": round(v_b1, 4), "cpu_model": cpu_model()}


def run_with_h2d(key, steps, warmup, hip):
    """Secondary figure: each step first copies the batch's input from pinned
    host memory to the device input buffer, on the run's stream, then runs the
    plan (Sec. 6 measures with device-resident I/O; this adds the host side)."""
    import torch
    import workloads
    from paper_1907_01989_amd import engine

    net, batch = WORKLOADS[key]
    desc = workloads.WORKLOADS[net](batch)
    plan = engine.Plan(desc)
    xs = plan.input_tensors()
    outs = plan.alloc_outputs()
    host = [x.cpu().pin_memory() for x in xs]
    sh = torch.cuda.current_stream().cuda_stream
    plan.autotune(xs, outs, reps=10, stream=sh)

    def step():
        for h, x in zip(host, xs):
            x.copy_(h, non_blocking=True)
        plan.run(xs, outs, stream=sh)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    total_s = time.perf_counter() - t0
    nbytes = sum(h.numel() * h.element_size() for h in host)
    plan.close()
    return {"images_per_s": round(batch * steps / total_s, 1), "ms_per_step": round(total_s / steps * 1e3, 4),
            "h2d_bytes_per_step": nbytes}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="v1_b64", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true")
    ap.add_argument("--fuse-dwpw", action="store_true",
                    help="fuse 3x3 depthwise convolutions into the pointwise convolutions "
                         "that consume them (mgi_options.fuse_dwpw)")
    ap.add_argument("--no-fuse-pwdw", action="store_true",
                    help="keep pointwise convolutions and the 3x3 depthwise convolutions "
                         "that read them as separate kernels (mgi_options.fuse_pwdw = 0)")
    ap.add_argument("--no-fuse-stemdw", action="store_true",
                    help="keep the stem and the depthwise convolution that reads it as separate "
                         "kernels (mgi_options.fuse_stemdw = 0)")
    ap.add_argument("--no-autotune", action="store_true",
                    help="keep the finalize-time kernel configurations")
    ap.add_argument("--copy-only", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB, 20 times (the "
                         "reference kernel for scaling HBM traffic counters)")
    ap.add_argument("--config-sweep", type=int, default=0, metavar="REPS",
                    help="only run every candidate configuration of every node of the workload "
                         "REPS times, one node at a time (the sequence the HBM traffic counters "
                         "are collected over), and print the order as JSON")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this engine runs on one GPU; --gpus {args.gpus} is not supported "
              "(batch sharding across GPUs is described in the design notes, not built)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        eprint("bench.py: no GPU visible")
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_only:
        n = args.copy_only * 1024 * 1024
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(20):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 20}), flush=True)
        return
    if args.config_sweep:
        config_sweep(args.workload, args.config_sweep)
        return
    hip = Hip()
    eprint(f"[bench] workload {args.workload}: warmup {args.warmup}, steps {args.steps}")
    tune = not args.no_autotune
    main_res = run_workload(args.workload, args.steps, args.warmup, hip, tune=tune,
                            fuse_dwpw=args.fuse_dwpw, fuse_pwdw=not args.no_fuse_pwdw,
                            fuse_stemdw=not args.no_fuse_stemdw)
    eprint(f"[bench] {main_res['images_per_s']:.1f} images/s, {main_res['ms_per_step']:.4f} ms/step")
    also = {}
    if not args.no_extra:
        # every configuration of the metric: the single depthwise-separable
        # block, both networks at batch 1 and 64, and the 513x513 dense net
        for key in ("dw_block", "v1_b1", "v2_b1", "v1_b64", "v2_b64", "deeplab"):
            if key == args.workload:
                continue
            r = run_workload(key, 100, 10, hip, detail=False, tune=tune)
            also[key] = {"images_per_s": round(r["images_per_s"], 1),
                         "ms_per_step": round(r["ms_per_step"], 4),
                         "step_ms_device": r["step_ms_device"]}
            eprint(f"[bench] {key}: {r['images_per_s']:.1f} images/s")
        for key in ("v1_b1", "v2_b1", "v1_b64", "v2_b64"):
            r = run_graph_replay(key, 100, 10, hip, tune=tune)
            also[key + "_graph"] = {"images_per_s": round(r["images_per_s"], 1),
                                    "ms_per_step": round(r["ms_per_step"], 4),
                                    "step_ms_device": r["step_ms_device"]}
            eprint(f"[bench] {key} graph replay: {r['images_per_s']:.1f} images/s")
        r = run_with_h2d(args.workload, 50, 5, hip)
        also[args.workload + "_with_h2d"] = r
        eprint(f"[bench] {args.workload} with the input copied from pinned host memory each step: "
               f"{r['images_per_s']:.1f} images/s")
    cpu = None
    if not args.no_cpu_baseline:
        net0, batch0 = WORKLOADS[args.workload]
        cpu = cpu_baseline(main_res["net"], batch0)
        eprint(f"[bench] cpu oracle: {cpu}")
    net, batch = WORKLOADS[args.workload]
    out = {
        "metric": "images/sec MobileNet-v1/v2 224 fp16 at batch 1 and 64; per-layer % roofline",
        "value": round(main_res["images_per_s"], 2),
        "unit": "images/sec",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_res["ms_per_step"], 5),
        "step_ms_device": main_res["step_ms_device"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp16",
        "data": "synthetic",
        "config": {"workload": main_res["desc"]["name"], "network": net, "batch": batch,
                   "input": "NHWC fp16 uniform[0,1], device-resident",
                   "weights": "He-normal seed 0, fp16", "planner": "greedy", "fused": True,
                   "autotuned": tune, "dw_pw_fused": args.fuse_dwpw,
                   "pw_dw_fused": not args.no_fuse_pwdw, "stem_dw_fused": not args.no_fuse_stemdw},
        "roofline": main_res["roofline"],
        "cpu_baseline": cpu,
        "per_layer": main_res["layers"],
        "sum_of_layer_us": round(main_res["sum_layer_us"], 2),
        "also": also,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

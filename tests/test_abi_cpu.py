"""Host-side tests of the C ABI (no GPU call is made).

The library is loaded, its exports are checked against include/mgi.h, and the
pure-host entry points (graph building, validation, fusion, planning) are run
and compared with the oracle planner.
"""
import ctypes
import os
import random
import re

import numpy as np
import pytest

import oracle
import workloads
from oracle import planner as oplan
from workloads import ACT_NONE, NetBuilder
from paper_1907_01989_amd import _binding as B
from paper_1907_01989_amd import engine

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "mgi.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mgi_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 30
    L = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(L, n), f"{n} declared in mgi.h but not exported"
    assert set(names) == set(B._SIGS), "binding and header disagree"


def test_status_strings():
    assert B.mgi_status_str(0) == "MGI_OK"
    assert B.mgi_status_str(3) == "MGI_ERR_UNSUPPORTED"
    assert B.mgi_status_str(8) == "MGI_ERR_INTERNAL"
    assert B.mgi_status_str(99) == "MGI_ERR_UNKNOWN"


def err(fn, *a, **k):
    with pytest.raises(B.MgiError) as e:
        fn(*a, **k)
    return e.value.status


def test_graph_validation_errors():
    L = B.lib()
    g = B.mgi_graph_create()
    try:
        assert err(B.mgi_graph_add_input, g, 0, 4, 4, 3) == 1
        assert err(B.mgi_graph_add_input, g, 1, 4, 4, 3, B.DTYPE_INT32) == 3
        x = B.mgi_graph_add_input(g, 1, 4, 4, 8)
        w = np.zeros((8, 3, 3, 8), np.float32)
        # bad stride, window larger than padded input, bad tensor id, bad activation
        assert err(B.mgi_graph_add_conv2d, g, x, B.conv_desc(3, 3, (0, 1), cout=8), w) == 1
        assert err(B.mgi_graph_add_conv2d, g, x, B.conv_desc(7, 7, cout=8), np.zeros((8, 7, 7, 8), np.float32)) == 2
        assert err(B.mgi_graph_add_conv2d, g, 5, B.conv_desc(3, 3, cout=8), w) == 1
        assert err(B.mgi_graph_add_conv2d, g, x, B.conv_desc(3, 3, cout=8, act=7), w) == 1
        y = B.mgi_graph_add_conv2d(g, x, B.conv_desc(3, 3, pads=(1, 1, 1, 1), cout=8), w)
        z = B.mgi_graph_add_input(g, 1, 4, 4, 16)
        assert err(B.mgi_graph_add_add, g, y, z) == 2
        assert err(B.mgi_graph_add_fc, g, y, 10, np.zeros((10, 128), np.float32)) == 3
        other = B.mgi_graph_add_input(g, 2, 4, 4, 8)
        assert err(B.mgi_graph_add_concat, g, [y, other]) == 2
        assert err(B.mgi_graph_mark_output, g, x) == 3
        B.mgi_graph_mark_output(g, y)
        assert err(B.mgi_graph_mark_output, g, y) == 1
        # null pointers straight through the C ABI
        assert L.mgi_graph_add_input(g, 1, 1, 1, 1, 2, None) == 1
        assert L.mgi_graph_add_conv2d(g, x, None, None, None, None) == 1
        assert L.mgi_graph_finalize(None, None, None) == 1
        assert "null" in B.mgi_last_error()
    finally:
        B.mgi_graph_destroy(g)
    assert B.lib().mgi_graph_destroy(None) == 0
    assert B.lib().mgi_plan_destroy(None) == 0


def test_finalize_state_errors_and_run_before_bind():
    g = B.mgi_graph_create()
    try:
        x = B.mgi_graph_add_input(g, 1, 4, 4, 8)
        y = B.mgi_graph_add_activation(g, x, B.ACT_RELU)
        assert err(B.mgi_graph_finalize, g) == 4          # no output marked
        B.mgi_graph_mark_output(g, y)
        o = B.mgi_options_default()
        o.planner = 9
        assert err(B.mgi_graph_finalize, g, o) == 3
        p = B.mgi_graph_finalize(g)
    finally:
        B.mgi_graph_destroy(g)
    try:
        assert err(B.mgi_plan_run, p, [1], [1]) == 4        # not bound
        assert err(B.mgi_plan_capture, p, [1], [1]) == 4    # not bound
        assert err(B.mgi_plan_autotune, p, [1], [1], None, 0) == 1   # reps out of range
        assert err(B.mgi_plan_autotune, p, [1], [1], None, 3) == 4   # not bound
        assert err(B.mgi_plan_replay, p) == 4               # nothing captured
        assert err(B.mgi_plan_bind, p, 0, 0) == 5           # no buffers
        assert err(B.mgi_plan_bind, p, 0x1001, 0x2000) == 5  # misaligned
        assert err(B.mgi_plan_read_node, p, 0, 0x1000) == 4  # not materialized
        assert err(B.mgi_plan_node_info, p, 99) == 1
    finally:
        B.mgi_plan_destroy(p)


def test_fusion_structure():
    v1 = engine.Plan(workloads.mobilenet_v1(1), bind=False, fuse_pwdw=False, fuse_stemdw=False, fuse_pool=False,
                     fuse_softmax=False)
    kinds = [n["kind"] for n in v1.nodes()]
    assert kinds[0] == "conv_stem" and kinds.count("dw_conv") == 13 and kinds.count("pw_gemm") == 13
    assert kinds[-3:] == ["global_avgpool", "fc_gemm", "softmax"]
    assert len(kinds) == 30
    v2 = engine.Plan(workloads.mobilenet_v2(1), bind=False, fuse_pwdw=False, fuse_stemdw=False, fuse_pool=False,
                     fuse_softmax=False)
    nodes = v2.nodes()
    assert sum(1 for n in nodes if n["n_fused"] == 2) == 10      # residual adds absorbed
    assert not any(n["kind"] == "add" for n in nodes)
    v2u = engine.Plan(workloads.mobilenet_v2(1), fuse=False, bind=False)
    assert sum(1 for n in v2u.nodes() if n["kind"] == "add") == 10
    dl = engine.Plan(workloads.deeplab_v2_os16(1), bind=False)
    assert dl.nodes()[-1]["kind"] == "resize_argmax"


def test_pointwise_depthwise_fusion_structure():
    # v1: pw1..pw12 each feed one depthwise convolution (whole-image tiles on
    # 14x14 and 7x7 planes, row bands on 112..28); dw1 reads the stem (fused
    # with it), pw13 feeds the pooling (fused with it), the FC feeds the
    # softmax (fused with it; the logits are a graph output as well)
    v1 = engine.Plan(workloads.mobilenet_v1(64), bind=False)
    nodes = v1.nodes()
    kinds = [n["kind"] for n in nodes]
    assert kinds.count("pw_dw") == 12 and kinds.count("stem_dw") == 1 and kinds.count("pw_pool") == 1
    assert kinds[0] == "stem_dw" and "dw_conv" not in kinds and "conv_stem" not in kinds
    assert kinds[-2:] == ["pw_pool", "fc_softmax"] and len(kinds) == 15
    k_nostem = [n["kind"] for n in engine.Plan(workloads.mobilenet_v1(64), bind=False, fuse_stemdw=False).nodes()]
    assert k_nostem[:2] == ["conv_stem", "dw_conv"] and len(k_nostem) == 16
    k_nopool = [n["kind"] for n in engine.Plan(workloads.mobilenet_v1(64), bind=False, fuse_pool=False).nodes()]
    assert k_nopool[-3:] == ["pw_gemm", "global_avgpool", "fc_softmax"] and len(k_nopool) == 16
    k_nosm = [n["kind"] for n in engine.Plan(workloads.mobilenet_v1(64), bind=False, fuse_softmax=False).nodes()]
    assert k_nosm[-3:] == ["pw_pool", "fc_gemm", "softmax"] and len(k_nosm) == 16
    # the fused node produces the probabilities; the logits output keeps its buffer
    k_nologits = engine.Plan(workloads.mobilenet_v1(64, logits_output=False), bind=False)
    assert [n["kind"] for n in k_nologits.nodes()][-1] == "fc_softmax" and k_nologits.n_outputs == 1
    for n in nodes:
        if n["kind"] == "pw_dw":
            assert n["n_fused"] == 2
    # the fused node's output is the depthwise tensor
    desc = workloads.mobilenet_v1(64)
    fused_tensors = [n["tensor"] for n in nodes if n["kind"] == "pw_dw"]
    assert all(desc["ops"][t]["op"] == "depthwise" for t in fused_tensors)
    # v2: every expansion feeds the block's depthwise convolution (16 blocks)
    v2 = engine.Plan(workloads.mobilenet_v2(64), bind=False, fuse_irb=False)
    k2 = [n["kind"] for n in v2.nodes()]
    assert k2.count("pw_dw") == 16
    cf = [c for n, c in zip(nodes, v1.node_configs()) if n["kind"] == "pw_dw"]
    assert all(name.startswith(("img", "band")) and k >= 2 for _, k, name in cf)
    # at batch 1 the fused kernel would get 8..16 workgroups: the node runs as
    # the two separate kernels by default, fused when asked for (fuse_pwdw = 2)
    b1 = engine.Plan(workloads.mobilenet_v1(1), bind=False)
    b1c = [c for n, c in zip(b1.nodes(), b1.node_configs()) if n["kind"] == "pw_dw"]
    assert len(b1c) == 12 and all(name.startswith("split") for _, _, name in b1c)
    b1f = engine.Plan(workloads.mobilenet_v1(1), bind=False, fuse_pwdw=2)
    b1fc = [c for n, c in zip(b1f.nodes(), b1f.node_configs()) if n["kind"] == "pw_dw"]
    assert len(b1fc) == 12 and all(name.startswith(("img", "band")) for _, _, name in b1fc)
    for o in (engine.options(fuse_pwdw=3), engine.options(fuse_stemdw=3), engine.options(fuse_stemdw=-1),
              engine.options(fuse_pool=3), engine.options(fuse_softmax=2), engine.options(fuse_irb=3)):
        g = engine.build_graph(workloads.mobilenet_v1(1))
        try:
            assert err(B.mgi_graph_finalize, g, o) == 1
        finally:
            B.mgi_graph_destroy(g)


def test_stem_depthwise_fusion_structure():
    # the stem node absorbs dw1: at batch 64 the fused kernel (4- or 2-row
    # bands, or rolling strips of 14, 15 or 28 rows) is the default and the
    # split pair a candidate; at batch 1 (28 bands) the split pair is the
    # default unless asked for (fuse_stemdw = 2)
    for net in (workloads.mobilenet_v1, workloads.mobilenet_v2):
        p = engine.Plan(net(64), bind=False)
        n0 = p.nodes()[0]
        assert n0["kind"] == "stem_dw" and n0["n_fused"] == 2 and tuple(n0["shape"]) == (64, 112, 112, 32)
        cfg, k, name = p.node_configs()[0]
        assert name == "band4" and k == 6
        names = []
        for c in range(k):
            B.mgi_plan_set_node_config(p.handle, 0, c)
            names.append(p.node_configs()[0][2])
        assert names == ["band4", "band2", "roll14", "roll15r3", "roll28", "split"]
    assert engine.Plan(workloads.mobilenet_v1(1), bind=False).node_configs()[0][2] == "split"
    assert engine.Plan(workloads.mobilenet_v1(1), bind=False, fuse_stemdw=2).node_configs()[0][2] == "band4"
    # a stride-2 depthwise after the stem is not fused
    g = workloads.NetBuilder(0)
    x = g.input(2, 64, 64, 3, 0, 1)
    s = g.conv(x, 32, 3, s=2)
    y = g.dw(s, 3, s=2)
    g.mark_output(y)
    kinds = [n["kind"] for n in engine.Plan(g.graph("s2"), bind=False).nodes()]
    assert kinds[:2] == ["conv_stem", "dw_conv"] and "stem_dw" not in kinds, kinds


def test_standalone_activation_and_add_fusion():
    g = workloads.NetBuilder(0)
    x = g.input(1, 8, 8, 64, -1, 1)
    c = g.conv(x, 16, 1, act=workloads.ACT_NONE)
    a = g.activation(c, workloads.ACT_RELU6)
    d = g.conv(a, 16, 1, act=workloads.ACT_NONE)
    s = g.add(d, a, act=workloads.ACT_RELU)
    g.mark_output(s)
    p = engine.Plan(g.graph("t"), bind=False)
    nodes = p.nodes()
    assert [n["kind"] for n in nodes] == ["ingest", "pw_gemm", "pw_gemm", "export"]
    assert [n["n_fused"] for n in nodes[1:3]] == [2, 2]
    pu = engine.Plan(g.graph("t"), fuse=False, bind=False)
    assert [n["kind"] for n in pu.nodes()] == ["ingest", "pw_gemm", "activation", "pw_gemm", "add",
                                                "export"]


def _kinds(desc, **kw):
    return [n["kind"] for n in engine.Plan(desc, bind=False, **kw).nodes()]


def test_identity_removal_and_pad_merge():
    g = NetBuilder(seed=3)
    x = g.activation(g.input(2, 9, 9, 16, -1, 1), ACT_NONE)       # kept: the input's layout conversion
    a = g.conv(x, 32, 1)
    i1 = g.activation(a, ACT_NONE)                                # a has two consumers: not fusable
    i2 = g.concat([i1])                                            # one-input concat
    i3 = g.resize(i2, 9, 9, True)                                  # resize to its own size
    p1 = g.pad(i3, (0, 1, 0, 1))                                   # TF-style stride-2 padding
    c1 = g.conv(p1, 24, 3, s=2, pads=(0, 0, 0, 0))
    p2 = g.pad(a, (1, 1, 1, 1))
    d1 = g.dw(p2, 3, s=1, pads=(0, 0, 0, 0))
    y = g.add(g.gap(c1), g.gap(g.conv(g.gap(d1), 24, 1)))
    g.gap(d1)                                                      # dead: reaches no output
    g.mark_output(y)
    desc = g.graph("cleanup")
    fused = _kinds(desc)
    assert "pad" not in fused and "concat" not in fused
    assert fused.count("activation") == 1                          # only the one on the graph input
    assert "resize_bilinear" not in fused
    # the dead pool has no node (the pool of the 1x1 convolution is fused into it)
    assert fused.count("global_avgpool") == 2 and fused.count("pw_pool") == 1
    assert fused.count("conv_igemm") == 1 and fused.count("dw_conv") == 1
    unfused = _kinds(desc, fuse=False)
    assert unfused.count("pad") == 2 and "concat" in unfused and "resize_bilinear" in unfused
    # merged pads leave the convolutions' output shapes unchanged
    sh = {n["tensor"]: n["shape"] for n in engine.Plan(desc, bind=False).nodes()}
    ref = oracle.tensor_shapes(desc)
    for t in (c1, d1):
        assert sh[t] == tuple(ref[t])


def test_storage_types():
    d = workloads.WORKLOADS["mobilenet_v1"](1)
    f16 = engine.Plan(d, bind=False)
    bf = engine.Plan(d, bind=False, dtype=B.DTYPE_BF16)
    assert bf.weight_bytes == f16.weight_bytes and bf.workspace_bytes == f16.workspace_bytes
    g = engine.build_graph(d)
    try:
        o = engine.options(dtype=B.DTYPE_FP32)
        assert err(B.mgi_graph_finalize, g, o) == 3
    finally:
        B.mgi_graph_destroy(g)


def test_node_configuration_candidates():
    # every pointwise GEMM and 3x3 depthwise node offers several kernel
    # configurations; index 0 is the finalize-time choice
    d = workloads.WORKLOADS["mobilenet_v2"](2)
    pl = engine.Plan(d, bind=False)
    nodes = pl.nodes()
    cfgs = pl.node_configs()
    for n, (c, k, name) in zip(nodes, cfgs):
        assert c == 0
        if n["kind"] == "pw_gemm":
            assert k >= 5 and name.startswith(("pipe", "slab", "lds"))
        elif n["kind"] == "dw_conv":
            assert k == 3 and name.startswith("rows")
        elif n["kind"] == "pw_dw":
            assert 2 <= k <= 12 and name.startswith(("img", "band", "split"))
        elif n["kind"] == "stem_dw":
            assert k == 6 and name.startswith(("band", "split"))
        elif n["kind"] == "pw_pool":
            assert 5 <= k <= 9 and name.startswith(("pool", "split"))
        elif n["kind"] == "irb":
            assert k >= 3 and name.startswith(("irb", "img", "band", "split3"))
        elif n["kind"] == "fc_gemm":
            assert k >= 1 and name.startswith("fc")
        elif n["kind"] == "fc_softmax":
            assert k >= 2 and name.startswith("fc")
        else:
            assert k == 1
    i = next(j for j, n in enumerate(nodes) if n["kind"] == "pw_gemm")
    B.mgi_plan_set_node_config(pl.handle, i, 2)
    assert pl.node_configs()[i][0] == 2
    assert err(B.mgi_plan_set_node_config, pl.handle, i, 99) == 1
    assert err(B.mgi_plan_set_node_config, pl.handle, 9999, 0) == 1


def test_pad_that_cannot_merge_runs_as_a_node():
    g = NetBuilder(seed=4)
    x = g.activation(g.input(1, 5, 6, 8, -1, 1), ACT_NONE)
    p = g.pad(x, (1, 2, 0, 3))
    y = g.add(p, g.pad(x, (1, 2, 0, 3)))
    g.mark_output(y)
    kinds = _kinds(g.graph("pad_add"))
    assert kinds.count("pad") == 2
    assert err(B.mgi_graph_add_pad, B.mgi_graph_create(), 0, 0, 0, 0, 0) == 1   # no tensor 0


@pytest.mark.parametrize("net,key", [("mobilenet_v1", "MobileNet"), ("mobilenet_v2", "MobileNetV2")])
@pytest.mark.parametrize("fuse", [True, False])
def test_library_memory_report_reproduces_table3(net, key, fuse):
    t3 = {"MobileNet": (9.6, 2.3), "MobileNetV2": (13.2, 4.0)}[key]
    d = workloads.WORKLOADS[net](1, logits_output=False)
    # Algorithm 1 on the model graph: the fusions of two convolution-like ops
    # (which keep the first op's output as a node scratch tensor) are left out
    naive, planned, nobj = engine.Plan(d, fuse=fuse, bind=False, fuse_pwdw=False, fuse_stemdw=False,
                                       fuse_pool=False).memory_report()
    ops, sizes, inter = oplan.graph_problem(d, oracle.tensor_shapes(d))
    _, ref = oplan.greedy(ops, sizes, inter)
    assert planned == oplan.total(ref)
    assert round(planned / 2 ** 20, 1) == t3[1]
    if not fuse:
        assert round(naive / 2 ** 20, 1) == t3[0]
    materialized = engine.Plan(d, fuse=fuse, materialize_all=True, bind=False).memory_report()
    assert materialized[1] == materialized[0] == naive


def to_lifetimes(ops, sizes, inter):
    first, last = oplan.lifetimes(ops, inter)
    consumed = {t for _, ins in ops for t in ins}
    ts = sorted(t for t in inter if t in first)
    return (ts, [sizes[t] for t in ts], [first[t] for t in ts],
            [last[t] if t in consumed else -1 for t in ts])


def test_library_planner_equals_oracle_on_random_dags():
    rng = random.Random(77)
    for _ in range(400):
        n = rng.randint(3, 14)
        ops = [([0], [])]
        for i in range(1, n):
            ops.append(([i], rng.sample(range(i), rng.randint(1, min(3, i)))))
        sizes = {i: rng.choice([16, 32, 48, 64, 100, 128, 256]) for i in range(n)}
        inter = set(range(1, n - 1))
        ts, sz, fi, la = to_lifetimes(ops, sizes, inter)
        obj, osz = B.mgi_planner_assign(B.PLANNER_GREEDY, sz, fi, la)
        ref_assign, ref_obj = oplan.greedy(ops, sizes, inter)
        assert osz == ref_obj
        assert obj == [ref_assign[t] for t in ts]
        nobj, nsz = B.mgi_planner_assign(B.PLANNER_NAIVE, sz, fi, la)
        assert nobj == list(range(len(ts))) and nsz == sz


def test_library_planner_fig5(golden_dir):
    import json
    with open(os.path.join(golden_dir, "fig5_planner_example.json")) as f:
        gd = json.load(f)
    ops = [(o[0], o[1]) for o in gd["graph"]["ops"]]
    sizes = dict(enumerate(gd["graph"]["sizes"]))
    ts, sz, fi, la = to_lifetimes(ops, sizes, set(sizes))
    obj, osz = B.mgi_planner_assign(B.PLANNER_GREEDY, sz, fi, la)
    assert sum(osz) == gd["greedy"]["total"]
    for a, b in gd["greedy"]["reuse"]:
        assert obj[ts.index(a)] == obj[ts.index(b)]


@pytest.mark.parametrize("net,key,mib", [("mobilenet_v1", "MobileNet", 2.7), ("mobilenet_v2", "MobileNetV2", 3.8)])
def test_library_mcfp_reproduces_table3(net, key, mib):
    # Table 3 counts the graph's tensors as given (fusion off); fusing the
    # residual adds of v2 into the projections removes tensors and changes
    # the flow solution, which must stay no larger than the unfused one (the
    # pointwise -> depthwise fusion adds a scratch tensor per fused node and
    # is left out here)
    d = workloads.WORKLOADS[net](1, logits_output=False)
    naive, planned, nobj = engine.Plan(d, planner=B.PLANNER_MCFP, fuse=False, bind=False).memory_report()
    ops, sizes, inter = oplan.graph_problem(d, oracle.tensor_shapes(d))
    _, ref, _ = oplan.mcfp(ops, sizes, inter)
    assert round(planned / 2 ** 20, 1) == mib
    assert planned == oplan.total(ref) and nobj == len(ref)
    fused = engine.Plan(d, planner=B.PLANNER_MCFP, fuse=True, bind=False, fuse_pwdw=False,
                        fuse_stemdw=False, fuse_pool=False).memory_report()
    assert fused[1] <= planned


def test_library_mcfp_matches_oracle_on_random_dags():
    rng = random.Random(99)
    for _ in range(300):
        n = rng.randint(3, 14)
        ops = [([0], [])]
        for i in range(1, n):
            ops.append(([i], rng.sample(range(i), rng.randint(1, min(3, i)))))
        sizes = {i: rng.choice([16, 32, 48, 64, 100, 128, 256]) for i in range(n)}
        inter = set(range(1, n - 1))
        ts, sz, fi, la = to_lifetimes(ops, sizes, inter)
        obj, osz = B.mgi_planner_assign(B.PLANNER_MCFP, sz, fi, la)
        assign = {t: obj[i] for i, t in enumerate(ts)}
        oplan.check_assignment(ops, sizes, inter, assign, osz)
        for k, size in enumerate(osz):
            assert size == max(sizes[t] for t in ts if assign[t] == k)
        _, _, ref_cost = oplan.mcfp(ops, sizes, inter)
        assert oplan.chain_cost(ops, sizes, inter, assign) == ref_cost


def test_library_mcfp_fig5(golden_dir):
    import json
    with open(os.path.join(golden_dir, "fig5_planner_example.json")) as f:
        gd = json.load(f)
    ops = [(o[0], o[1]) for o in gd["graph"]["ops"]]
    sizes = dict(enumerate(gd["graph"]["sizes"]))
    ts, sz, fi, la = to_lifetimes(ops, sizes, set(sizes))
    obj, osz = B.mgi_planner_assign(B.PLANNER_MCFP, sz, fi, la)
    assert sum(osz) == gd["mcfp"]["total"]
    for a, b in gd["mcfp"]["reuse"]:
        assert obj[ts.index(a)] == obj[ts.index(b)]


def test_planner_assign_rejects_bad_lifetimes():
    assert err(B.mgi_planner_assign, B.PLANNER_GREEDY, [4, 4], [0, 3], [2, 1]) == 1
    assert err(B.mgi_planner_assign, 7, [4], [0], [1]) == 3
    assert B.mgi_planner_assign(B.PLANNER_GREEDY, [], [], []) == ([], [])


def test_inverted_residual_block_fusion_structure():
    """MobileNet-v2: each of the 16 expansion -> depthwise -> projection blocks
    (with its residual add where there is one) becomes one node; its output
    is the block's output tensor (the add, else the projection), its
    configurations are the block kernel's, the fused pointwise -> depthwise
    kernel's followed by the projection GEMM, and three separate kernels."""
    desc = workloads.mobilenet_v2(64)
    plan = engine.Plan(desc, bind=False, fuse_irb=True)
    nodes, cfgs = plan.nodes(), plan.node_configs()
    kinds = [n["kind"] for n in nodes]
    assert kinds.count("irb") == 16 and "pw_dw" not in kinds and len(kinds) == 20
    ops = desc["ops"]
    adds = 0
    for n, (cur, k, name) in zip(nodes, cfgs):
        if n["kind"] != "irb":
            continue
        t = n["tensor"]
        assert ops[t]["op"] in ("conv2d", "add")
        adds += ops[t]["op"] == "add"
        assert n["n_fused"] >= (4 if ops[t]["op"] == "add" else 3)
        assert k >= 3 and name.startswith("irb")     # batch 64: the block kernel fills the GPU
    assert adds == 10
    # the unfused plan (the default) keeps the separate projections; batch 1
    # defaults to a split form
    assert len(engine.Plan(desc, bind=False).nodes()) == 36
    b1 = engine.Plan(workloads.mobilenet_v2(1), bind=False, fuse_irb=True)
    for n, (_, k, name) in zip(b1.nodes(), b1.node_configs()):
        if n["kind"] == "irb":
            assert not name.startswith("irb")
    # MobileNet-v1 has no projection after a depthwise convolution's pointwise pair
    assert "irb" not in [n["kind"] for n in engine.Plan(workloads.mobilenet_v1(64), bind=False, fuse_irb=True).nodes()]


def test_softmax_fusion_state_region():
    # the fused FC + softmax node keeps one arrival counter per 16 rows in a
    # state region past the arena: the workspace grows by that region (one
    # 256-byte block for up to 1024 rows), the arena is unchanged
    for d in (workloads.mobilenet_v1(64), workloads.mobilenet_v1(100, logits_output=False)):
        fused = engine.Plan(d, bind=False)
        split = engine.Plan(d, bind=False, fuse_softmax=False)
        assert fused.nodes()[-1]["kind"] == "fc_softmax" and fused.nodes()[-1]["n_fused"] == 2
        assert B.mgi_plan_workspace_bytes(fused.handle) == B.mgi_plan_workspace_bytes(split.handle) + 256


def test_io_counts_and_tensor_checks_before_any_pointer_is_passed():
    """The C calls take pointer arrays with no length: the binding checks the
    counts against the plan, and the engine checks every tensor's device,
    dtype, contiguity and byte size, before the library sees a pointer."""
    import torch

    import workloads
    from paper_1907_01989_amd import engine
    g = workloads.NetBuilder(seed=0)
    x = g.input(1, 8, 8, 3, 0.0, 1.0)
    t = g.conv(x, 16, 3, 2, name="stem")
    p = g.gap(t, name="pool")
    z = g.fc(p, 10, name="fc")
    g.mark_output(z)
    plan = engine.Plan(g.graph("io_checks"), bind=False)
    try:
        assert (plan.n_inputs, plan.n_outputs) == (1, 1)
        with pytest.raises(ValueError, match="1 inputs and 1 outputs"):
            B.mgi_plan_run(plan.handle, [], [1])
        with pytest.raises(ValueError, match="1 inputs and 1 outputs"):
            B.mgi_plan_capture(plan.handle, [1, 2], [1])
        with pytest.raises(ValueError, match="1 inputs and 1 outputs"):
            B.mgi_plan_autotune(plan.handle, [1], [], None, 3)
        with pytest.raises(ValueError, match="node"):
            B.mgi_plan_run_timed(plan.handle, [1], [1], [None], [None])
        with pytest.raises(RuntimeError, match="not bound"):
            plan.run([torch.zeros(1)])
        xin = torch.zeros((1, 8, 8, 3), dtype=torch.float16)
        out = torch.zeros((1, 10), dtype=torch.float32)
        with pytest.raises(ValueError, match="inputs"):
            plan.check_io([], [out])
        with pytest.raises(ValueError, match="inputs"):
            plan.check_io([xin], [out, out])
        with pytest.raises(ValueError, match="input 0: tensor on cpu"):
            plan.check_io([xin], [out])           # host memory is not a device pointer
        with pytest.raises(ValueError, match="expected a torch tensor"):
            plan.check_io([0x1000], [out])
    finally:
        plan.close()


def test_read_node_raw_sizes_and_errors():
    """mgi_plan_read_node_raw: the stored size of a sliced node output can be
    queried without a run; fp32 outputs are refused; a copy needs
    materialize_all and an enqueued run."""
    g = workloads.NetBuilder(seed=0)
    x = g.input(2, 9, 9, 3, 0.0, 1.0)
    t = g.conv(x, 13, 3, 2, name="stem")
    p = g.gap(t, name="pool")
    z = g.fc(p, 10, name="fc")
    g.mark_output(z)
    desc = g.graph("raw")
    plan = engine.Plan(desc, bind=False, materialize_all=True)
    try:
        kinds = [n["kind"] for n in plan.nodes()]
        i_stem = kinds.index("conv_stem")
        n, h, w, c = plan.nodes()[i_stem]["shape"]
        assert B.mgi_plan_read_node_raw(plan.handle, i_stem) == 2 * n * h * w * 16     # 13 -> 2 slices
        i_fc = len(kinds) - 1
        assert err(B.mgi_plan_read_node_raw, plan.handle, i_fc) == 3
        assert err(B.mgi_plan_read_node_raw, plan.handle, 99) == 1
        assert err(B.mgi_plan_read_node_raw, plan.handle, i_stem, 0x1000) == 4       # no run yet
    finally:
        plan.close()
    plan = engine.Plan(desc, bind=False)
    try:
        kinds = [n["kind"] for n in plan.nodes()]
        assert err(B.mgi_plan_read_node_raw, plan.handle, kinds.index("conv_stem"), 0x1000) == 4
    finally:
        plan.close()


def _config_names(plan, i):
    names = []
    for k in range(plan.node_configs()[i][1]):
        B.mgi_plan_set_node_config(plan.handle, i, k)
        names.append(plan.node_configs()[i][2])
    B.mgi_plan_set_node_config(plan.handle, i, 0)
    return names


def test_grid_dependent_candidates():
    # candidates that exist for some grid sizes only: the four-image 7x7 tile
    # where it changes the number of image groups (batch 64, not batch 1);
    # the four-fragment 14x14 tile; weight-slab tiles with the 8-step
    # prefetch, 16-channel slabs and pooled slab tiles only for grids of less
    # than one workgroup per compute unit
    v1 = engine.Plan(workloads.mobilenet_v1(64), bind=False)
    kinds = [n["kind"] for n in v1.nodes()]
    shapes = [n["shape"] for n in v1.nodes()]
    n7 = [i for i, (k, s) in enumerate(zip(kinds, shapes)) if k == "pw_dw" and s[1] == 7 and s[3] == 1024][0]
    assert "img64i4" in _config_names(v1, n7)
    n14 = [i for i, (k, s) in enumerate(zip(kinds, shapes)) if k == "pw_dw" and s[1] == 14 and s[3] == 512][0]
    assert "img64f4" in _config_names(v1, n14)
    pool64 = _config_names(v1, kinds.index("pw_pool"))
    assert not any(n.startswith("poolslab") for n in pool64)
    v1b1 = engine.Plan(workloads.mobilenet_v1(1), bind=False)
    kinds1 = [n["kind"] for n in v1b1.nodes()]
    assert not any(n == "img64i4" for i, k in enumerate(kinds1) if k == "pw_dw" for n in _config_names(v1b1, i))
    pool1 = _config_names(v1b1, kinds1.index("pw_pool"))
    assert {"poolslab64x16p8", "poolslab64x32p8", "poolslab64x64p8"} <= set(pool1)
    v2b1 = engine.Plan(workloads.mobilenet_v2(1), bind=False)
    v2b64 = engine.Plan(workloads.mobilenet_v2(64), bind=False)
    for plan, few in ((v2b1, True), (v2b64, False)):
        for i, n in enumerate(plan.nodes()):
            if n["kind"] != "pw_gemm":
                continue
            names = _config_names(plan, i)
            slabs = [x for x in names if x.startswith("slab")]
            # 16-channel slabs only with the 8-step prefetch, and only for few workgroups
            assert all(x.endswith("p8") for x in slabs if "x16" in x)
            if not few and n["shape"][1] >= 28:
                assert not any(x.endswith("p8") for x in slabs)

"""bf16 storage (mgi_options.dtype = MGI_DTYPE_BF16) against the oracle.

Inputs and weights are rounded to bf16 values first (workloads.as_bf16_graph),
so both sides consume identical numbers; each operator is then held to one
bf16 rounding of its output (half an ulp is 2^-9 relative; the bound leaves a
factor of two) plus fp32 accumulation, on exact operands.  Networks are held
to the drift that bf16 storage alone causes in the exact oracle.
"""
import numpy as np
import pytest

import oracle
import workloads
from workloads import ACT_NONE, ACT_RELU, ACT_RELU6, NetBuilder

from gpu_util import ISO_RTOL_BF16, check_isolated, isolated_reference, log, logits_check, run_gpu

pytestmark = pytest.mark.gpu
BF16 = 1


def run_bf16(g, name):
    desc = workloads.as_bf16_graph(g.graph(name))
    log(f"[case] bf16 {name}")
    _, outs, nodes = run_gpu(desc, materialize_all=True, dtype=BF16)
    return desc, outs, nodes


def check_node(desc, nodes, t):
    check_isolated(f"{desc['name']} t{t}", nodes[t], isolated_reference(desc, t, nodes), rtol=ISO_RTOL_BF16)


def sliced(g, x):
    return g.activation(x, ACT_NONE)


@pytest.mark.parametrize("n,h,w,cin,cout,res", [(2, 13, 11, 96, 40, True), (1, 28, 28, 256, 256, False),
                                                 (3, 7, 7, 24, 144, False), (1, 14, 14, 512, 1024, True)])
def test_bf16_pointwise(n, h, w, cin, cout, res):
    g = NetBuilder(seed=cin)
    x = sliced(g, g.input(n, h, w, cin, -1, 1))
    y = g.conv(x, cout, 1, act=ACT_NONE if res else ACT_RELU6)
    if res:
        y = g.add(y, sliced(g, g.input(n, h, w, cout, -1, 1, name="r")), act=ACT_RELU)
    g.mark_output(y)
    desc, outs, nodes = run_bf16(g, f"pw{cin}x{cout}")
    check_node(desc, nodes, y)


@pytest.mark.parametrize("n,h,w,cin,cout", [(1, 14, 14, 512, 160), (1, 7, 7, 960, 320)])
def test_bf16_pointwise_every_configuration(n, h, w, cin, cout):
    # every candidate kernel configuration of a small-grid pointwise GEMM
    # (pipelined tiles, weight-slab tiles with the 8-step prefetch, 16-channel
    # and up-to-160 KiB slabs) gives the default's bits in bf16 too
    from paper_1907_01989_amd import engine, _binding as B
    g = NetBuilder(seed=cin + cout)
    x = sliced(g, g.input(n, h, w, cin, -1, 1))
    y = g.conv(x, cout, 1, act=ACT_NONE)
    g.mark_output(y)
    desc = workloads.as_bf16_graph(g.graph(f"pwcfg{cin}x{cout}"))
    plan = engine.Plan(desc, bind=False, dtype=BF16)
    idx = [i for i, k in enumerate(plan.nodes()) if k["kind"] == "pw_gemm"]
    assert len(idx) == 1
    ncfg = plan.node_configs()[idx[0]][1]
    names = []
    for c in range(ncfg):
        B.mgi_plan_set_node_config(plan.handle, idx[0], c)
        names.append(plan.node_configs()[idx[0]][2])
    log(f"[case] bf16 {desc['name']} configurations {names}")
    assert any(nm.endswith("p8") for nm in names)
    _, base, _ = run_gpu(desc, materialize_all=False, dtype=BF16)
    for c, nm in enumerate(names):
        _, o, _ = run_gpu(desc, materialize_all=False, dtype=BF16, configs={idx[0]: c})
        np.testing.assert_array_equal(o[0], base[0], err_msg=nm)
    ref = oracle.run_graph(desc, keep=[y], store_bf16=True)[y]
    check_isolated(desc["name"], base[0], ref.reshape(base[0].shape), rtol=ISO_RTOL_BF16)


@pytest.mark.parametrize("k,s,d", [(3, 1, 1), (3, 2, 1), (3, 1, 2), (5, 1, 1)])
def test_bf16_depthwise_and_conv(k, s, d):
    g = NetBuilder(seed=k + s + d)
    x = sliced(g, g.input(2, 17, 15, 40, -1, 1))
    a = g.dw(x, k, s, d)
    b = g.conv(x, 24, 3, s, d)
    g.mark_output(a)
    g.mark_output(b)
    desc, outs, nodes = run_bf16(g, f"dwconv_k{k}s{s}d{d}")
    check_node(desc, nodes, a)
    check_node(desc, nodes, b)


@pytest.mark.parametrize("fp16_in", [False, True])
def test_bf16_stem(fp16_in):
    g = NetBuilder(seed=5)
    x = g.input(2, 31, 33, 3, 0, 1, dtype=workloads.DTYPE_FP16 if fp16_in else workloads.DTYPE_FP32)
    y = g.conv(x, 32, 3, 2)
    g.mark_output(y)
    desc, outs, nodes = run_bf16(g, f"stem_f16in{int(fp16_in)}")
    check_node(desc, nodes, y)


def test_bf16_head_and_glue():
    g = NetBuilder(seed=9)
    x = sliced(g, g.input(3, 9, 9, 20, -1, 1))
    p = g.gap(x)
    z = g.fc(p, 37)
    sm = g.softmax(z)
    cat = g.concat([x, g.activation(x, ACT_RELU)])
    up = g.resize(cat, 17, 17, True)
    lab = g.argmax(g.resize(x, 33, 33, True))
    pad = g.add(g.pad(x, (1, 0, 2, 1)), g.pad(x, (0, 1, 1, 2)))
    for t in (z, sm, up, lab, pad):
        g.mark_output(t)
    desc, outs, nodes = run_bf16(g, "glue")
    ref = oracle.run_graph(desc)
    for t in (p, up, pad):
        check_node(desc, nodes, t)
    rel, tg, tr, _ = logits_check(outs[0].reshape(3, -1), isolated_reference(desc, z, nodes).reshape(3, -1))
    assert rel.max() < 4e-3 and (tg == tr).all()
    np.testing.assert_allclose(outs[1].reshape(3, -1), oracle.softmax(isolated_reference(desc, z, nodes)).reshape(3, -1),
                               rtol=1e-4, atol=1e-6)
    # labels: equal wherever the oracle's top-2 margin exceeds the bf16 error of the upsampled values
    upr = oracle.resize_bilinear(isolated_reference(desc, lab - 1, nodes), 33, 33, 1)
    srt = np.sort(upr, axis=-1)
    mask = (srt[..., -1] - srt[..., -2]) > 2.0 ** -6 * np.abs(upr).max()
    got = outs[3].reshape(mask.shape)
    assert ((got == upr.argmax(-1)) | ~mask).all()


@pytest.mark.parametrize("net", ["mobilenet_v1", "mobilenet_v2"])
def test_bf16_network_logits(net):
    desc = workloads.as_bf16_graph(workloads.WORKLOADS[net](1))
    log(f"[case] bf16 {net} b1")
    _, outs, _ = run_gpu(desc, materialize_all=False, dtype=BF16)
    t_logits = desc["outputs"][0]
    exact = oracle.run_graph(desc, keep=[t_logits])[t_logits].reshape(1, -1)
    emul = oracle.run_graph(desc, keep=[t_logits], store_bf16=True)[t_logits].reshape(1, -1)
    drift = float(np.linalg.norm(emul - exact) / np.linalg.norm(exact))
    rel, tg, tr, gap = logits_check(outs[0].reshape(1, -1), exact)
    log(f"[case] relL2 {rel[0]:.3e}  bf16 storage drift of the oracle {drift:.3e}  top-2 gap {gap[0]:.3e}")
    assert rel[0] <= max(1e-2, 2.0 * drift)
    assert tg[0] == emul.argmax() or gap[0] < 4 * float(np.abs(outs[0] - exact).max())

"""End-to-end parity of the five workloads against the oracle, layer by layer.

Each side consumes its own previous outputs (a chained check): the GPU keeps
fp16 activations with fp32 accumulation, the oracle computes in float64.
Bars, per fused node output (real channels, every image checked):
  * isolated: within single-op rounding of the oracle run on the node's own
    GPU inputs (this is where a kernel error shows);
  * chained, float64 oracle: max|gpu - ref| <= 2e-2 * max|ref| for the
    dw-separable block and MobileNet-v1; for MobileNet-v2 and the DeepLab-style
    network, whose float64 chains drift further than that under fp16 storage
    alone, the bar is max(2e-2, 2 x that drift), the drift being that of the
    fp16-storage oracle ref16: the float64 chain that rounds each stored tensor
    to fp16 where the engine stores fp16 (fp16 storage, exact arithmetic);
  * chained, fp16-storage oracle: max|gpu - ref16| within the same bar.
Logits: relative L2 <= 1e-2 per image with the same top-1 class, on all
images of a batch; probabilities equal to the softmax of the GPU's own logits
and within the factor exp(+-2 max|dlogit|) of the oracle's.  Segmentation labels: equal wherever the oracle's top-2
margin exceeds twice the largest logit deviation, and at margin 1e-2 no more
mismatches than the fp16-storage oracle itself has.
"""
import numpy as np
import pytest

import oracle
import workloads

from gpu_util import (LAYER_TOL, LOGITS_RELL2, check_isolated, check_layer, isolated_reference,
                      labels_check, layer_error, log, logits_check, run_gpu)

pytestmark = pytest.mark.gpu

# networks whose float64 chain stays within the flat bar under fp16 storage
FLAT_BAR = {"dw_block", "mobilenet_v1"}


def per_layer(desc, nodes, ref, ref16, images=None, flat=True):
    """Per-layer checks on every fused node output (see the module docstring)."""
    bad = []
    gvals = {t: (g[images] if images is not None else g) for t, g in nodes.items()}
    for t, g in sorted(gvals.items()):
        if t not in ref or desc["ops"][t]["op"] == "argmax":
            continue
        r = ref[t]
        g = g.reshape(r.shape)
        name = f"{t}:{desc['ops'][t]['name']}"
        iso = isolated_reference(desc, t, gvals)
        try:
            check_isolated(f"{name} isolated", g, iso)
        except AssertionError as e:
            bad.append(str(e))
        drift16, denom = layer_error(ref16[t], r)
        drift = drift16 / max(denom, 1e-30)
        tol = LAYER_TOL if flat else max(LAYER_TOL, 2.0 * drift)
        ok, msg = check_layer(name, g, r, tol)
        ok16, msg16 = check_layer(f"{name} vs fp16-storage oracle", g, ref16[t], tol)
        rel2 = float(np.linalg.norm(np.asarray(g, np.float64) - r) / max(np.linalg.norm(r), 1e-30))
        log(f"   {msg} relL2={rel2:.2e} (fp16-storage drift {drift:.3e}, bar {tol:.3e}); "
            f"vs fp16-storage oracle {msg16.split(': ', 1)[1]}")
        if not ok:
            bad.append(msg)
        if not ok16:
            bad.append(msg16)
    assert not bad, "layers out of tolerance:\n" + "\n".join(bad)


def classify_checks(desc, outs, ref, images=None):
    """Logits relative L2 and top-1 per image, probabilities elementwise.  An
    image whose oracle top-1/top-2 gap is under 10x its largest logit error is
    flagged (logged): its top-1 agreement then says little."""
    logit_t, prob_t = desc["outputs"][0], desc["outputs"][1]
    gl, gp = outs[0], outs[1]
    if images is not None:
        gl, gp = gl[images], gp[images]
    rl = ref[logit_t].reshape(gl.shape)
    rel, tg, tr, gap = logits_check(gl, rl)
    err = np.abs(np.asarray(gl, np.float64).reshape(len(rel), -1) - rl.reshape(len(rel), -1)).max(1)
    flagged = np.nonzero(gap < 10.0 * err)[0]
    log(f"   logits relL2 max={rel.max():.3e} over {len(rel)} images; top1 gpu={tg.tolist()[:8]} "
        f"ref={tr.tolist()[:8]} ({len(set(tr.tolist()))} distinct); min top-2 gap={gap.min():.3e}, "
        f"max |dlogit|={err.max():.3e}, min gap/err={(gap / np.maximum(err, 1e-30)).min():.1f}")
    for i in flagged:
        log(f"   FLAG image {i}: oracle top-2 gap {gap[i]:.3e} < 10 x logit error {err[i]:.3e}")
    # the input-dependent part of the logits (each image minus the batch mean)
    if len(rel) > 1:
        gc = np.asarray(gl, np.float64).reshape(len(rel), -1)
        rc = rl.reshape(len(rel), -1)
        gc = gc - gc.mean(0)
        rc = rc - rc.mean(0)
        relc = np.linalg.norm(gc - rc, axis=1) / np.linalg.norm(rc, axis=1)
        log(f"   input-dependent logits (minus batch mean) relL2 max={relc.max():.3e}, "
            f"mean={relc.mean():.3e}")
    assert (rel <= LOGITS_RELL2).all(), rel
    assert (tg == tr).all()
    # probabilities: the softmax of the GPU's own logits (isolated, fp32
    # rounding only); against the oracle's, the bound the logit error implies:
    # if every logit moves by at most M, every probability moves by a factor
    # within [exp(-2M), exp(2M)]
    gp = np.asarray(gp, np.float64).reshape(len(rel), -1)
    iso = oracle.softmax(np.asarray(gl, np.float64).reshape(len(rel), -1))
    np.testing.assert_allclose(gp, iso, rtol=1e-5, atol=1e-9)
    rp = ref[prob_t].reshape(gp.shape)
    bound = rp * (np.expm1(2.0 * err)[:, None] + 1e-5) + 1e-9
    relp = np.linalg.norm(gp - rp, axis=1) / np.linalg.norm(rp, axis=1)
    log(f"   probabilities relL2 max={relp.max():.3e}; worst |dp| / bound = "
        f"{(np.abs(gp - rp) / bound).max():.3f}")
    assert (np.abs(gp - rp) <= bound).all()


@pytest.mark.parametrize("name", ["dw_block", "mobilenet_v1", "mobilenet_v2"])
def test_network_b1(name):
    desc = workloads.WORKLOADS[name](1)
    log(f"[net] {desc['name']}")
    plan, outs, nodes = run_gpu(desc, materialize_all=True)
    ref = oracle.run_graph(desc)
    ref16 = oracle.run_graph(desc, store_fp16=True)
    per_layer(desc, nodes, ref, ref16, flat=name in FLAT_BAR)
    if name != "dw_block":
        classify_checks(desc, outs, ref)
    else:
        ok, msg = check_layer("output", outs[0], ref[desc["outputs"][0]])
        assert ok, msg
    # the greedy-planned launch sequence gives bit-identical outputs
    _, outs_g, _ = run_gpu(desc, materialize_all=False)
    for a, b in zip(outs_g, outs):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name", ["mobilenet_v1", "mobilenet_v2"])
def test_network_b64(name):
    """Full batch of 64 with the greedy plan the benchmark runs: logits and
    top-1 of all 64 images against the oracle; per-layer checks on three
    images (batch entries are independent) from a run that keeps every node
    output."""
    desc = workloads.WORKLOADS[name](64)
    log(f"[net] {desc['name']} (all 64 images)")
    _, outs, _ = run_gpu(desc, materialize_all=False)
    ref = oracle.run_graph(desc, keep=desc["outputs"])
    classify_checks(desc, outs, ref)
    images = [0, 31, 63]
    _, outs_m, nodes = run_gpu(desc, materialize_all=True)
    for a, b in zip(outs, outs_m):
        np.testing.assert_array_equal(a, b)
    sub = workloads.subset_batch(desc, images)
    log(f"   per-layer on images {images}")
    per_layer(sub, nodes, oracle.run_graph(sub), oracle.run_graph(sub, store_fp16=True), images,
              flat=name in FLAT_BAR)


def test_deeplab_513():
    desc = workloads.deeplab_v2_os16(1)
    log(f"[net] {desc['name']}")
    plan, outs, nodes = run_gpu(desc, materialize_all=True)
    ref = oracle.run_graph(desc)
    names = {op["name"]: i for i, op in enumerate(desc["ops"])}
    ref16 = oracle.run_graph(desc, store_fp16=True)
    per_layer(desc, nodes, ref, ref16, flat=False)
    # labels against the oracle's resize + argmax of the GPU's own logits
    # (isolated), and against the float64 chain where its top-2 margin > 1e-2
    iso_up = oracle.resize_bilinear(nodes[names["logits"]].astype(np.float64), 513, 513, True)
    bad_iso, cov_iso, _ = labels_check(outs[1], iso_up, margin=1e-4)
    log(f"   labels vs isolated upsample: {bad_iso} mismatches (margin > 1e-4 covers {cov_iso:.5f})")
    assert bad_iso == 0 and cov_iso > 0.99
    # against the float64 chain: bilinear weights are convex, so a label can
    # only change where the top-2 margin is below 2 * max |logit deviation|;
    # above that margin the labels must be identical.
    lg = nodes[names["logits"]].reshape(ref[names["logits"]].shape)
    dmax = float(np.abs(lg - ref[names["logits"]]).max())
    bad, covered, raw = labels_check(outs[1], ref[names["upsample"]], margin=2 * dmax)
    log(f"   labels: {bad} mismatches where margin > 2*max|dlogits| = {2 * dmax:.3e} "
        f"(covering {covered:.4f}); {raw} overall")
    assert bad == 0
    assert covered > 0.5
    # the stated criterion, labels equal wherever the float64 oracle's top-2
    # margin exceeds 1e-2: fp16 storage alone breaks it (the fp16-storage
    # oracle chain misses b16 of those pixels), so the GPU must do no worse
    # than fp16 storage itself; against the fp16-storage oracle's own labels
    # and margins the same criterion is asserted on its own.
    up16 = ref16[names["upsample"]]
    b16, _, _ = labels_check(up16.argmax(-1), ref[names["upsample"]])
    b_gpu, cov, _ = labels_check(outs[1], ref[names["upsample"]])
    b_vs16, cov16, _ = labels_check(outs[1], up16)
    log(f"   margin > 1e-2 of the float64 oracle (covering {cov:.4f}): gpu {b_gpu} mismatches, "
        f"fp16-storage oracle {b16}; against the fp16-storage oracle (covering {cov16:.4f}): "
        f"{b_vs16} mismatches")
    assert b_gpu <= b16
    _, outs_g, _ = run_gpu(desc, materialize_all=False)
    for a, b in zip(outs_g, outs):
        np.testing.assert_array_equal(a, b)

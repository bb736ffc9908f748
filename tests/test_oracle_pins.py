"""Pins of the CPU oracle against facts fixed by mathematics and by the paper.

Each check is chosen so that a plausible slip in the oracle (a dropped tap, a
wrong padding offset, a transposed weight, a swapped interpolation weight, a
wrong activation bound) fails at least one of them.
"""
import math

import numpy as np
import pytest

import oracle
import workloads


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ----------------------------------------------------------------------------
# convolution
# ----------------------------------------------------------------------------
def test_delta_kernel_reproduces_input():
    x = rnd((2, 7, 9, 5), 1)
    w = np.zeros((5, 3, 3, 5))
    for c in range(5):
        w[c, 1, 1, c] = 1.0
    y = oracle.conv2d(x, w, None, (1, 1), (1, 1), (1, 1, 1, 1))
    np.testing.assert_array_equal(y, x)
    wd = np.zeros((5, 3, 3))
    wd[:, 1, 1] = 1.0
    np.testing.assert_array_equal(oracle.depthwise(x, wd, None, (1, 1), (1, 1), (1, 1, 1, 1)), x)


def test_off_centre_delta_shifts_with_zero_fill():
    # a delta at tap (0, 2) reads x[oy - 1, ox + 1]
    x = rnd((1, 5, 6, 3), 2)
    w = np.zeros((3, 3, 3))
    w[:, 0, 2] = 1.0
    y = oracle.depthwise(x, w, None, (1, 1), (1, 1), (1, 1, 1, 1))
    ref = np.zeros_like(x)
    ref[:, 1:, :-1, :] = x[:, :-1, 1:, :]
    np.testing.assert_array_equal(y, ref)


def test_stride2_same_is_subsampled_stride1():
    # TF-SAME at stride 2 on an even size pads (0, 1): output i is stride-1
    # output 2i+1 of the symmetric pad-1 convolution.
    x = rnd((1, 8, 10, 4), 3)
    w = rnd((6, 3, 3, 4), 4)
    b = rnd((6,), 5)
    y2 = oracle.conv2d(x, w, b, (2, 2), (1, 1), (0, 1, 0, 1))
    y1 = oracle.conv2d(x, w, b, (1, 1), (1, 1), (1, 1, 1, 1))
    np.testing.assert_allclose(y2, y1[:, 1::2, 1::2, :], rtol=1e-12, atol=1e-12)


def test_pointwise_equals_matmul():
    x = rnd((3, 4, 5, 16), 6)
    w = rnd((24, 1, 1, 16), 7)
    b = rnd((24,), 8)
    y = oracle.conv2d(x, w, b)
    ref = x.reshape(-1, 16) @ w.reshape(24, 16).T + b
    np.testing.assert_allclose(y.reshape(-1, 24), ref, rtol=1e-12, atol=1e-12)


def test_hand_5x5_all_ones():
    x = np.ones((1, 5, 5, 1))
    w = np.ones((1, 3, 3, 1))
    y = oracle.conv2d(x, w, None, (1, 1), (1, 1), (1, 1, 1, 1))[0, :, :, 0]
    ref = np.array([[4, 6, 6, 6, 4],
                    [6, 9, 9, 9, 6],
                    [6, 9, 9, 9, 6],
                    [6, 9, 9, 9, 6],
                    [4, 6, 6, 6, 4]], float)
    np.testing.assert_array_equal(y, ref)
    yd = oracle.depthwise(x, np.ones((1, 3, 3)), None, (1, 1), (1, 1), (1, 1, 1, 1))[0, :, :, 0]
    np.testing.assert_array_equal(yd, ref)


def test_hand_5x5_ramp_borders():
    # x[h, w] = 10 h + w; kernel with distinct taps k[ky, kx] = 3 ky + kx + 1.
    x = (10 * np.arange(5)[:, None] + np.arange(5)[None, :]).astype(float).reshape(1, 5, 5, 1)
    k = (3 * np.arange(3)[:, None] + np.arange(3)[None, :] + 1).astype(float)
    y = oracle.depthwise(x, k.reshape(1, 3, 3), np.array([0.5]), (1, 1), (1, 1), (1, 1, 1, 1))
    y = y[0, :, :, 0]
    # corner (0,0): taps (1,1)->x[0,0]=0, (1,2)->x[0,1]=1, (2,1)->x[1,0]=10, (2,2)->x[1,1]=11
    assert y[0, 0] == 0.5 + 5 * 0 + 6 * 1 + 8 * 10 + 9 * 11
    # edge (0,2): rows 0..1, cols 1..3 with taps (1,0..2),(2,0..2)
    assert y[0, 2] == 0.5 + (4 * 1 + 5 * 2 + 6 * 3) + (7 * 11 + 8 * 12 + 9 * 13)
    # interior (2,2): full window
    assert y[2, 2] == 0.5 + sum(k[a, b] * x[0, 1 + a, 1 + b, 0] for a in range(3) for b in range(3))
    # bottom-right corner (4,4): rows 3..4, cols 3..4 with taps (0,0),(0,1),(1,0),(1,1)
    assert y[4, 4] == 0.5 + 1 * 33 + 2 * 34 + 4 * 43 + 5 * 44


def test_hand_6x6_stride2_same():
    # 6x6 ramp, 3x3 all-ones, stride 2, TF-SAME pads (0,1): windows start at 0,2,4
    x = np.arange(36, dtype=float).reshape(1, 6, 6, 1)
    y = oracle.conv2d(x, np.ones((1, 3, 3, 1)), None, (2, 2), (1, 1), (0, 1, 0, 1))[0, :, :, 0]
    assert y.shape == (3, 3)
    assert y[0, 0] == sum(6 * r + c for r in range(3) for c in range(3))
    assert y[1, 2] == sum(6 * r + c for r in range(2, 5) for c in range(4, 6))
    assert y[2, 2] == 28 + 29 + 34 + 35


def test_dilation_equals_zero_inserted_kernel():
    x = rnd((1, 9, 8, 3), 9)
    w = rnd((4, 3, 3, 3), 10)
    w5 = np.zeros((4, 5, 5, 3))
    w5[:, ::2, ::2, :] = w
    y = oracle.conv2d(x, w, None, (1, 1), (2, 2), (2, 2, 2, 2))
    ref = oracle.conv2d(x, w5, None, (1, 1), (1, 1), (2, 2, 2, 2))
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    wd = rnd((3, 3, 3), 11)
    wd5 = np.zeros((3, 5, 5))
    wd5[:, ::2, ::2] = wd
    np.testing.assert_allclose(oracle.depthwise(x, wd, None, (1, 1), (2, 2), (2, 2, 2, 2)),
                               oracle.depthwise(x, wd5, None, (1, 1), (1, 1), (2, 2, 2, 2)),
                               rtol=1e-12, atol=1e-12)


def test_depthwise_is_block_diagonal_dense_conv():
    x = rnd((2, 6, 7, 5), 12)
    wd = rnd((5, 3, 3), 13)
    b = rnd((5,), 14)
    dense = np.zeros((5, 3, 3, 5))
    for c in range(5):
        dense[c, :, :, c] = wd[c]
    for stride, pads in (((1, 1), (1, 1, 1, 1)), ((2, 2), (0, 1, 1, 1))):
        np.testing.assert_allclose(oracle.depthwise(x, wd, b, stride, (1, 1), pads),
                                   oracle.conv2d(x, dense, b, stride, (1, 1), pads),
                                   rtol=1e-12, atol=1e-12)


def test_conv_linear_and_translation_equivariant():
    x1, x2 = rnd((1, 10, 10, 3), 15), rnd((1, 10, 10, 3), 16)
    w = rnd((2, 3, 3, 3), 17)
    f = lambda x: oracle.conv2d(x, w, None, (1, 1), (1, 1), (1, 1, 1, 1))
    np.testing.assert_allclose(f(2.0 * x1 - 3.0 * x2), 2.0 * f(x1) - 3.0 * f(x2), atol=1e-11)
    xs = np.roll(x1, (2, 3), axis=(1, 2))
    np.testing.assert_allclose(f(xs)[:, 4:9, 5:9], f(x1)[:, 2:7, 2:6], atol=1e-12)


def im2col_conv(x, w, b, s, d, pads):
    """Independent formulation: gather patches into a matrix, then one matmul."""
    N, H, W, C = x.shape
    CO, KH, KW, _ = w.shape
    pt, pb, pl, pr = pads
    xp = np.pad(x, ((0, 0), (pt, pb), (pl, pr), (0, 0)))
    OH = (H + pt + pb - d * (KH - 1) - 1) // s + 1
    OW = (W + pl + pr - d * (KW - 1) - 1) // s + 1
    cols = np.empty((N, OH, OW, KH, KW, C))
    for ky in range(KH):
        for kx in range(KW):
            cols[:, :, :, ky, kx, :] = xp[:, ky * d: ky * d + s * (OH - 1) + 1: s,
                                          kx * d: kx * d + s * (OW - 1) + 1: s, :]
    return (cols.reshape(-1, KH * KW * C) @ w.reshape(CO, -1).T + b).reshape(N, OH, OW, CO)


@pytest.mark.parametrize("s,d,pads", [(1, 1, (1, 1, 1, 1)), (2, 1, (0, 1, 0, 1)),
                                      (2, 1, (1, 1, 1, 1)), (1, 2, (2, 2, 2, 2)),
                                      (3, 1, (0, 0, 2, 1))])
def test_conv_matches_im2col(s, d, pads):
    x = rnd((2, 7, 8, 5), 18)
    w = rnd((6, 3, 3, 5), 19)
    b = rnd((6,), 20)
    np.testing.assert_allclose(oracle.conv2d(x, w, b, (s, s), (d, d), pads),
                               im2col_conv(x, w, b, s, d, pads), rtol=1e-10, atol=1e-10)


# ----------------------------------------------------------------------------
# element-wise, pooling and head operators
# ----------------------------------------------------------------------------
def test_zero_pad_hand_values():
    x = np.array([[1.0, 2.0], [3.0, 4.0]]).reshape(1, 2, 2, 1)
    y = oracle.zero_pad(x, (1, 0, 0, 2))[0, :, :, 0]
    np.testing.assert_array_equal(y, [[0, 0, 0, 0], [1, 2, 0, 0], [3, 4, 0, 0]])


@pytest.mark.parametrize("pads,s,d", [((1, 1, 1, 1), 1, 1), ((0, 1, 0, 1), 2, 1), ((2, 2, 2, 2), 1, 2),
                                      ((3, 0, 1, 2), 2, 1)])
def test_conv_of_zero_padded_input_equals_padded_conv(pads, s, d):
    # PAD folded into a convolution (Sec. 3.1) is exact: a convolution over a
    # zero-padded tensor equals the convolution with the pads added
    x = rnd((2, 7, 6, 5), 31)
    w = rnd((4, 3, 3, 5), 32)
    b = rnd(4, 33)
    direct = oracle.conv2d(x, w, b, (s, s), (d, d), pads)
    folded = oracle.conv2d(oracle.zero_pad(x, pads), w, b, (s, s), (d, d), (0, 0, 0, 0))
    np.testing.assert_allclose(folded, direct, rtol=0, atol=1e-12)
    wd = rnd((5, 3, 3), 34)
    np.testing.assert_allclose(oracle.depthwise(oracle.zero_pad(x, pads), wd, None, (s, s), (d, d), (0, 0, 0, 0)),
                               oracle.depthwise(x, wd, None, (s, s), (d, d), pads), rtol=0, atol=1e-12)


def test_relu_relu6_hand_values():
    v = np.array([-1.0, 0.0, 3.0, 6.0, 7.5, -0.0, 5.999])
    np.testing.assert_array_equal(oracle.activation(v, 0), v)
    np.testing.assert_array_equal(oracle.activation(v, 1), [0, 0, 3, 6, 7.5, 0, 5.999])
    np.testing.assert_array_equal(oracle.activation(v, 2), [0, 0, 3, 6, 6, 0, 5.999])


def test_add():
    a, b = rnd((2, 3, 4, 5), 21), rnd((2, 3, 4, 5), 22)
    np.testing.assert_array_equal(oracle.add(a, b), a + b)


def test_global_avgpool():
    x = np.full((2, 7, 7, 3), 2.5)
    np.testing.assert_allclose(oracle.global_avgpool(x), np.full((2, 1, 1, 3), 2.5), rtol=1e-15)
    x = rnd((2, 5, 3, 4), 23)
    np.testing.assert_allclose(oracle.global_avgpool(x)[:, 0, 0, :], x.mean(axis=(1, 2)), rtol=1e-12)


def test_fc_equals_matmul():
    x = rnd((3, 1, 1, 20), 24)
    w = rnd((7, 20), 25)
    b = rnd((7,), 26)
    np.testing.assert_allclose(oracle.fc(x, w, b)[:, 0, 0, :], x.reshape(3, 20) @ w.T + b, rtol=1e-12)


def test_softmax_properties():
    np.testing.assert_allclose(oracle.softmax(np.array([[0.0, math.log(2.0)]])), [[1 / 3, 2 / 3]],
                               rtol=1e-15)
    z = rnd((4, 1000), 27) * 3
    p = oracle.softmax(z)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(oracle.softmax(z + 17.0), p, rtol=1e-12)
    assert (p.argmax(axis=1) == z.argmax(axis=1)).all()
    assert (p > 0).all()


def test_concat_order():
    a, b = rnd((1, 2, 3, 4), 28), rnd((1, 2, 3, 2), 29)
    y = oracle.concat([a, b])
    np.testing.assert_array_equal(y[..., :4], a)
    np.testing.assert_array_equal(y[..., 4:], b)


def test_bilinear_align_corners_exact_at_grid_points():
    x = rnd((1, 33, 33, 3), 30)
    y = oracle.resize_bilinear(x, 513, 513, True)
    np.testing.assert_array_equal(y[:, ::16, ::16, :], x)


def test_bilinear_reproduces_affine_and_constants():
    H, W = 5, 4
    hh, ww = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    x = (3.0 * hh - 2.0 * ww + 1.0).reshape(1, H, W, 1)
    y = oracle.resize_bilinear(x, 17, 13, True)
    oy = np.arange(17)[:, None] * (H - 1) / 16.0
    ox = np.arange(13)[None, :] * (W - 1) / 12.0
    np.testing.assert_allclose(y[0, :, :, 0], 3.0 * oy - 2.0 * ox + 1.0, atol=1e-12)
    c = oracle.resize_bilinear(np.full((1, 3, 3, 2), 1.25), 9, 7, True)
    np.testing.assert_array_equal(c, np.full((1, 9, 7, 2), 1.25))
    # a single pixel is broadcast
    one = rnd((2, 1, 1, 3), 31)
    np.testing.assert_array_equal(oracle.resize_bilinear(one, 4, 5, True), np.broadcast_to(one, (2, 4, 5, 3)))


def test_bilinear_midpoint_weights():
    # between samples a and b at fraction 1/4 the value is 3/4 a + 1/4 b
    x = np.array([0.0, 8.0]).reshape(1, 1, 2, 1)
    y = oracle.resize_bilinear(x, 1, 5, True)[0, 0, :, 0]
    np.testing.assert_array_equal(y, [0, 2, 4, 6, 8])
    x = np.array([0.0, 8.0]).reshape(1, 2, 1, 1)
    y = oracle.resize_bilinear(x, 5, 1, True)[0, :, 0, 0]
    np.testing.assert_array_equal(y, [0, 2, 4, 6, 8])


def test_bilinear_half_scale_branch_by_hand():
    """align_corners = 0: output sample d reads source coordinate d * in / out
    (no half-pixel offset), the upper neighbour clamped to the last sample.
    Worked by hand:
      2 -> 4: src = 0, 0.5, 1, 1.5  ->  [a, (a+b)/2, b, b]  (1.5 clamps to b)
      3 -> 2: src = 0, 1.5          ->  [x0, (x1+x2)/2]
      4 -> 3: src = 0, 4/3, 8/3     ->  [x0, x1 + (x2-x1)/3, x2 + 2(x3-x2)/3]
    A half-pixel-centre reading (src = (d+0.5)*in/out - 0.5) would give
    [a, a + (b-a)/4, a + 3(b-a)/4, b] for the first case instead."""
    a, b = 2.0, 10.0
    x = np.array([a, b]).reshape(1, 1, 2, 1)
    np.testing.assert_array_equal(oracle.resize_bilinear(x, 1, 4, False)[0, 0, :, 0],
                                  [2.0, 6.0, 10.0, 10.0])
    np.testing.assert_array_equal(oracle.resize_bilinear(x.reshape(1, 2, 1, 1), 4, 1, False)[0, :, 0, 0],
                                  [2.0, 6.0, 10.0, 10.0])
    x3 = np.array([1.0, 4.0, 10.0]).reshape(1, 1, 3, 1)
    np.testing.assert_array_equal(oracle.resize_bilinear(x3, 1, 2, False)[0, 0, :, 0], [1.0, 7.0])
    x4 = np.array([0.0, 3.0, 9.0, 12.0]).reshape(1, 4, 1, 1)
    np.testing.assert_allclose(oracle.resize_bilinear(x4, 3, 1, False)[0, :, 0, 0],
                               [0.0, 3.0 + 6.0 / 3.0, 9.0 + 2.0 * 3.0 / 3.0], rtol=0, atol=1e-14)
    # 2-D: 2x2 -> 4x4 is the separable product of the 1-D weights above
    q = np.array([[1.0, 3.0], [5.0, 11.0]]).reshape(1, 2, 2, 1)
    row_w = np.array([[1, 0], [0.5, 0.5], [0, 1], [0, 1]])   # 2 -> 4, by hand
    expect = row_w @ q[0, :, :, 0] @ row_w.T
    np.testing.assert_array_equal(oracle.resize_bilinear(q, 4, 4, False)[0, :, :, 0], expect)
    # 2x downscale 4 -> 2 takes samples 0 and 2 exactly (integer sources)
    r = rnd((1, 4, 4, 3), 33)
    np.testing.assert_array_equal(oracle.resize_bilinear(r, 2, 2, False), r[:, ::2, ::2, :])


def test_argmax_ties_lowest_index():
    x = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0], [-1.0, -2.0, -0.5, -0.5]]).reshape(1, 1, 3, 4)
    np.testing.assert_array_equal(oracle.argmax(x).ravel(), [1, 0, 2])


# ----------------------------------------------------------------------------
# network graphs: topology and shapes pinned by published counts
# ----------------------------------------------------------------------------
def count(graph):
    shapes = oracle.tensor_shapes(graph)
    macs = params = 0
    for i, op in enumerate(graph["ops"]):
        n, h, w, c = shapes[i]
        if op["op"] == "conv2d":
            cin = shapes[op["in"]][3]
            macs += h * w * c * op["kh"] * op["kw"] * cin
            params += op["w"].size + op["b"].size
        elif op["op"] == "depthwise":
            macs += h * w * c * op["kh"] * op["kw"]
            params += op["w"].size + op["b"].size
        elif op["op"] == "fc":
            macs += op["w"].size
            params += op["w"].size + op["b"].size
    return macs, params, shapes


def test_mobilenet_v1_counts():
    # MobileNet v1 1.0-224: 569 million multiply-adds, 4.2 million parameters
    macs, params, shapes = count(workloads.mobilenet_v1(1))
    assert round(macs / 1e6) == 569
    assert round(params / 1e5) == 42
    assert shapes[1] == (1, 112, 112, 32)
    assert shapes[-3] == (1, 1, 1, 1024) and shapes[-1] == (1, 1, 1, 1000)


def test_mobilenet_v2_counts():
    # MobileNet v2 1.0-224: about 300 million multiply-adds, 3.4 million parameters
    macs, params, shapes = count(workloads.mobilenet_v2(1))
    assert 295e6 < macs < 305e6
    assert 3.4e6 <= params < 3.55e6
    assert shapes[-4] == (1, 7, 7, 1280)


def test_deeplab_shapes():
    g = workloads.deeplab_v2_os16(1)
    shapes = oracle.tensor_shapes(g)
    names = {op["name"]: i for i, op in enumerate(g["ops"])}
    assert shapes[names["b17_project"]] == (1, 33, 33, 320)
    assert shapes[names["concat"]] == (1, 33, 33, 512)
    assert shapes[names["logits"]] == (1, 33, 33, 21)
    assert shapes[names["labels"]] == (1, 513, 513, 1)
    dils = [op["dil"][0] for op in g["ops"] if op["op"] == "depthwise"]
    assert dils[-4:] == [2, 2, 2, 2] and set(dils[:-4]) == {1}


def test_seeded_draws_are_fp16_values_and_he_scaled():
    g = workloads.mobilenet_v1(1)
    x = g["ops"][0]["data"]
    assert x.dtype == np.float32 and x.min() >= 0 and x.max() <= 1
    np.testing.assert_array_equal(x.astype(np.float16).astype(np.float32), x)
    w = g["ops"][-4]["w"]          # pw13: 1024 -> 1024
    assert abs(w.std() - math.sqrt(2 / 1024)) < 0.02 * math.sqrt(2 / 1024)
    g2 = workloads.mobilenet_v1(1)
    np.testing.assert_array_equal(g2["ops"][3]["w"], g["ops"][3]["w"])


def test_store_fp16_rounds_stored_tensors_only():
    g = workloads.NetBuilder(3)
    x = g.input(1, 6, 6, 8, -1, 1)
    c = g.conv(x, 16, 3, 1, act=workloads.ACT_NONE)
    p = g.gap(c)
    z = g.fc(p, 5)
    g.mark_output(z)
    d = g.graph("t")
    exact = oracle.run_graph(d)
    r16 = oracle.run_graph(d, store_fp16=True)
    np.testing.assert_array_equal(r16[c], exact[c].astype(np.float16).astype(np.float64))
    assert not np.array_equal(r16[c], exact[c])
    pooled = r16[c].mean(axis=(1, 2), keepdims=True)
    np.testing.assert_allclose(r16[p], pooled.astype(np.float16).astype(np.float64), rtol=0, atol=0)
    # logits are kept in fp32 by the engine: not rounded, computed from the rounded pool
    np.testing.assert_allclose(r16[z], oracle.fc(r16[p], d["ops"][z]["w"], d["ops"][z]["b"]), rtol=1e-15)


def test_bf16_storage_rounding_matches_library():
    # the oracle's bf16 storage emulation is round-to-nearest-even on the
    # float32 pattern; torch's bfloat16 conversion is an independent route
    torch = pytest.importorskip("torch")
    x = np.concatenate([rnd(4000, 77) * 10.0 ** np.arange(-3, 5).repeat(500),
                        np.array([1.0, 1.00390625, 1.01171875, -0.0, 3.3895314e38])])
    ref = torch.tensor(x.astype(np.float32)).to(torch.bfloat16).float().numpy().astype(np.float64)
    np.testing.assert_array_equal(oracle._round_bf16(x), ref)
    g = workloads.NetBuilder(seed=1)
    t = g.conv(g.input(1, 3, 3, 8, -1, 1), 8, 1)
    g.mark_output(t)
    out = oracle.run_graph(g.graph("b"), store_bf16=True)[t]
    np.testing.assert_array_equal(out, oracle._round_bf16(out))

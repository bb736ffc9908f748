"""Seeded synthetic workloads: network descriptions, weights and inputs.

This module is shared by the GPU engine's tests and benchmark and by the CPU
oracle.  It holds no arithmetic of the inference method itself: it only draws
seeded random numbers and lists the operators of each network with their
attributes (kernel size, stride, dilation, explicit four-sided padding, output
channels, activation).  Output shapes are *not* computed here; each side derives
them from the operator attributes on its own.

Network shapes follow the MobileNet family that the paper benchmarks
(Sec. 6, Tables 3-5).  Tensor layout of every array handed out is NHWC; weight
layouts are OHWI for full convolutions, C x KH x KW for depthwise and
COUT x CIN for fully-connected layers.

Random draws.  Every tensor index ``i`` of the op list (the input is index 0)
gets its own PCG64 stream ``default_rng(SeedSequence([seed, i]))``; weights are
drawn first, then the bias.  Weights are He-normal, N(0, 2 / fan_in), with
fan_in = KH*KW*CIN/groups; biases are N(0, 0.01^2).  Inputs and weights are
rounded to fp16 (round-to-nearest-even) and handed out as float32 arrays holding
those fp16 values, so both sides consume identical numbers; biases stay fp32.
"""
from __future__ import annotations

import numpy as np

ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2
DTYPE_FP16, DTYPE_FP32 = 0, 2     # element types of graph inputs


# ----------------------------------------------------------------------------
# seeded draws
# ----------------------------------------------------------------------------
def rng_for(seed: int, index: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(index)]))


def fp16_round(a: np.ndarray) -> np.ndarray:
    """Round to the nearest fp16 value (ties to even) and return float32."""
    return np.asarray(a, dtype=np.float64).astype(np.float16).astype(np.float32)


def he_normal(rng, shape, fan_in):
    return fp16_round(rng.standard_normal(size=shape) * np.sqrt(2.0 / fan_in))


def bias_normal(rng, n):
    return (rng.standard_normal(size=n) * 0.01).astype(np.float32)


def make_input(shape, lo, hi, seed=0):
    rng = rng_for(seed, 0)
    return fp16_round(rng.uniform(lo, hi, size=shape))


# ----------------------------------------------------------------------------
# padding conventions (attributes of a network description, not arithmetic of
# the engine: the engine and the oracle both take explicit four-sided pads)
# ----------------------------------------------------------------------------
def same_pads(size, k, s, d):
    """TensorFlow 'SAME' padding: output = ceil(size / s); extra pad at the end."""
    out = -(-size // s)
    total = max((out - 1) * s + (k - 1) * d + 1 - size, 0)
    return total // 2, total - total // 2, out


# ----------------------------------------------------------------------------
# graph builder
# ----------------------------------------------------------------------------
class NetBuilder:
    """Builds a list of op dicts.  Tensor ``i`` is the output of ``ops[i]``.

    Each builder tracks the spatial size of the tensors it creates only to pick
    SAME padding for the next op; the engine and the oracle recompute shapes
    independently from the explicit pads.
    """

    def __init__(self, seed=0):
        self.seed = seed
        self.ops: list[dict] = []
        self._hwc: list[tuple] = []
        self.outputs: list[int] = []

    def _push(self, op, hwc):
        self.ops.append(op)
        self._hwc.append(hwc)
        return len(self.ops) - 1

    def hwc(self, t):
        return self._hwc[t]

    def input(self, n, h, w, c, lo, hi, name="input", dtype=DTYPE_FP16):
        """A graph input of fp16-representable values, handed to the engine
        as fp16 (``dtype`` 0) or fp32 (2) NHWC."""
        x = make_input((n, h, w, c), lo, hi, self.seed)
        return self._push({"op": "input", "name": name, "shape": (n, h, w, c), "data": x,
                           "dtype": dtype}, (h, w, c))

    def conv(self, x, cout, k=1, s=1, d=1, act=ACT_RELU6, name=None, pads=None):
        h, w, cin = self._hwc[x]
        idx = len(self.ops)
        if pads is None:
            pt, pb, oh = same_pads(h, k, s, d)
            pl, pr, ow = same_pads(w, k, s, d)
        else:
            pt, pb, pl, pr = pads
            oh = (h + pt + pb - d * (k - 1) - 1) // s + 1
            ow = (w + pl + pr - d * (k - 1) - 1) // s + 1
        rng = rng_for(self.seed, idx)
        wt = he_normal(rng, (cout, k, k, cin), k * k * cin)
        b = bias_normal(rng, cout)
        op = {"op": "conv2d", "name": name or f"conv{idx}", "in": x, "kh": k, "kw": k,
              "stride": (s, s), "dil": (d, d), "pads": (pt, pb, pl, pr), "cout": cout,
              "act": act, "w": wt, "b": b}
        return self._push(op, (oh, ow, cout))

    def dw(self, x, k=3, s=1, d=1, act=ACT_RELU6, name=None, pads=None):
        h, w, c = self._hwc[x]
        idx = len(self.ops)
        if pads is None:
            pt, pb, oh = same_pads(h, k, s, d)
            pl, pr, ow = same_pads(w, k, s, d)
        else:
            pt, pb, pl, pr = pads
            oh = (h + pt + pb - d * (k - 1) - 1) // s + 1
            ow = (w + pl + pr - d * (k - 1) - 1) // s + 1
        rng = rng_for(self.seed, idx)
        wt = he_normal(rng, (c, k, k), k * k)
        b = bias_normal(rng, c)
        op = {"op": "depthwise", "name": name or f"dw{idx}", "in": x, "kh": k, "kw": k,
              "stride": (s, s), "dil": (d, d), "pads": (pt, pb, pl, pr), "act": act,
              "w": wt, "b": b}
        return self._push(op, (oh, ow, c))

    def add(self, a, b, act=ACT_NONE, name=None):
        return self._push({"op": "add", "name": name or f"add{len(self.ops)}", "a": a, "b": b,
                           "act": act}, self._hwc[a])

    def activation(self, x, act, name=None):
        return self._push({"op": "activation", "name": name or f"act{len(self.ops)}", "in": x,
                           "act": act}, self._hwc[x])

    def pad(self, x, pads, name=None):
        """Zero padding (top, bottom, left, right) of the spatial dimensions."""
        h, w, c = self._hwc[x]
        pt, pb, pl, pr = pads
        return self._push({"op": "pad", "name": name or f"pad{len(self.ops)}", "in": x,
                           "pads": tuple(pads)}, (h + pt + pb, w + pl + pr, c))

    def gap(self, x, name=None):
        _, _, c = self._hwc[x]
        return self._push({"op": "gap", "name": name or f"gap{len(self.ops)}", "in": x}, (1, 1, c))

    def fc(self, x, cout, name=None):
        _, _, cin = self._hwc[x]
        idx = len(self.ops)
        rng = rng_for(self.seed, idx)
        wt = he_normal(rng, (cout, cin), cin)
        b = bias_normal(rng, cout)
        return self._push({"op": "fc", "name": name or f"fc{idx}", "in": x, "cout": cout,
                           "w": wt, "b": b}, (1, 1, cout))

    def softmax(self, x, name=None):
        return self._push({"op": "softmax", "name": name or f"softmax{len(self.ops)}", "in": x},
                          self._hwc[x])

    def concat(self, xs, name=None):
        h, w, _ = self._hwc[xs[0]]
        c = sum(self._hwc[t][2] for t in xs)
        return self._push({"op": "concat", "name": name or f"concat{len(self.ops)}",
                           "ins": list(xs)}, (h, w, c))

    def resize(self, x, oh, ow, align_corners=True, name=None):
        c = self._hwc[x][2]
        return self._push({"op": "resize_bilinear", "name": name or f"resize{len(self.ops)}",
                           "in": x, "oh": oh, "ow": ow, "align_corners": int(align_corners)},
                          (oh, ow, c))

    def argmax(self, x, name=None):
        h, w, _ = self._hwc[x]
        return self._push({"op": "argmax", "name": name or f"argmax{len(self.ops)}", "in": x},
                          (h, w, 1))

    def mark_output(self, t):
        self.outputs.append(t)

    def graph(self, name):
        return {"name": name, "ops": self.ops, "outputs": list(self.outputs)}


# ----------------------------------------------------------------------------
# the five workloads
# ----------------------------------------------------------------------------
def dw_separable_block(batch=1, seed=0):
    """One MobileNet-v1 block: 1x56x56x128 fp16 input in U[-1,1], depthwise 3x3 s1
    pad 1 + bias + ReLU6, then pointwise 128->128 + bias + ReLU6."""
    g = NetBuilder(seed)
    x = g.input(batch, 56, 56, 128, -1.0, 1.0)
    d = g.dw(x, 3, 1, name="dw")
    p = g.conv(d, 128, 1, name="pw")
    g.mark_output(p)
    return g.graph(f"dw_block_56x56x128_b{batch}")


V1_BLOCKS = [(64, 1), (128, 2), (128, 1), (256, 2), (256, 1), (512, 2), (512, 1), (512, 1),
             (512, 1), (512, 1), (512, 1), (1024, 2), (1024, 1)]


def mobilenet_v1(batch=1, res=224, seed=0, logits_output=True):
    """MobileNet v1, width 1.0: stem conv 3x3 s2 -> 32, 13 depthwise-separable
    blocks, global average pool, FC 1024 -> 1000, softmax."""
    g = NetBuilder(seed)
    x = g.input(batch, res, res, 3, 0.0, 1.0)
    t = g.conv(x, 32, 3, 2, name="stem")
    for i, (c, s) in enumerate(V1_BLOCKS, 1):
        t = g.dw(t, 3, s, name=f"dw{i}")
        t = g.conv(t, c, 1, name=f"pw{i}")
    t = g.gap(t, name="pool")
    logits = g.fc(t, 1000, name="fc")
    prob = g.softmax(logits, name="softmax")
    if logits_output:
        g.mark_output(logits)
    g.mark_output(prob)
    return g.graph(f"mobilenet_v1_{res}_b{batch}")


# (expansion t, channels c, repeats n, first stride s)
V2_STAGES = [(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1),
             (6, 160, 3, 2), (6, 320, 1, 1)]


def _v2_backbone(g, x, os16=False):
    t = g.conv(x, 32, 3, 2, name="stem")
    cin = 32
    blk = 0
    for si, (e, c, n, s) in enumerate(V2_STAGES):
        for r in range(n):
            blk += 1
            stride = s if r == 0 else 1
            dil = 1
            if os16 and si >= 5:          # last two stages: no extra stride, dilation 2
                stride, dil = 1, 2
            inp = t
            if e != 1:
                t = g.conv(t, cin * e, 1, name=f"b{blk}_expand")
            t = g.dw(t, 3, stride, dil, name=f"b{blk}_dw")
            t = g.conv(t, c, 1, act=ACT_NONE, name=f"b{blk}_project")
            if stride == 1 and cin == c:
                t = g.add(t, inp, name=f"b{blk}_add")
            cin = c
    return t


def mobilenet_v2(batch=1, res=224, seed=0, logits_output=True):
    """MobileNet v2, width 1.0: stem, 17 inverted-residual blocks, 1x1 -> 1280
    (ReLU6), global average pool, FC 1280 -> 1000, softmax."""
    g = NetBuilder(seed)
    x = g.input(batch, res, res, 3, 0.0, 1.0)
    t = _v2_backbone(g, x)
    t = g.conv(t, 1280, 1, name="head_conv")
    t = g.gap(t, name="pool")
    logits = g.fc(t, 1000, name="fc")
    prob = g.softmax(logits, name="softmax")
    if logits_output:
        g.mark_output(logits)
    g.mark_output(prob)
    return g.graph(f"mobilenet_v2_{res}_b{batch}")


def deeplab_v2_os16(batch=1, res=513, classes=21, seed=0, logits_output=True):
    """Dense prediction: MobileNet-v2 backbone at output stride 16 (last two
    stages stride 1, dilation 2), a 1x1 -> 256 branch (ReLU) beside an image
    pooling branch (global pool, 1x1 -> 256, ReLU, bilinear back to the feature
    size), channel concat, 1x1 -> classes, bilinear x16 (align corners) to the
    input size and per-pixel argmax."""
    g = NetBuilder(seed)
    x = g.input(batch, res, res, 3, 0.0, 1.0)
    f = _v2_backbone(g, x, os16=True)
    fh, fw, _ = g.hwc(f)
    a0 = g.conv(f, 256, 1, act=ACT_RELU, name="aspp0")
    p = g.gap(f, name="image_pool")
    p = g.conv(p, 256, 1, act=ACT_RELU, name="image_pool_conv")
    p = g.resize(p, fh, fw, True, name="image_pool_up")
    cat = g.concat([a0, p], name="concat")
    logits = g.conv(cat, classes, 1, act=ACT_NONE, name="logits")
    up = g.resize(logits, res, res, True, name="upsample")
    lab = g.argmax(up, name="labels")
    if logits_output:
        g.mark_output(logits)
    g.mark_output(lab)
    return g.graph(f"deeplab_mnv2_os16_{res}_b{batch}")


WORKLOADS = {
    "dw_block": lambda batch=1, **kw: dw_separable_block(batch, **kw),
    "mobilenet_v1": lambda batch=1, **kw: mobilenet_v1(batch, **kw),
    "mobilenet_v2": lambda batch=1, **kw: mobilenet_v2(batch, **kw),
    "deeplab": lambda batch=1, **kw: deeplab_v2_os16(batch, **kw),
}


def bf16_round(a):
    """Nearest bf16 value (ties to even) of each element, as float32."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).reshape(np.shape(a))


def as_bf16_graph(graph):
    """The same network with its input data and weights rounded to bf16 values
    (biases stay fp32), so that a bf16-storage engine and the oracle consume
    identical numbers."""
    ops = []
    for op in graph["ops"]:
        op = dict(op)
        if op["op"] == "input":
            op["data"] = bf16_round(op["data"])
        if "w" in op:
            op["w"] = bf16_round(op["w"])
        ops.append(op)
    return {"name": graph["name"] + "_bf16", "ops": ops, "outputs": list(graph["outputs"])}


def subset_batch(graph, images):
    """The same network applied to a subset of the batch images (batch entries
    are independent, so a sampled check can run the oracle on them alone)."""
    ops = []
    for op in graph["ops"]:
        if op["op"] == "input":
            op = dict(op)
            op["data"] = op["data"][list(images)]
            op["shape"] = (len(images),) + tuple(op["shape"][1:])
        ops.append(op)
    return {"name": graph["name"] + "_subset", "ops": ops, "outputs": list(graph["outputs"])}

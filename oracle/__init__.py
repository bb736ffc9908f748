"""CPU oracle for the MobileNet-class forward pass and the intermediate-buffer
planner.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the engine.  It shares no code with the
HIP engine; the two meet only in the seeded workload descriptions.

``run_graph`` walks an op list in declaration order (which is a topological
order) and evaluates every tensor in float64 NHWC with the plain C loops of
``oracle.c``.  Shapes are derived here from the op attributes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c with gcc (-O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        D = ctypes.POINTER(ctypes.c_double)
        I = ctypes.c_int
        S = ctypes.c_size_t
        L.orc_conv2d.argtypes = [D, I, I, I, I, D, D, I, I, I, I, I, I, I, I, I, D, I, I]
        L.orc_depthwise.argtypes = [D, I, I, I, I, D, D, I, I, I, I, I, I, I, I, D, I, I]
        L.orc_activation.argtypes = [D, S, I]
        L.orc_add.argtypes = [D, D, D, S]
        L.orc_global_avgpool.argtypes = [D, I, I, I, I, D]
        L.orc_fc.argtypes = [D, I, I, D, D, I, D]
        L.orc_softmax.argtypes = [D, I, I, D]
        L.orc_concat2.argtypes = [D, I, D, I, S, D]
        L.orc_resize_bilinear.argtypes = [D, I, I, I, I, D, I, I, I]
        L.orc_argmax.argtypes = [D, S, I, ctypes.POINTER(ctypes.c_int)]
        L.orc_set_threads.argtypes = [I]
        L.orc_set_threads.restype = None
        L.orc_max_threads.argtypes = []
        L.orc_max_threads.restype = I
        for f in ("orc_conv2d", "orc_depthwise", "orc_activation", "orc_add", "orc_global_avgpool",
                  "orc_fc", "orc_softmax", "orc_concat2", "orc_resize_bilinear", "orc_argmax"):
            getattr(L, f).restype = None
        _lib = L
    return _lib


def set_threads(n: int) -> int:
    """Set the thread count of the oracle's OpenMP loops; returns the previous
    one.  Results do not depend on it (each output element is one sequential
    sum)."""
    prev = lib().orc_max_threads()
    lib().orc_set_threads(int(n))
    return prev


def _d(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------
# single operators (NHWC float64)
# ----------------------------------------------------------------------------
def conv_out_size(size, k, s, d, p0, p1):
    return (size + p0 + p1 - d * (k - 1) - 1) // s + 1


def conv2d(x, w, b, stride=(1, 1), dil=(1, 1), pads=(0, 0, 0, 0)):
    x = _f64(x); w = _f64(w)
    N, H, W, C = x.shape
    CO, KH, KW, CI = w.shape
    assert CI == C
    pt, pb, pl, pr = pads
    OH = conv_out_size(H, KH, stride[0], dil[0], pt, pb)
    OW = conv_out_size(W, KW, stride[1], dil[1], pl, pr)
    y = np.empty((N, OH, OW, CO), np.float64)
    bb = _f64(b) if b is not None else None
    lib().orc_conv2d(_d(x), N, H, W, C, _d(w), _d(bb) if bb is not None else None, CO, KH, KW,
                     stride[0], stride[1], dil[0], dil[1], pt, pl, _d(y), OH, OW)
    return y


def depthwise(x, w, b, stride=(1, 1), dil=(1, 1), pads=(0, 0, 0, 0)):
    x = _f64(x); w = _f64(w)
    N, H, W, C = x.shape
    CW, KH, KW = w.shape
    assert CW == C
    pt, pb, pl, pr = pads
    OH = conv_out_size(H, KH, stride[0], dil[0], pt, pb)
    OW = conv_out_size(W, KW, stride[1], dil[1], pl, pr)
    y = np.empty((N, OH, OW, C), np.float64)
    bb = _f64(b) if b is not None else None
    lib().orc_depthwise(_d(x), N, H, W, C, _d(w), _d(bb) if bb is not None else None, KH, KW,
                        stride[0], stride[1], dil[0], dil[1], pt, pl, _d(y), OH, OW)
    return y


def activation(x, act):
    y = np.array(x, dtype=np.float64, copy=True, order="C")
    lib().orc_activation(_d(y), y.size, int(act))
    return y


def zero_pad(x, pads):
    """Spatial zero padding (Sec. 3.1, PAD): the input is placed at row pt,
    column pl of an all-zero (n, h + pt + pb, w + pl + pr, c) tensor."""
    x = _f64(x)
    pt, pb, pl, pr = pads
    n, h, w, c = x.shape
    y = np.zeros((n, h + pt + pb, w + pl + pr, c))
    for yy in range(h):
        for xx in range(w):
            y[:, pt + yy, pl + xx, :] = x[:, yy, xx, :]
    return y


def add(a, b):
    a = _f64(a); b = _f64(b)
    assert a.shape == b.shape
    y = np.empty_like(a)
    lib().orc_add(_d(a), _d(b), _d(y), a.size)
    return y


def global_avgpool(x):
    x = _f64(x)
    N, H, W, C = x.shape
    y = np.empty((N, 1, 1, C), np.float64)
    lib().orc_global_avgpool(_d(x), N, H, W, C, _d(y))
    return y


def fc(x, w, b):
    x = _f64(x); w = _f64(w)
    N = x.shape[0]
    CIN = int(np.prod(x.shape[1:]))
    COUT = w.shape[0]
    assert w.shape[1] == CIN
    y = np.empty((N, 1, 1, COUT), np.float64)
    bb = _f64(b) if b is not None else None
    lib().orc_fc(_d(x), N, CIN, _d(w), _d(bb) if bb is not None else None, COUT, _d(y))
    return y


def softmax(z):
    z = _f64(z)
    cols = z.shape[-1]
    y = np.empty_like(z)
    lib().orc_softmax(_d(z), z.size // cols, cols, _d(y))
    return y


def concat(xs):
    y = _f64(xs[0])
    for b in xs[1:]:
        b = _f64(b)
        assert b.shape[:3] == y.shape[:3]
        out = np.empty(y.shape[:3] + (y.shape[3] + b.shape[3],), np.float64)
        pixels = int(np.prod(y.shape[:3]))
        lib().orc_concat2(_d(y), y.shape[3], _d(b), b.shape[3], pixels, _d(out))
        y = out
    return y


def resize_bilinear(x, oh, ow, align_corners=True):
    x = _f64(x)
    N, H, W, C = x.shape
    y = np.empty((N, oh, ow, C), np.float64)
    lib().orc_resize_bilinear(_d(x), N, H, W, C, _d(y), oh, ow, int(align_corners))
    return y


def argmax(x):
    x = _f64(x)
    C = x.shape[-1]
    y = np.empty(x.shape[:-1] + (1,), np.int32)
    lib().orc_argmax(_d(x), x.size // C, C, y.ctypes.data_as(ctypes.POINTER(ctypes.c_int)))
    return y


# ----------------------------------------------------------------------------
# graphs
# ----------------------------------------------------------------------------
def tensor_shapes(graph):
    """NHWC shape of every tensor, derived from the op attributes."""
    shapes = []
    for op in graph["ops"]:
        k = op["op"]
        if k == "input":
            shapes.append(tuple(op["shape"]))
        elif k in ("conv2d", "depthwise"):
            n, h, w, c = shapes[op["in"]]
            pt, pb, pl, pr = op["pads"]
            oh = conv_out_size(h, op["kh"], op["stride"][0], op["dil"][0], pt, pb)
            ow = conv_out_size(w, op["kw"], op["stride"][1], op["dil"][1], pl, pr)
            shapes.append((n, oh, ow, op["cout"] if k == "conv2d" else c))
        elif k in ("add",):
            shapes.append(shapes[op["a"]])
        elif k in ("activation", "softmax"):
            shapes.append(shapes[op["in"]])
        elif k == "pad":
            n, h, w, c = shapes[op["in"]]
            pt, pb, pl, pr = op["pads"]
            shapes.append((n, h + pt + pb, w + pl + pr, c))
        elif k == "gap":
            n, h, w, c = shapes[op["in"]]
            shapes.append((n, 1, 1, c))
        elif k == "fc":
            shapes.append((shapes[op["in"]][0], 1, 1, op["cout"]))
        elif k == "concat":
            s0 = shapes[op["ins"][0]]
            shapes.append(s0[:3] + (sum(shapes[t][3] for t in op["ins"]),))
        elif k == "resize_bilinear":
            n, h, w, c = shapes[op["in"]]
            shapes.append((n, op["oh"], op["ow"], c))
        elif k == "argmax":
            n, h, w, c = shapes[op["in"]]
            shapes.append((n, h, w, 1))
        else:
            raise ValueError(f"unknown op {k}")
    return shapes


def op_inputs(op):
    k = op["op"]
    if k == "input":
        return []
    if k == "add":
        return [op["a"], op["b"]]
    if k == "concat":
        return list(op["ins"])
    return [op["in"]]


# ops whose output the paper's engine keeps in fp16 storage (everything but
# the fp32 logits / probabilities and the integer labels)
FP16_STORED = {"conv2d", "depthwise", "add", "activation", "gap", "concat", "resize_bilinear", "pad"}


def eval_op(op, operands):
    """Evaluate one op on its operand arrays (float64 NHWC), in the order the
    operands appear in ``op_inputs(op)``."""
    k = op["op"]
    if k == "input":
        return _f64(op["data"])
    if k == "conv2d":
        return activation(conv2d(operands[0], op["w"], op["b"], op["stride"], op["dil"], op["pads"]),
                          op["act"])
    if k == "depthwise":
        return activation(depthwise(operands[0], op["w"], op["b"], op["stride"], op["dil"],
                                    op["pads"]), op["act"])
    if k == "add":
        return activation(add(operands[0], operands[1]), op["act"])
    if k == "activation":
        return activation(operands[0], op["act"])
    if k == "pad":
        return zero_pad(operands[0], op["pads"])
    if k == "gap":
        return global_avgpool(operands[0])
    if k == "fc":
        return fc(operands[0], op["w"], op["b"])
    if k == "softmax":
        return softmax(operands[0])
    if k == "concat":
        return concat(operands)
    if k == "resize_bilinear":
        return resize_bilinear(operands[0], op["oh"], op["ow"], op["align_corners"])
    if k == "argmax":
        return argmax(operands[0])
    raise ValueError(f"unknown op {k}")


def _round_bf16(y):
    """Nearest bf16 value (ties to even) of each element, via the float32 bit
    pattern: bf16 keeps the upper 16 bits of a float32."""
    u = np.asarray(y, dtype=np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64).reshape(np.shape(y))


def run_graph(graph, keep=None, store_fp16=False, store_bf16=False):
    """Evaluate every tensor of ``graph``; returns {tensor id: float64 NHWC array}
    (argmax outputs are int32).  ``keep`` limits which tensors are returned;
    others are dropped as soon as their last consumer has run.

    ``store_fp16`` rounds each tensor that the paper's engine stores in fp16
    (Table 1 frames the GPU side as FP16) to the nearest fp16 value after its
    op, everything else staying exact: it measures how much a network amplifies
    the rounding that fp16 storage alone introduces.  ``store_bf16`` does the
    same for bf16 storage."""
    ops = graph["ops"]
    last_use = {}
    for i, op in enumerate(ops):
        for t in op_inputs(op):
            last_use[t] = i
    want = set(range(len(ops))) if keep is None else set(keep)
    vals: dict[int, np.ndarray] = {}
    for i, op in enumerate(ops):
        y = eval_op(op, [vals[t] for t in op_inputs(op)])
        if store_fp16 and op["op"] in FP16_STORED:
            y = y.astype(np.float16).astype(np.float64)
        if store_bf16 and op["op"] in FP16_STORED:
            y = _round_bf16(y)
        vals[i] = y
        for t in op_inputs(op):
            if last_use.get(t) == i and t not in want:
                vals.pop(t, None)
    return {t: v for t, v in vals.items() if t in want}

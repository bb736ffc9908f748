"""ctypes binding of libmgi.so.  Every C entry point of include/mgi.h is
exposed under the same name; a non-zero status raises MgiError carrying
mgi_last_error().  This module only marshals arguments: all computation runs
in the library.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# the engine library; MGI_LIB_PATH selects another build of it (e.g. the
# sanitizer build of build_lib --sanitize)
LIB_PATH = os.environ.get("MGI_LIB_PATH") or os.path.join(_HERE, "libmgi.so")

MGI_OK = 0
STATUS = {0: "MGI_OK", 1: "MGI_ERR_INVALID_ARG", 2: "MGI_ERR_SHAPE", 3: "MGI_ERR_UNSUPPORTED",
          4: "MGI_ERR_STATE", 5: "MGI_ERR_WORKSPACE", 6: "MGI_ERR_HIP", 7: "MGI_ERR_OOM_HOST",
          8: "MGI_ERR_INTERNAL"}
ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2
DTYPE_FP16, DTYPE_BF16, DTYPE_FP32, DTYPE_INT32 = 0, 1, 2, 3
PLANNER_NAIVE, PLANNER_GREEDY, PLANNER_MCFP = 0, 1, 2


class MgiError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("kh", "kw", "stride_h", "stride_w", "dil_h", "dil_w",
                                           "pad_t", "pad_b", "pad_l", "pad_r", "cout", "act")]


class Options(ctypes.Structure):
    _fields_ = [("planner", ctypes.c_int), ("fuse", ctypes.c_int),
                ("materialize_all", ctypes.c_int), ("dtype", ctypes.c_int),
                ("fuse_dwpw", ctypes.c_int),
                ("fuse_pwdw", ctypes.c_int),
                ("fuse_stemdw", ctypes.c_int),
                ("fuse_pool", ctypes.c_int),
                ("fuse_softmax", ctypes.c_int),
                ("fuse_irb", ctypes.c_int)]


_lib = None
P = ctypes.c_void_p
I = ctypes.c_int
IP = ctypes.POINTER(ctypes.c_int)
SP = ctypes.POINTER(ctypes.c_size_t)
FP = ctypes.POINTER(ctypes.c_float)

_SIGS = {
    "mgi_status_str": ([I], ctypes.c_char_p),
    "mgi_last_error": ([], ctypes.c_char_p),
    "mgi_graph_create": ([ctypes.POINTER(P)], I),
    "mgi_graph_destroy": ([P], I),
    "mgi_graph_add_input": ([P, I, I, I, I, I, IP], I),
    "mgi_graph_add_conv2d": ([P, I, ctypes.POINTER(ConvDesc), FP, FP, IP], I),
    "mgi_graph_add_depthwise": ([P, I, ctypes.POINTER(ConvDesc), FP, FP, IP], I),
    "mgi_graph_add_add": ([P, I, I, I, IP], I),
    "mgi_graph_add_activation": ([P, I, I, IP], I),
    "mgi_graph_add_pad": ([P, I, I, I, I, I, IP], I),
    "mgi_graph_add_global_avgpool": ([P, I, IP], I),
    "mgi_graph_add_fc": ([P, I, I, FP, FP, IP], I),
    "mgi_graph_add_softmax": ([P, I, IP], I),
    "mgi_graph_add_concat": ([P, IP, I, IP], I),
    "mgi_graph_add_resize_bilinear": ([P, I, I, I, I, IP], I),
    "mgi_graph_add_argmax": ([P, I, IP], I),
    "mgi_graph_mark_output": ([P, I], I),
    "mgi_options_default": ([ctypes.POINTER(Options)], None),
    "mgi_graph_finalize": ([P, ctypes.POINTER(Options), ctypes.POINTER(P)], I),
    "mgi_plan_destroy": ([P], I),
    "mgi_plan_workspace_bytes": ([P, SP], I),
    "mgi_plan_weight_bytes": ([P, SP], I),
    "mgi_plan_memory_report": ([P, SP, SP, IP], I),
    "mgi_plan_num_io": ([P, IP, IP], I),
    "mgi_plan_io_info": ([P, I, I, IP, IP, IP, IP, IP, SP], I),
    "mgi_plan_bind": ([P, P, P, P], I),
    "mgi_plan_run": ([P, ctypes.POINTER(P), ctypes.POINTER(P), P], I),
    "mgi_plan_run_noalloc": ([P, ctypes.POINTER(P), ctypes.POINTER(P), P], I),
    "mgi_plan_read_node_raw": ([P, I, P, SP, P], I),
    "mgi_plan_run_timed": ([P, ctypes.POINTER(P), ctypes.POINTER(P), P, ctypes.POINTER(P),
                            ctypes.POINTER(P)], I),
    "mgi_plan_capture": ([P, ctypes.POINTER(P), ctypes.POINTER(P)], I),
    "mgi_plan_autotune": ([P, ctypes.POINTER(P), ctypes.POINTER(P), P, I], I),
    "mgi_plan_node_config": ([P, I, IP, IP, ctypes.POINTER(ctypes.c_char_p)], I),
    "mgi_plan_set_node_config": ([P, I, I], I),
    "mgi_plan_replay": ([P, P], I),
    "mgi_plan_node_count": ([P, IP], I),
    "mgi_plan_node_info": ([P, I, ctypes.POINTER(ctypes.c_char_p), IP, IP, IP, IP, IP, IP], I),
    "mgi_plan_read_node": ([P, I, P, P], I),
    "mgi_planner_assign": ([I, I, SP, IP, IP, IP, SP, IP], I),
}


def lib():
    """Load libmgi.so (built by paper_1907_01989_amd.build_lib).  There is no
    fallback: a missing library is an error."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_1907_01989_amd.build_lib`")
        # One HIP runtime per process: PyTorch-ROCm carries its own copy of
        # the HIP runtime, and the device buffers and streams handed to the
        # library come from it.  Loading the library first would bind it to
        # the system copy and give the process two runtimes, in which the
        # library's calls find no device.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(status):
    if status != MGI_OK:
        raise MgiError(status, lib().mgi_last_error().decode())


def _fptr(a):
    return a.ctypes.data_as(FP) if a is not None else None


def _f32(a):
    import numpy as np
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# same-named wrappers
# --------------------------------------------------------------------------
def mgi_status_str(s):
    return lib().mgi_status_str(s).decode()


def mgi_last_error():
    return lib().mgi_last_error().decode()


def mgi_graph_create():
    g = P()
    _check(lib().mgi_graph_create(ctypes.byref(g)))
    return g


def mgi_graph_destroy(g):
    _check(lib().mgi_graph_destroy(g))


def _out(fn, *args):
    o = ctypes.c_int(-1)
    _check(fn(*args, ctypes.byref(o)))
    return o.value


def mgi_graph_add_input(g, n, h, w, c, dtype=DTYPE_FP32):
    return _out(lib().mgi_graph_add_input, g, n, h, w, c, dtype)


def conv_desc(kh, kw, stride=(1, 1), dil=(1, 1), pads=(0, 0, 0, 0), cout=0, act=ACT_NONE):
    return ConvDesc(kh, kw, stride[0], stride[1], dil[0], dil[1], pads[0], pads[1], pads[2],
                    pads[3], cout, act)


def mgi_graph_add_conv2d(g, x, desc, w, b=None):
    w, b = _f32(w), _f32(b)
    return _out(lib().mgi_graph_add_conv2d, g, x, ctypes.byref(desc), _fptr(w), _fptr(b))


def mgi_graph_add_depthwise(g, x, desc, w, b=None):
    w, b = _f32(w), _f32(b)
    return _out(lib().mgi_graph_add_depthwise, g, x, ctypes.byref(desc), _fptr(w), _fptr(b))


def mgi_graph_add_add(g, a, b, act=ACT_NONE):
    return _out(lib().mgi_graph_add_add, g, a, b, act)


def mgi_graph_add_activation(g, x, act):
    return _out(lib().mgi_graph_add_activation, g, x, act)


def mgi_graph_add_pad(g, x, pt, pb, pl, pr):
    return _out(lib().mgi_graph_add_pad, g, x, pt, pb, pl, pr)


def mgi_graph_add_global_avgpool(g, x):
    return _out(lib().mgi_graph_add_global_avgpool, g, x)


def mgi_graph_add_fc(g, x, cout, w, b=None):
    w, b = _f32(w), _f32(b)
    return _out(lib().mgi_graph_add_fc, g, x, cout, _fptr(w), _fptr(b))


def mgi_graph_add_softmax(g, x):
    return _out(lib().mgi_graph_add_softmax, g, x)


def mgi_graph_add_concat(g, ins):
    arr = (ctypes.c_int * len(ins))(*ins)
    return _out(lib().mgi_graph_add_concat, g, arr, len(ins))


def mgi_graph_add_resize_bilinear(g, x, oh, ow, align_corners=1):
    return _out(lib().mgi_graph_add_resize_bilinear, g, x, oh, ow, int(align_corners))


def mgi_graph_add_argmax(g, x):
    return _out(lib().mgi_graph_add_argmax, g, x)


def mgi_graph_mark_output(g, t):
    _check(lib().mgi_graph_mark_output(g, t))


def mgi_options_default():
    o = Options()
    lib().mgi_options_default(ctypes.byref(o))
    return o


def mgi_graph_finalize(g, opts=None):
    opts = opts or mgi_options_default()
    p = P()
    _check(lib().mgi_graph_finalize(g, ctypes.byref(opts), ctypes.byref(p)))
    return p


def mgi_plan_destroy(p):
    _check(lib().mgi_plan_destroy(p))


def _size(fn, p):
    v = ctypes.c_size_t(0)
    _check(fn(p, ctypes.byref(v)))
    return v.value


def mgi_plan_workspace_bytes(p):
    return _size(lib().mgi_plan_workspace_bytes, p)


def mgi_plan_weight_bytes(p):
    return _size(lib().mgi_plan_weight_bytes, p)


def mgi_plan_memory_report(p):
    a, b, k = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_int()
    _check(lib().mgi_plan_memory_report(p, ctypes.byref(a), ctypes.byref(b), ctypes.byref(k)))
    return a.value, b.value, k.value


def mgi_plan_num_io(p):
    a, b = ctypes.c_int(), ctypes.c_int()
    _check(lib().mgi_plan_num_io(p, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def mgi_plan_io_info(p, is_output, index):
    v = [ctypes.c_int() for _ in range(5)]
    nb = ctypes.c_size_t()
    _check(lib().mgi_plan_io_info(p, int(is_output), index, *[ctypes.byref(x) for x in v],
                                  ctypes.byref(nb)))
    n, h, w, c, dt = (x.value for x in v)
    return (n, h, w, c), dt, nb.value


def mgi_plan_bind(p, dev_ws, dev_w, stream=None):
    _check(lib().mgi_plan_bind(p, P(dev_ws), P(dev_w), P(stream or 0)))


def _io_arrays(p, in_ptrs, out_ptrs):
    """ctypes pointer arrays for a plan's inputs and outputs.  The C calls take
    arrays with no length, so the counts are checked against the plan here."""
    n_in, n_out = mgi_plan_num_io(p)
    if len(in_ptrs) != n_in or len(out_ptrs) != n_out:
        raise ValueError(f"plan takes {n_in} inputs and {n_out} outputs, "
                         f"got {len(in_ptrs)} and {len(out_ptrs)}")
    ins = (P * max(1, n_in))(*in_ptrs)
    outs = (P * max(1, n_out))(*out_ptrs)
    return ins, outs


def mgi_plan_run(p, in_ptrs, out_ptrs, stream=None):
    ins, outs = _io_arrays(p, in_ptrs, out_ptrs)
    _check(lib().mgi_plan_run(p, ins, outs, P(stream or 0)))


def mgi_plan_run_noalloc(p, in_ptrs, out_ptrs, stream=None):
    ins, outs = _io_arrays(p, in_ptrs, out_ptrs)
    _check(lib().mgi_plan_run_noalloc(p, ins, outs, P(stream or 0)))


NOALLOC_WORKSPACE_BYTES = 64 << 20


def mgi_plan_run_timed(p, in_ptrs, out_ptrs, start_events, stop_events, stream=None):
    ins, outs = _io_arrays(p, in_ptrs, out_ptrs)
    n = mgi_plan_node_count(p)
    if len(start_events) != n or len(stop_events) != n:
        raise ValueError(f"plan has {n} nodes: one start and one stop event slot each")
    ev0 = (P * max(1, n))(*[e or None for e in start_events])
    ev1 = (P * max(1, n))(*[e or None for e in stop_events])
    _check(lib().mgi_plan_run_timed(p, ins, outs, P(stream or 0), ev0, ev1))


def mgi_plan_capture(p, in_ptrs, out_ptrs):
    ins, outs = _io_arrays(p, in_ptrs, out_ptrs)
    _check(lib().mgi_plan_capture(p, ins, outs))


def mgi_plan_autotune(p, in_ptrs, out_ptrs, stream=None, reps=5):
    ins, outs = _io_arrays(p, in_ptrs, out_ptrs)
    _check(lib().mgi_plan_autotune(p, ins, outs, P(stream or 0), reps))


def mgi_plan_read_node_raw(p, i, dev_dst=None, stream=None):
    """Bytes of node i's stored sliced output; copies them to dev_dst if given."""
    nb = ctypes.c_size_t()
    _check(lib().mgi_plan_read_node_raw(p, i, P(dev_dst or 0), ctypes.byref(nb), P(stream or 0)))
    return nb.value


def mgi_plan_node_config(p, i):
    cfg, n = ctypes.c_int(), ctypes.c_int()
    name = ctypes.c_char_p()
    _check(lib().mgi_plan_node_config(p, i, ctypes.byref(cfg), ctypes.byref(n), ctypes.byref(name)))
    return cfg.value, n.value, name.value.decode()


def mgi_plan_set_node_config(p, i, config):
    _check(lib().mgi_plan_set_node_config(p, i, config))


def mgi_plan_replay(p, stream=None):
    _check(lib().mgi_plan_replay(p, P(stream or 0)))


def mgi_plan_node_count(p):
    return _out(lib().mgi_plan_node_count, p)


def mgi_plan_node_info(p, i):
    kind = ctypes.c_char_p()
    v = [ctypes.c_int() for _ in range(6)]
    _check(lib().mgi_plan_node_info(p, i, ctypes.byref(kind), *[ctypes.byref(x) for x in v]))
    t, n, h, w, c, nf = (x.value for x in v)
    return {"kind": kind.value.decode(), "tensor": t, "shape": (n, h, w, c), "n_fused": nf}


def mgi_plan_read_node(p, i, dev_dst, stream=None):
    _check(lib().mgi_plan_read_node(p, i, P(dev_dst), P(stream or 0)))


def mgi_planner_assign(planner, sizes, first, last):
    n = len(sizes)
    S = (ctypes.c_size_t * max(1, n))(*sizes)
    F = (ctypes.c_int * max(1, n))(*first)
    L = (ctypes.c_int * max(1, n))(*last)
    obj = (ctypes.c_int * max(1, n))()
    osz = (ctypes.c_size_t * max(1, n))()
    k = ctypes.c_int()
    _check(lib().mgi_planner_assign(planner, n, S, F, L, obj, osz, ctypes.byref(k)))
    return list(obj[:n]), list(osz[:k.value])

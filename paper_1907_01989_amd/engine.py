"""Thin Python front end: builds an mgi graph from a network description
(a list of operator dicts, see the workload generators), finalises it, and
binds it to torch-allocated device memory.  torch supplies device memory and
streams only; every step of the forward pass runs in libmgi's kernels.
"""
from __future__ import annotations

import numpy as np

from . import _binding as B


def _stream_handle(stream):
    """A torch stream, a raw hipStream_t (int), or None for torch's current stream."""
    if isinstance(stream, int):
        return stream
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def build_graph(desc):
    """Create an mgi graph from ``desc`` (dict with "ops" and "outputs").
    Returns the graph handle; tensor ids equal op indices."""
    g = B.mgi_graph_create()
    try:
        for i, op in enumerate(desc["ops"]):
            k = op["op"]
            if k == "input":
                n, h, w, c = op["shape"]
                t = B.mgi_graph_add_input(g, n, h, w, c, op.get("dtype", B.DTYPE_FP32))
            elif k == "conv2d":
                d = B.conv_desc(op["kh"], op["kw"], op["stride"], op["dil"], op["pads"],
                                op["cout"], op["act"])
                t = B.mgi_graph_add_conv2d(g, op["in"], d, op["w"], op["b"])
            elif k == "depthwise":
                d = B.conv_desc(op["kh"], op["kw"], op["stride"], op["dil"], op["pads"], 0,
                                op["act"])
                t = B.mgi_graph_add_depthwise(g, op["in"], d, op["w"], op["b"])
            elif k == "add":
                t = B.mgi_graph_add_add(g, op["a"], op["b"], op["act"])
            elif k == "activation":
                t = B.mgi_graph_add_activation(g, op["in"], op["act"])
            elif k == "pad":
                t = B.mgi_graph_add_pad(g, op["in"], *op["pads"])
            elif k == "gap":
                t = B.mgi_graph_add_global_avgpool(g, op["in"])
            elif k == "fc":
                t = B.mgi_graph_add_fc(g, op["in"], op["cout"], op["w"], op["b"])
            elif k == "softmax":
                t = B.mgi_graph_add_softmax(g, op["in"])
            elif k == "concat":
                t = B.mgi_graph_add_concat(g, op["ins"])
            elif k == "resize_bilinear":
                t = B.mgi_graph_add_resize_bilinear(g, op["in"], op["oh"], op["ow"],
                                                    op["align_corners"])
            elif k == "argmax":
                t = B.mgi_graph_add_argmax(g, op["in"])
            else:
                raise ValueError(f"unknown op {k}")
            if t != i:
                raise RuntimeError(f"tensor id {t} != op index {i}")
        for t in desc["outputs"]:
            B.mgi_graph_mark_output(g, t)
    except Exception:
        B.mgi_graph_destroy(g)
        raise
    return g


def options(planner=B.PLANNER_GREEDY, fuse=True, materialize_all=False, fuse_dwpw=False,
            dtype=B.DTYPE_FP16, fuse_pwdw=True, fuse_stemdw=True, fuse_pool=True, fuse_softmax=True,
            fuse_irb=False):
    o = B.mgi_options_default()
    o.dtype = dtype
    o.planner = planner
    o.fuse = int(fuse)
    o.materialize_all = int(materialize_all)
    o.fuse_dwpw = int(fuse_dwpw)
    o.fuse_pwdw = int(fuse_pwdw)     # False/True or 2 (fuse regardless of workgroup count)
    o.fuse_stemdw = int(fuse_stemdw)  # likewise
    o.fuse_pool = int(fuse_pool)      # likewise
    o.fuse_softmax = int(fuse_softmax)
    o.fuse_irb = int(fuse_irb)        # False/True or 2
    return o


class Plan:
    """A finalised, device-bound network."""

    def __init__(self, desc, planner=B.PLANNER_GREEDY, fuse=True, materialize_all=False,
                 device="cuda:0", bind=True, fuse_dwpw=False, dtype=B.DTYPE_FP16, fuse_pwdw=True,
                 fuse_stemdw=True, fuse_pool=True, fuse_softmax=True, fuse_irb=False):
        self.desc = desc
        g = build_graph(desc)
        try:
            self.handle = B.mgi_graph_finalize(
                g, options(planner, fuse, materialize_all, fuse_dwpw, dtype, fuse_pwdw, fuse_stemdw,
                           fuse_pool, fuse_softmax, fuse_irb))
        finally:
            B.mgi_graph_destroy(g)
        self.device = device
        self.n_inputs, self.n_outputs = B.mgi_plan_num_io(self.handle)
        self.inputs_info = [B.mgi_plan_io_info(self.handle, 0, i) for i in range(self.n_inputs)]
        self.outputs_info = [B.mgi_plan_io_info(self.handle, 1, i) for i in range(self.n_outputs)]
        self.workspace_bytes = B.mgi_plan_workspace_bytes(self.handle)
        self.weight_bytes = B.mgi_plan_weight_bytes(self.handle)
        self.bound = False
        if bind:
            self.bind()

    # ---------------------------------------------------------------- device
    def bind(self, stream=None):
        import torch
        self.ws = torch.empty(self.workspace_bytes + 256, dtype=torch.uint8, device=self.device)
        self.wts = torch.empty(self.weight_bytes + 256, dtype=torch.uint8, device=self.device)
        self._ws_ptr = (self.ws.data_ptr() + 255) & ~255
        self._w_ptr = (self.wts.data_ptr() + 255) & ~255
        B.mgi_plan_bind(self.handle, self._ws_ptr, self._w_ptr, _stream_handle(stream))
        self.bound = True

    def alloc_outputs(self):
        import torch
        outs = []
        for shape, dt, _ in self.outputs_info:
            n, h, w, c = shape
            tdt = torch.int32 if dt == B.DTYPE_INT32 else torch.float32
            if dt == B.DTYPE_INT32:
                outs.append(torch.empty((n, h, w), dtype=tdt, device=self.device))
            elif h == 1 and w == 1:
                outs.append(torch.empty((n, c), dtype=tdt, device=self.device))
            else:
                outs.append(torch.empty((n, h, w, c), dtype=tdt, device=self.device))
        return outs

    def check_io(self, inputs, outputs):
        """Raise ValueError unless ``inputs`` and ``outputs`` match the plan:
        as many tensors as it has graph inputs and outputs, each a contiguous
        tensor on this plan's device with the element type and byte size the
        plan reads or writes.  The library receives raw device pointers, so a
        tensor that fails any of these would make its kernels read or write
        outside the buffer."""
        import torch
        inputs, outputs = list(inputs), list(outputs)
        if len(inputs) != self.n_inputs or len(outputs) != self.n_outputs:
            raise ValueError(f"plan takes {self.n_inputs} inputs and {self.n_outputs} outputs, "
                             f"got {len(inputs)} and {len(outputs)}")
        dev = torch.device(self.device)
        in_types = {B.DTYPE_FP16: torch.float16, B.DTYPE_FP32: torch.float32}
        out_types = {B.DTYPE_INT32: torch.int32, B.DTYPE_FP32: torch.float32}
        for role, ts, info, types in (("input", inputs, self.inputs_info, in_types),
                                      ("output", outputs, self.outputs_info, out_types)):
            for i, (x, (shape, dt, nbytes)) in enumerate(zip(ts, info)):
                if not isinstance(x, torch.Tensor):
                    raise ValueError(f"{role} {i}: expected a torch tensor, got {type(x).__name__}")
                if not x.is_cuda or x.device.index != (dev.index if dev.index is not None else
                                                       torch.cuda.current_device()):
                    raise ValueError(f"{role} {i}: tensor on {x.device}, plan on {self.device}")
                if x.dtype != types.get(dt):
                    raise ValueError(f"{role} {i}: dtype {x.dtype}, plan expects {types.get(dt)}")
                if not x.is_contiguous() or x.numel() * x.element_size() != nbytes:
                    raise ValueError(f"{role} {i}: must be a contiguous tensor of {nbytes} bytes "
                                     f"(NHWC {shape}), got {tuple(x.shape)}")

    def run(self, inputs, outputs=None, stream=None):
        """Enqueue one forward pass; returns the output tensors (not synchronised)."""
        if not self.bound:
            raise RuntimeError("plan is not bound to device memory (call bind())")
        if outputs is None:
            outputs = self.alloc_outputs()
        self.check_io(inputs, outputs)
        B.mgi_plan_run(self.handle, [x.data_ptr() for x in inputs],
                       [y.data_ptr() for y in outputs], _stream_handle(stream))
        return outputs

    def autotune(self, inputs, outputs=None, reps=5, stream=None):
        """Time every candidate kernel configuration per node on these buffers
        and keep the fastest (see mgi_plan_autotune); synchronises."""
        if outputs is None:
            outputs = self.alloc_outputs()
        self.check_io(inputs, outputs)
        B.mgi_plan_autotune(self.handle, [x.data_ptr() for x in inputs], [y.data_ptr() for y in outputs],
                            _stream_handle(stream), reps)
        self._graph_io = None

    def node_configs(self):
        return [B.mgi_plan_node_config(self.handle, i) for i in range(B.mgi_plan_node_count(self.handle))]

    def capture(self, inputs, outputs=None):
        """Record one run over these tensors as a HIP graph (see replay); the
        tensors stay referenced by the plan so that their memory outlives it."""
        if outputs is None:
            outputs = self.alloc_outputs()
        self.check_io(inputs, outputs)
        B.mgi_plan_capture(self.handle, [x.data_ptr() for x in inputs], [y.data_ptr() for y in outputs])
        self._graph_io = (list(inputs), list(outputs))
        return outputs

    def replay(self, stream=None):
        """Enqueue the captured run; returns its output tensors (not synchronised)."""
        B.mgi_plan_replay(self.handle, _stream_handle(stream))
        return self._graph_io[1]

    def input_tensors(self):
        """Device copies of the description's input arrays."""
        import torch
        xs = []
        for op in self.desc["ops"]:
            if op["op"] == "input":
                dt = torch.float16 if op.get("dtype", B.DTYPE_FP32) == B.DTYPE_FP16 else torch.float32
                xs.append(torch.from_numpy(np.ascontiguousarray(op["data"])).to(self.device, dt))
        return xs

    # --------------------------------------------------------- introspection
    def nodes(self):
        return [B.mgi_plan_node_info(self.handle, i) for i in range(B.mgi_plan_node_count(self.handle))]

    def read_node(self, i, stream=None):
        import torch
        info = B.mgi_plan_node_info(self.handle, i)
        n, h, w, c = info["shape"]
        if info["kind"] in ("argmax", "resize_argmax"):
            dst = torch.empty((n, h, w, 1), dtype=torch.int32, device=self.device)
        else:
            dst = torch.empty((n, h, w, c), dtype=torch.float32, device=self.device)
        B.mgi_plan_read_node(self.handle, i, dst.data_ptr(), _stream_handle(stream))
        return info, dst

    def memory_report(self):
        return B.mgi_plan_memory_report(self.handle)

    def close(self):
        if getattr(self, "handle", None):
            B.mgi_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

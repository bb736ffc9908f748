/*
 * mgi.h -- C ABI of an MI355X (gfx950) inference engine for MobileNet-class
 * convolutional networks.
 *
 * The calls follow the structure of the GPU inference engine described in
 * "On-Device Neural Net Inference with Mobile GPUs" (Lee et al., 2019):
 *
 *   1. the caller describes the network as a graph of operators with their
 *      weights (Sec. 3.1, the delegate receives a graph of supported ops);
 *   2. finalize transforms the graph: it folds padding into the operators,
 *      fuses element-wise operators into the expensive operator that produces
 *      their input, and specialises kernels, e.g. 1x1 convolution
 *      (Sec. 3.2, "Shader Program Optimization");
 *   3. finalize plans the intermediate tensors into shared objects after a
 *      topological ordering of the graph (Sec. 5, Algorithm 1);
 *   4. run enqueues every kernel on one stream with no host synchronisation
 *      (Sec. 3.2, "Running Inference"), reading and writing device-resident
 *      inputs and outputs (Sec. 6, tensors placed in GPU buffers).
 *
 * Conventions shared by every entry point:
 *   - Every call returns an mgi_status; nothing throws across the ABI.  On a
 *     failure mgi_last_error() returns a thread-local message.
 *   - Host pointers passed to graph-building calls are read during the call
 *     only; the library copies what it keeps.  The caller keeps ownership.
 *   - The library never allocates device memory.  The caller allocates the
 *     workspace, the packed-weight buffer, the inputs and the outputs, and
 *     passes device pointers; they must stay valid while a plan uses them.
 *   - Streams are passed as `void *` holding a hipStream_t (NULL = the null
 *     stream).  A plan runs all of its kernels, in order, on that one stream;
 *     its buffer sharing is valid only under that in-order execution.
 *   - A plan is not re-entrant: at most one mgi_plan_run per plan may be in
 *     flight on the device at a time unless the runs are ordered by the stream.
 *   - Tensor shapes are (n, h, w, c): batch, height, width, channels.  Graph
 *     inputs are NHWC arrays in fp32 or fp16.  Graph outputs are NHWC arrays
 *     of fp32 values (an output of global_avgpool / fc / softmax is (n, c));
 *     argmax outputs are int32 arrays of shape (n, h, w).
 *   - Tensor ids are assigned in call order, starting at 0, one per
 *     graph-building call that returns an id.
 */
#ifndef MGI_H_
#define MGI_H_

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MGI_OK = 0,
    MGI_ERR_INVALID_ARG = 1, /* null pointer, bad id, non-positive size */
    MGI_ERR_SHAPE = 2,       /* operand shapes that do not fit the operator */
    MGI_ERR_UNSUPPORTED = 3, /* a valid request this engine does not implement */
    MGI_ERR_STATE = 4,       /* call out of order (e.g. run before bind) */
    MGI_ERR_WORKSPACE = 5,   /* a device buffer is missing or misaligned */
    MGI_ERR_HIP = 6,         /* the HIP runtime reported an error */
    MGI_ERR_OOM_HOST = 7,    /* host allocation failed */
    MGI_ERR_INTERNAL = 8     /* any other failure inside the library (a C++
                                exception stopped at the boundary); the
                                message is in mgi_last_error() */
} mgi_status;

typedef enum { MGI_ACT_NONE = 0, MGI_ACT_RELU = 1, MGI_ACT_RELU6 = 2 } mgi_act;

typedef enum {
    MGI_DTYPE_FP16 = 0,
    MGI_DTYPE_BF16 = 1,
    MGI_DTYPE_FP32 = 2,
    MGI_DTYPE_INT32 = 3
} mgi_dtype;

typedef enum {
    MGI_PLANNER_NAIVE = 0,  /* one buffer per intermediate tensor (Sec. 5, baseline) */
    MGI_PLANNER_GREEDY = 1, /* shared objects, Algorithm 1 (Sec. 5) */
    MGI_PLANNER_MCFP = 2    /* shared objects from a minimum-cost flow (Sec. 5, flow network
                               solved by successive shortest paths with SPFA); a tensor that
                               nothing consumes is free right after its producer */
} mgi_planner;

typedef struct mgi_graph mgi_graph;
typedef struct mgi_plan mgi_plan;

/* Convolution attributes.  Window (kh, kw), stride, dilation, explicit
 * four-sided zero padding (a separate PAD op folded into the convolution,
 * Sec. 3.1), output channels and the activation fused after it (Sec. 3.2).
 * Output size: oh = (h + pad_t + pad_b - dil_h * (kh - 1) - 1) / stride_h + 1,
 * likewise for ow.  cout is ignored by mgi_graph_add_depthwise. */
typedef struct {
    int kh, kw;
    int stride_h, stride_w;
    int dil_h, dil_w;
    int pad_t, pad_b, pad_l, pad_r;
    int cout;
    int act; /* mgi_act */
} mgi_conv_desc;

/* Options of mgi_graph_finalize.  Zero-initialised options are not valid;
 * call mgi_options_default first. */
typedef struct {
    int planner;         /* mgi_planner; default GREEDY */
    int fuse;            /* 1: fuse activations / residual adds into producers (default 1) */
    int materialize_all; /* 1: every node output keeps its own buffer so that
                            mgi_plan_read_node works after a run (default 0) */
    int dtype;           /* storage type of activations and weights: FP16 (default) or
                            BF16 (round to nearest even; MFMA and accumulation in fp32
                            either way); other values give MGI_ERR_UNSUPPORTED */
    int fuse_dwpw;       /* 1: run a 3x3 depthwise convolution (stride 1 or 2, no dilation)
                            inside the pointwise convolution that alone consumes it, when
                            that convolution has at most 320 output channels and enough
                            pixels to fill the GPU; the depthwise output then never reaches
                            memory (default 0; needs fuse = 1) */
    int fuse_pwdw;       /* run a 3x3 depthwise convolution (stride 1 or 2, no dilation, top
                            and left padding of at most one, planes up to 112 wide) inside
                            the pointwise convolution that produces its input, when that
                            output feeds nothing else; the pointwise output then never
                            reaches memory (Sec. 3.2's fusion extended to the pointwise ->
                            depthwise pair).  0: never; 1 (default): the fused kernel is the
                            default configuration when it gets at least 128 workgroups (tiles
                            x channel tiles; below that the separate kernels are), the other
                            one an autotune candidate; 2: the fused kernel is the default
                            whenever the shapes allow.  Needs fuse = 1. */
    int fuse_stemdw;     /* the same for the stem (a convolution over the graph input with
                            kh*kw*c <= 32 and at most 64 output channels) and a 3x3 depthwise
                            convolution at stride 1 that alone reads its output: 0, 1
                            (default) or 2 as for fuse_pwdw.  Needs fuse = 1. */
    int fuse_pool;       /* the same for a pointwise convolution (no residual) and a global
                            average pool over planes of at most 64 pixels that alone reads
                            its output: the means are written directly, bit-identical to the
                            two operators.  0, 1 (default) or 2 as for fuse_pwdw.  Needs
                            fuse = 1. */
    int fuse_softmax;    /* the same for a fully connected layer and the softmax that alone
                            reads its logits: the workgroup that completes a tile of rows
                            last runs their softmax, bit-identical to the two operators.  Its
                            arrival counters live in the workspace past the arena, zeroed by
                            mgi_plan_bind and left at zero by every run.  The fused kernel is
                            the default configuration for at most 16 rows (the two kernels
                            above that), the other one an autotune candidate.  0 or 1
                            (default).  Needs fuse = 1. */
    int fuse_irb;        /* run a 1x1 projection convolution (stride 1, at most 320 output
                            channels, optional residual add) inside a fused pointwise ->
                            depthwise node (fuse_pwdw) whose output only it reads: MobileNet-v2's
                            inverted residual block as one kernel, the expanded and depthwise
                            tensors kept on chip; bit-identical to the separate operators,
                            which stay autotune candidates.  0 (default): never; 1: the block
                            kernel is the default configuration when it gets at least 256
                            workgroups; 2: whenever the shapes allow.  Needs fuse_pwdw.  Off by
                            default: measured on MI355X it is not faster than the separate
                            kernels on most MobileNet-v2 blocks (they are bound by depthwise
                            vector-ALU work, not by the memory traffic it removes). */
} mgi_options;

/* ---------------------------------------------------------------------------
 * errors
 * ------------------------------------------------------------------------- */
/* Static text naming a status code (an mgi_status value; any other int gives
 * "MGI_ERR_UNKNOWN").  Never NULL. */
const char *mgi_status_str(int status);
/* Message of the most recent failed call on this thread ("" if none).  The
 * pointer stays valid until the next failing call on the same thread. */
const char *mgi_last_error(void);

/* ---------------------------------------------------------------------------
 * graph building (Sec. 3.1: the engine receives a graph of supported ops)
 * Every add call validates its operands and writes the id of the new tensor
 * to *out.  Shape errors are reported here; unsupported attribute
 * combinations are reported here or by finalize.
 * ------------------------------------------------------------------------- */
mgi_status mgi_graph_create(mgi_graph **g);
mgi_status mgi_graph_destroy(mgi_graph *g); /* NULL is accepted */

/* A graph input: an NHWC array of `dtype` (FP32 or FP16) supplied to run. */
mgi_status mgi_graph_add_input(mgi_graph *g, int n, int h, int w, int c, int dtype, int *out);

/* 2D convolution (Sec. 4.1, convolution over a kernel_height x kernel_width
 * window; the 1x1 case gets its own kernel, Sec. 3.2).
 * w: cout x kh x kw x cin floats (OHWI), bias: cout floats (NULL = zeros).
 * y = act(b + sum over window and input channels of w * x) with x zero
 * outside the input. */
mgi_status mgi_graph_add_conv2d(mgi_graph *g, int in, const mgi_conv_desc *d,
                                const float *w, const float *bias, int *out);

/* Depthwise convolution, channel multiplier 1: each channel is convolved with
 * its own kh x kw filter.  w: c x kh x kw floats, bias: c floats (NULL = 0). */
mgi_status mgi_graph_add_depthwise(mgi_graph *g, int in, const mgi_conv_desc *d,
                                   const float *w, const float *bias, int *out);

/* Element-wise y = act(a + b); a and b have equal shapes (Sec. 3.1, ADD). */
mgi_status mgi_graph_add_add(mgi_graph *g, int a, int b, int act, int *out);

/* Standalone activation; finalize fuses it into its producer when it can
 * (Sec. 3.2: element-wise operators fused with the expensive operator).
 * With fusion on, an activation NONE whose input is not a graph input and
 * whose output is not a graph output is an identity and is removed (Sec. 3.1:
 * graph transformations drop identity operations). */
mgi_status mgi_graph_add_activation(mgi_graph *g, int in, int act, int *out);

/* Spatial zero padding: output (n, h + pad_t + pad_b, w + pad_l + pad_r, c).
 * With fusion on, a PAD whose consumers are all conv2d / depthwise ops is
 * merged into their padding (Sec. 3.1); otherwise it runs as its own kernel.
 * Pads must be non-negative (MGI_ERR_INVALID_ARG). */
mgi_status mgi_graph_add_pad(mgi_graph *g, int in, int pad_t, int pad_b, int pad_l, int pad_r,
                             int *out);

/* Mean over h and w: (n, h, w, c) -> (n, 1, 1, c). */
mgi_status mgi_graph_add_global_avgpool(mgi_graph *g, int in, int *out);

/* Fully connected: input (n, h, w, c) is flattened per image to h*w*c values
 * (h = w = 1 is required); w: cout x cin floats, bias: cout floats.
 * Output (n, 1, 1, cout). */
mgi_status mgi_graph_add_fc(mgi_graph *g, int in, int cout, const float *w, const float *bias,
                            int *out);

/* Softmax over the channel axis: exp(z - max z) / sum exp(z - max z). */
mgi_status mgi_graph_add_softmax(mgi_graph *g, int in, int *out);

/* Channel concatenation in the given order; all inputs share n, h, w.  A
 * single-input concatenation is an identity (removed like activation NONE). */
mgi_status mgi_graph_add_concat(mgi_graph *g, const int *ins, int count, int *out);

/* Bilinear resize to (oh, ow).  align_corners = 1: source coordinate
 * d * (in - 1) / (out - 1); 0: d * in / out.  The upper neighbour is clamped
 * to the last sample.  A resize to the input's own size is an identity
 * (removed like activation NONE). */
mgi_status mgi_graph_add_resize_bilinear(mgi_graph *g, int in, int oh, int ow, int align_corners,
                                         int *out);

/* Per-pixel index of the largest channel (ties: lowest index), int32. */
mgi_status mgi_graph_add_argmax(mgi_graph *g, int in, int *out);

/* Mark a tensor as a graph output (in call order: output index 0, 1, ...).
 * Graph inputs cannot be outputs. */
mgi_status mgi_graph_mark_output(mgi_graph *g, int id);

/* ---------------------------------------------------------------------------
 * planning (pure host code; no device call)
 * ------------------------------------------------------------------------- */
void mgi_options_default(mgi_options *o);

/* Fuse, order, plan intermediate buffers and pack weights (Sec. 3.2, Sec. 5).
 * The graph is not modified and may be destroyed afterwards.  The plan owns
 * host copies of the packed weights until mgi_plan_bind uploads them. */
mgi_status mgi_graph_finalize(const mgi_graph *g, const mgi_options *o, mgi_plan **p);
mgi_status mgi_plan_destroy(mgi_plan *p); /* NULL is accepted */

/* Bytes of device workspace (the arena holding every intermediate tensor,
 * then a small state region: the arrival counters of fused FC + softmax
 * nodes) and of packed weights that the caller must allocate for
 * mgi_plan_bind.  Both buffers must be 256-byte aligned. */
mgi_status mgi_plan_workspace_bytes(const mgi_plan *p, size_t *bytes);
mgi_status mgi_plan_weight_bytes(const mgi_plan *p, size_t *bytes);

/* Memory of the intermediate tensors (Sec. 5, Table 3): `naive` = one buffer
 * per tensor, `planned` = the chosen planner's shared objects, `n_objects` =
 * number of shared objects.  Any out pointer may be NULL. */
mgi_status mgi_plan_memory_report(const mgi_plan *p, size_t *naive, size_t *planned,
                                  int *n_objects);

/* Graph inputs and outputs of the plan, in declaration / marking order. */
mgi_status mgi_plan_num_io(const mgi_plan *p, int *n_inputs, int *n_outputs);
/* Shape and element type (FP32 / FP16 for inputs, FP32 / INT32 for outputs)
 * of input or output `index` (is_output selects which); bytes = total size. */
mgi_status mgi_plan_io_info(const mgi_plan *p, int is_output, int index, int *n, int *h, int *w,
                            int *c, int *dtype, size_t *bytes);

/* Upload packed weights into dev_weights, adopt dev_workspace as the arena
 * and zero the workspace's state region (every run leaves it at zero again;
 * the caller must not write it).  The call waits for both before returning;
 * host copies of the weights are released once the upload is done with. */
mgi_status mgi_plan_bind(mgi_plan *p, void *dev_workspace, void *dev_weights, void *stream);

/* ---------------------------------------------------------------------------
 * running (Sec. 3.2: dispatch every program into the queue, no host sync)
 * ------------------------------------------------------------------------- */
/* dev_inputs[i] / dev_outputs[i]: device pointers for graph input / output i.
 * Enqueues all kernels on `stream` and returns without synchronising. */
mgi_status mgi_plan_run(mgi_plan *p, const void *const *dev_inputs, void *const *dev_outputs,
                        void *stream);

/* For callers that cannot allocate device memory while they run (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * as mgi_plan_run, but the plan's workspace (arena and state region) is the
 * library's own no-allocation workspace, a static device array of
 * MGI_NOALLOC_WORKSPACE_BYTES on each device, instead of the buffer given to
 * mgi_plan_bind (which this call does not touch; weights still come from the
 * bound weight buffer).  The array is placed when the library's kernels are
 * loaded on a device and held until the process ends; the call allocates and
 * frees nothing, on the device or through any library.  Its device address is
 * looked up on the first call on each device (the device current at the
 * call), so the first call is not capturable; later ones are (the state
 * region is cleared with a kernel, not a memset).
 *   Every call on one device shares that device's array: calls that overlap
 * on a device (two streams, two threads, two plans) race and give undefined
 * results; serialise them.  The array keeps the last call's contents, so
 * mgi_plan_read_node after this call reads it and is valid only until the
 * next call that uses it.
 *   Errors: as mgi_plan_run; MGI_ERR_WORKSPACE, before anything is enqueued,
 * when mgi_plan_workspace_bytes exceeds MGI_NOALLOC_WORKSPACE_BYTES (run such
 * a plan with mgi_plan_run); MGI_ERR_HIP if the address lookup fails. */
#define MGI_NOALLOC_WORKSPACE_BYTES (64u << 20)
mgi_status mgi_plan_run_noalloc(mgi_plan *p, const void *const *dev_inputs, void *const *dev_outputs,
                                void *stream);

/* As mgi_plan_run, and timestamps node kernels: node i's kernel is launched
 * so that start_events[i] is recorded when it begins executing on the device
 * and stop_events[i] when it ends (hipEvent_t values; NULL entries are not
 * recorded).  Both arrays hold node-count entries and are read during the
 * call only.  hipEventElapsedTime(start_events[i], stop_events[i]) is then
 * node i's kernel duration, with no host synchronisation in the run (the
 * paper's per-program timing of Sec. 6). */
mgi_status mgi_plan_run_timed(mgi_plan *p, const void *const *dev_inputs, void *const *dev_outputs,
                              void *stream, void *const *start_events, void *const *stop_events);

/* ---------------------------------------------------------------------------
 * introspection, used for layer-by-layer checks
 * ------------------------------------------------------------------------- */
/* Number of executable nodes after fusion. */
mgi_status mgi_plan_node_count(const mgi_plan *p, int *count);

/* Node `i`: `kind` (static string such as "pw_gemm", "dw3x3"), the graph
 * tensor id its output represents (the last operator it absorbed), the shape
 * of that tensor, and the number of graph operators fused into it. */
mgi_status mgi_plan_node_info(const mgi_plan *p, int i, const char **kind, int *tensor_id, int *n,
                              int *h, int *w, int *c, int *n_fused);

/* Copy node i's output, as an NHWC fp32 array (int32 for argmax), to
 * dev_dst on `stream`.  Requires materialize_all (MGI_ERR_STATE otherwise)
 * and a completed or stream-ordered run. */
mgi_status mgi_plan_read_node(mgi_plan *p, int i, void *dev_dst, void *stream);

/* Copy node i's output as stored: the channel-sliced 16-bit tensor (Sec. 4's
 * slices, 8 channels each), [ceil(c/8)][n*h*w][8] values including the
 * padding lanes of the last slice, raw fp16 (or bf16) bits, to dev_dst
 * (ceil(c/8) * n*h*w * 16 bytes) on `stream`; *bytes receives that size (it
 * may be queried with dev_dst NULL).  For checking that padding lanes hold
 * zeros.  Requires materialize_all and an enqueued run (MGI_ERR_STATE), and a
 * node whose output is stored sliced (MGI_ERR_UNSUPPORTED for fp32 logits,
 * probabilities and labels). */
mgi_status mgi_plan_read_node_raw(mgi_plan *p, int i, void *dev_dst, size_t *bytes, void *stream);

/* Plan-time tuning (after Sec. 4.2, where work-group sizes are chosen by
 * measurement): runs the plan once with these device buffers (same
 * arguments and checks as mgi_plan_run), then, node by node in run order,
 * times every candidate kernel configuration of each node that has several
 * (pointwise / implicit-GEMM, depthwise, fused pointwise -> depthwise) inside
 * `reps` whole runs of the plan, queued back to back (plus one warm-up run;
 * only the node's kernels are timestamped, so it meets its input as in a
 * run), and keeps the one with the lowest median time (a candidate listed
 * later replaces an earlier one only when more than 2% faster; fused forms
 * are listed before split ones).  All candidates produce bit-identical
 * results.  Synchronises `stream` once per candidate; releases a captured
 * graph (capture again afterwards).  The output buffers hold no defined
 * result afterwards: run the plan again.  Errors: MGI_ERR_INVALID_ARG for reps outside 1..1000; run
 * errors; MGI_ERR_HIP if timing fails. */
mgi_status mgi_plan_autotune(mgi_plan *p, const void *const *dev_inputs, void *const *dev_outputs,
                             void *stream, int reps);

/* Configuration in use by node i: its index among the node's candidates
 * (0 = the finalize-time choice), the number of candidates (1 for nodes
 * without alternatives) and a short name such as "pipe128x64" or "rows4"
 * (valid while the plan lives). */
mgi_status mgi_plan_node_config(const mgi_plan *p, int i, int *config, int *n_configs,
                                const char **name);

/* Use candidate `config` (0 <= config < n_configs) for node i from now on, as
 * a tuned choice would be; releases a captured graph.  For callers that
 * tune elsewhere or replay a stored tuning. */
mgi_status mgi_plan_set_node_config(mgi_plan *p, int i, int config);

/* Record one run with these device inputs and outputs (same arguments and
 * checks as mgi_plan_run) as a HIP graph held by the plan, replacing any
 * earlier one.  Extends the no-synchronisation dispatch of Sec. 3.2: the
 * whole launch list becomes one graph launch.  The recorded pointers are
 * baked in: the caller keeps those buffers alive and unchanged in size, and
 * refreshes their contents before each replay.  Nothing is executed by the
 * capture itself.  Errors: MGI_ERR_STATE before mgi_plan_bind; the run's
 * argument errors; MGI_ERR_HIP if capture or instantiation fails. */
mgi_status mgi_plan_capture(mgi_plan *p, const void *const *dev_inputs, void *const *dev_outputs);

/* Launch the captured graph on `stream` (asynchronous, like mgi_plan_run;
 * one replay at a time per plan, since replays share the plan's arena).
 * MGI_ERR_STATE if nothing has been captured. */
mgi_status mgi_plan_replay(mgi_plan *p, void *stream);

/* ---------------------------------------------------------------------------
 * stand-alone planner (Sec. 5: Algorithm 1 or the minimum-cost flow), for
 * planning outside a graph
 * ------------------------------------------------------------------------- */
/* Intermediate tensor t (0 <= t < n_tensors) has `sizes[t]` bytes, is produced
 * by operator first_op[t] and last used by operator last_op[t]
 * (first_op[t] <= last_op[t]; last_op[t] = -1 if nothing consumes it).
 * Operators are numbered in execution order.  Writes the shared object of
 * every tensor to object_of[t] and the object sizes to object_sizes[k]
 * (capacity n_tensors); *n_objects receives the object count. */
mgi_status mgi_planner_assign(int planner, int n_tensors, const size_t *sizes, const int *first_op,
                              const int *last_op, int *object_of, size_t *object_sizes,
                              int *n_objects);

#ifdef __cplusplus
}
#endif

#endif /* MGI_H_ */

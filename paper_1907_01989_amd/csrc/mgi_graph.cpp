// Graph building, validation and error reporting of the C ABI.
//
// Each add call checks its operands the way the paper's delegate checks that
// an operator is supported before taking it over (Sec. 3.1); there is no CPU
// fallback, an unsupported operator is reported as MGI_ERR_UNSUPPORTED.
#include <cstdio>
#include <cstring>
#include <new>

#include "mgi_internal.h"

namespace mgi {

static thread_local std::string g_last_error;

mgi_status fail(mgi_status s, const std::string &msg) {
    g_last_error = msg;
    return s;
}

}  // namespace mgi

using namespace mgi;

extern "C" const char *mgi_status_str(int s) {
    switch (s) {
        case MGI_OK: return "MGI_OK";
        case MGI_ERR_INVALID_ARG: return "MGI_ERR_INVALID_ARG";
        case MGI_ERR_SHAPE: return "MGI_ERR_SHAPE";
        case MGI_ERR_UNSUPPORTED: return "MGI_ERR_UNSUPPORTED";
        case MGI_ERR_STATE: return "MGI_ERR_STATE";
        case MGI_ERR_WORKSPACE: return "MGI_ERR_WORKSPACE";
        case MGI_ERR_HIP: return "MGI_ERR_HIP";
        case MGI_ERR_OOM_HOST: return "MGI_ERR_OOM_HOST";
        case MGI_ERR_INTERNAL: return "MGI_ERR_INTERNAL";
    }
    return "MGI_ERR_UNKNOWN";
}

extern "C" const char *mgi_last_error(void) { return g_last_error.c_str(); }

extern "C" mgi_status mgi_graph_create(mgi_graph **g) {
    MGI_ABI_TRY
    if (!g) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_create: null out pointer");
    *g = new (std::nothrow) mgi_graph();
    if (!*g) return fail(MGI_ERR_OOM_HOST, "mgi_graph_create: out of host memory");
    return MGI_OK;
    MGI_ABI_CATCH("mgi_graph_create")
}

extern "C" mgi_status mgi_graph_destroy(mgi_graph *g) {
    MGI_ABI_TRY
    delete g;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_graph_destroy")
}

namespace {

bool valid_act(int a) { return a == MGI_ACT_NONE || a == MGI_ACT_RELU || a == MGI_ACT_RELU6; }

mgi_status check_tensor(const mgi_graph *g, int id, const char *who) {
    if (!g) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null graph");
    if (id < 0 || id >= (int)g->ops.size())
        return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": tensor id " + std::to_string(id) +
                                             " does not exist");
    return MGI_OK;
}

mgi_status push(mgi_graph *g, GOp &&op, int *out) {
    try {
        g->ops.push_back(std::move(op));
    } catch (const std::bad_alloc &) {
        return fail(MGI_ERR_OOM_HOST, "out of host memory");
    }
    *out = (int)g->ops.size() - 1;
    return MGI_OK;
}

// Validates window attributes shared by conv2d and depthwise and computes the
// output size.
mgi_status conv_geometry(const Shape &x, const mgi_conv_desc *d, const char *who, int *oh, int *ow) {
    if (!d) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null descriptor");
    if (d->kh <= 0 || d->kw <= 0 || d->stride_h <= 0 || d->stride_w <= 0 || d->dil_h <= 0 ||
        d->dil_w <= 0 || d->pad_t < 0 || d->pad_b < 0 || d->pad_l < 0 || d->pad_r < 0)
        return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": window, stride and dilation must "
                                                            "be positive and pads non-negative");
    if (!valid_act(d->act)) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": bad activation");
    long eh = (long)x.h + d->pad_t + d->pad_b - (long)d->dil_h * (d->kh - 1) - 1;
    long ew = (long)x.w + d->pad_l + d->pad_r - (long)d->dil_w * (d->kw - 1) - 1;
    if (eh < 0 || ew < 0)
        return fail(MGI_ERR_SHAPE, std::string(who) + ": window larger than the padded input");
    *oh = (int)(eh / d->stride_h + 1);
    *ow = (int)(ew / d->stride_w + 1);
    return MGI_OK;
}

}  // namespace

extern "C" mgi_status mgi_graph_add_input(mgi_graph *g, int n, int h, int w, int c, int dtype,
                                          int *out) {
    MGI_ABI_TRY
    if (!g || !out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_input: null pointer");
    if (n <= 0 || h <= 0 || w <= 0 || c <= 0)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_input: sizes must be positive");
    if (dtype != MGI_DTYPE_FP32 && dtype != MGI_DTYPE_FP16)
        return fail(MGI_ERR_UNSUPPORTED, "mgi_graph_add_input: inputs are fp32 or fp16");
    GOp op;
    op.kind = OpKind::Input;
    op.out = {n, h, w, c};
    op.in_dtype = dtype;
    mgi_status s = push(g, std::move(op), out);
    if (s == MGI_OK) g->inputs.push_back(*out);
    return s;
    MGI_ABI_CATCH("mgi_graph_add_input")
}

extern "C" mgi_status mgi_graph_add_conv2d(mgi_graph *g, int in, const mgi_conv_desc *d,
                                           const float *w, const float *bias, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_conv2d");
    if (s) return s;
    if (!out || !w) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_conv2d: null pointer");
    const Shape x = g->ops[in].out;
    int oh, ow;
    if ((s = conv_geometry(x, d, "mgi_graph_add_conv2d", &oh, &ow))) return s;
    if (d->cout <= 0) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_conv2d: cout must be positive");
    GOp op;
    op.kind = OpKind::Conv2d;
    op.in = {in};
    op.conv = *d;
    op.act = d->act;
    op.out = {x.n, oh, ow, d->cout};
    size_t wn = (size_t)d->cout * d->kh * d->kw * x.c;
    try {
        op.w.assign(w, w + wn);
        if (bias) op.b.assign(bias, bias + d->cout); else op.b.assign(d->cout, 0.0f);
    } catch (const std::bad_alloc &) {
        return fail(MGI_ERR_OOM_HOST, "mgi_graph_add_conv2d: out of host memory");
    }
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_conv2d")
}

extern "C" mgi_status mgi_graph_add_depthwise(mgi_graph *g, int in, const mgi_conv_desc *d,
                                              const float *w, const float *bias, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_depthwise");
    if (s) return s;
    if (!out || !w) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_depthwise: null pointer");
    const Shape x = g->ops[in].out;
    int oh, ow;
    if ((s = conv_geometry(x, d, "mgi_graph_add_depthwise", &oh, &ow))) return s;
    GOp op;
    op.kind = OpKind::Depthwise;
    op.in = {in};
    op.conv = *d;
    op.conv.cout = x.c;
    op.act = d->act;
    op.out = {x.n, oh, ow, x.c};
    size_t wn = (size_t)x.c * d->kh * d->kw;
    try {
        op.w.assign(w, w + wn);
        if (bias) op.b.assign(bias, bias + x.c); else op.b.assign(x.c, 0.0f);
    } catch (const std::bad_alloc &) {
        return fail(MGI_ERR_OOM_HOST, "mgi_graph_add_depthwise: out of host memory");
    }
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_depthwise")
}

static bool same_shape(const Shape &a, const Shape &b) {
    return a.n == b.n && a.h == b.h && a.w == b.w && a.c == b.c;
}

extern "C" mgi_status mgi_graph_add_add(mgi_graph *g, int a, int b, int act, int *out) {
    MGI_ABI_TRY
    mgi_status s;
    if ((s = check_tensor(g, a, "mgi_graph_add_add")) || (s = check_tensor(g, b, "mgi_graph_add_add")))
        return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_add: null pointer");
    if (!valid_act(act)) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_add: bad activation");
    if (!same_shape(g->ops[a].out, g->ops[b].out))
        return fail(MGI_ERR_SHAPE, "mgi_graph_add_add: operand shapes differ");
    GOp op;
    op.kind = OpKind::Add;
    op.in = {a, b};
    op.act = act;
    op.out = g->ops[a].out;
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_add")
}

extern "C" mgi_status mgi_graph_add_activation(mgi_graph *g, int in, int act, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_activation");
    if (s) return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_activation: null pointer");
    if (!valid_act(act)) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_activation: bad activation");
    GOp op;
    op.kind = OpKind::Activation;
    op.in = {in};
    op.act = act;
    op.out = g->ops[in].out;
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_activation")
}

extern "C" mgi_status mgi_graph_add_pad(mgi_graph *g, int in, int pad_t, int pad_b, int pad_l,
                                        int pad_r, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_pad");
    if (s) return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_pad: null pointer");
    if (pad_t < 0 || pad_b < 0 || pad_l < 0 || pad_r < 0)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_pad: pads must be non-negative");
    GOp op;
    op.kind = OpKind::Pad;
    op.in = {in};
    op.pads[0] = pad_t;
    op.pads[1] = pad_b;
    op.pads[2] = pad_l;
    op.pads[3] = pad_r;
    op.out = g->ops[in].out;
    op.out.h += pad_t + pad_b;
    op.out.w += pad_l + pad_r;
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_pad")
}

extern "C" mgi_status mgi_graph_add_global_avgpool(mgi_graph *g, int in, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_global_avgpool");
    if (s) return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_global_avgpool: null pointer");
    GOp op;
    op.kind = OpKind::GlobalAvgPool;
    op.in = {in};
    const Shape x = g->ops[in].out;
    op.out = {x.n, 1, 1, x.c};
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_global_avgpool")
}

extern "C" mgi_status mgi_graph_add_fc(mgi_graph *g, int in, int cout, const float *w,
                                       const float *bias, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_fc");
    if (s) return s;
    if (!out || !w) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_fc: null pointer");
    if (cout <= 0) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_fc: cout must be positive");
    const Shape x = g->ops[in].out;
    if (x.h != 1 || x.w != 1)
        return fail(MGI_ERR_UNSUPPORTED, "mgi_graph_add_fc: input must be 1x1 spatially");
    GOp op;
    op.kind = OpKind::FC;
    op.in = {in};
    op.cout = cout;
    op.out = {x.n, 1, 1, cout};
    try {
        op.w.assign(w, w + (size_t)cout * x.c);
        if (bias) op.b.assign(bias, bias + cout); else op.b.assign(cout, 0.0f);
    } catch (const std::bad_alloc &) {
        return fail(MGI_ERR_OOM_HOST, "mgi_graph_add_fc: out of host memory");
    }
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_fc")
}

extern "C" mgi_status mgi_graph_add_softmax(mgi_graph *g, int in, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_softmax");
    if (s) return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_softmax: null pointer");
    GOp op;
    op.kind = OpKind::Softmax;
    op.in = {in};
    op.out = g->ops[in].out;
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_softmax")
}

extern "C" mgi_status mgi_graph_add_concat(mgi_graph *g, const int *ins, int count, int *out) {
    MGI_ABI_TRY
    if (!g || !ins || !out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_concat: null pointer");
    if (count < 1 || count > 8)
        return fail(count < 1 ? MGI_ERR_INVALID_ARG : MGI_ERR_UNSUPPORTED,
                    "mgi_graph_add_concat: 1 to 8 inputs");
    Shape o{};
    for (int i = 0; i < count; ++i) {
        mgi_status s = check_tensor(g, ins[i], "mgi_graph_add_concat");
        if (s) return s;
        const Shape x = g->ops[ins[i]].out;
        if (i == 0) o = x, o.c = 0;
        if (x.n != o.n || x.h != o.h || x.w != o.w)
            return fail(MGI_ERR_SHAPE, "mgi_graph_add_concat: inputs differ in n, h or w");
        o.c += x.c;
    }
    GOp op;
    op.kind = OpKind::Concat;
    op.in.assign(ins, ins + count);
    op.out = o;
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_concat")
}

extern "C" mgi_status mgi_graph_add_resize_bilinear(mgi_graph *g, int in, int oh, int ow,
                                                    int align_corners, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_resize_bilinear");
    if (s) return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_resize_bilinear: null pointer");
    if (oh <= 0 || ow <= 0)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_resize_bilinear: sizes must be positive");
    GOp op;
    op.kind = OpKind::ResizeBilinear;
    op.in = {in};
    op.oh = oh;
    op.ow = ow;
    op.align_corners = align_corners ? 1 : 0;
    const Shape x = g->ops[in].out;
    op.out = {x.n, oh, ow, x.c};
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_resize_bilinear")
}

extern "C" mgi_status mgi_graph_add_argmax(mgi_graph *g, int in, int *out) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, in, "mgi_graph_add_argmax");
    if (s) return s;
    if (!out) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_add_argmax: null pointer");
    GOp op;
    op.kind = OpKind::Argmax;
    op.in = {in};
    const Shape x = g->ops[in].out;
    op.out = {x.n, x.h, x.w, 1};
    return push(g, std::move(op), out);
    MGI_ABI_CATCH("mgi_graph_add_argmax")
}

extern "C" mgi_status mgi_graph_mark_output(mgi_graph *g, int id) {
    MGI_ABI_TRY
    mgi_status s = check_tensor(g, id, "mgi_graph_mark_output");
    if (s) return s;
    if (g->ops[id].kind == OpKind::Input)
        return fail(MGI_ERR_UNSUPPORTED, "mgi_graph_mark_output: a graph input cannot be an output");
    for (int t : g->outputs)
        if (t == id) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_mark_output: already an output");
    g->outputs.push_back(id);
    return MGI_OK;
    MGI_ABI_CATCH("mgi_graph_mark_output")
}

extern "C" void mgi_options_default(mgi_options *o) {
    if (!o) return;
    o->planner = MGI_PLANNER_GREEDY;
    o->fuse = 1;
    o->materialize_all = 0;
    o->dtype = MGI_DTYPE_FP16;
    o->fuse_dwpw = 0;
    o->fuse_pwdw = 1;
    o->fuse_stemdw = 1;
    o->fuse_pool = 1;
    o->fuse_softmax = 1;
    o->fuse_irb = 0;
}

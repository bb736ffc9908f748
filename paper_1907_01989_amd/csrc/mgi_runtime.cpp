// Binding and running a plan.
//
// mgi_plan_run enqueues every node's kernel on the caller's stream and
// returns without synchronising (Sec. 3.2: programs are inserted into the
// command queue and the GPU drains it with no CPU/GPU synchronisation).  All
// operands are resolved from three bases: the arena, the caller's inputs and
// the caller's outputs.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

#include <algorithm>
#include <mutex>
#include <string>

#include "kernels.h"
#include "mgi_internal.h"

using namespace mgi;
using namespace mgi::kern;

namespace {

mgi_status hip_fail(hipError_t e, const char *what) {
    return fail(MGI_ERR_HIP, std::string(what) + ": " + hipGetErrorName(e) + " (" +
                                 hipGetErrorString(e) + ")");
}

struct Bases {
    char *ws;
    const void *const *ins;
    void *const *outs;
};

void *buf_ptr(const mgi_plan &p, int b, const Bases &B) {
    const Buf &f = p.bufs[b];
    switch (f.loc) {
        case Loc::Arena: return B.ws + f.offset;
        case Loc::Input: return const_cast<void *>(B.ins[f.index]);
        case Loc::Output: return B.outs[f.index];
    }
    return nullptr;
}

inline int slices(int c) { return (c + 7) / 8; }

// The depthwise half of a split fused node: the 3x3 depthwise kernel from the
// node's scratch tensor (the first half's output) to its output.
hipError_t launch_split_dw(const mgi_plan &p, const Node &nd, const void *sp, void *y, bool bf, hipStream_t st) {
    const Shape mid = nd.dw_in, os = nd.dw_out;
    DwParams q{};
    q.bf16 = bf;
    q.x = (const h8 *)sp;
    q.w = (const h8 *)(static_cast<const char *>(p.dev_w) + nd.dw_w_off);
    q.bias = (const float *)(static_cast<const char *>(p.dev_w) + nd.dw_b_off);
    q.zero = (const h8 *)(static_cast<const char *>(p.dev_w) + p.zero_off);
    q.y = (h8 *)y;
    q.N = mid.n; q.H = mid.h; q.W = mid.w; q.S = slices(mid.c);
    q.OH = os.h; q.OW = os.w; q.KH = q.KW = 3;
    q.sh = q.sw = nd.dw_conv.stride_h;
    q.dh = q.dw = 1;
    q.pt = nd.dw_conv.pad_t; q.pl = nd.dw_conv.pad_l;
    q.act = nd.dw_act;
    return launch_depthwise(q, nd.dw_rows, st);
}

// A pointwise GEMM (no window) with the kernel a tile names.
hipError_t launch_gemm_tile(const GemmParams &q, const GemmTile &t, hipStream_t st) {
    if (t.pipe && t.ks == 8) return launch_gemm_pipe_k8(q, false, st);
    if (t.pipe) return launch_gemm_pipe(q, t.bm, t.bn, st);
    if (t.slab) return launch_gemm_xs(q, t.wm, t.bn, t.pf, false, st);
    return launch_gemm(q, t.bm, t.bn, false, false, st);
}

// The fused pointwise -> depthwise kernel of a PwDw or Irb node from its
// input to `y` (the node's output, or an Irb node's depthwise scratch).
hipError_t launch_node_pwdw(const mgi_plan &p, const Node &nd, const Bases &B, void *y, int ns, bool bf,
                            hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    PwDwParams q{};
    q.bf16 = bf;
    q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
    q.w = (const h8 *)(wbase + nd.w_off);
    q.bias = (const float *)(wbase + nd.b_off);
    q.M = (int)nd.dw_in.pixels();
    q.ksl = nd.ksl; q.ksp = nd.ksp; q.nb16 = nd.nb16; q.act1 = nd.act1;
    q.dw_w = (const h8 *)(wbase + nd.dw_w_off);
    q.dw_b = (const float *)(wbase + nd.dw_b_off);
    q.y = (h8 *)y;
    q.N = nd.dw_in.n; q.H = nd.dw_in.h; q.W = nd.dw_in.w; q.OH = nd.dw_out.h; q.OW = nd.dw_out.w;
    q.S = nd.dw_conv.stride_h; q.pt = nd.dw_conv.pad_t; q.pl = nd.dw_conv.pad_l;
    q.act2 = nd.dw_act;
    q.ns = ns;
    return launch_pwdw(q, nd.pwdw_cfg, st);
}

// The pointwise GEMM of a PwDw or Irb node's expansion into its scratch
// tensor (the split forms).
hipError_t launch_node_expand(const mgi_plan &p, const Node &nd, const Bases &B, bool bf, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const Shape mid = nd.dw_in;
    GemmParams g{};
    g.bf16 = bf;
    g.x = (const h8 *)buf_ptr(p, nd.in[0], B);
    g.w = (const h8 *)(wbase + nd.w_off);
    g.bias = (const float *)(wbase + nd.b_off);
    g.y = buf_ptr(p, nd.scratch, B);
    g.M = g.Min = (int)mid.pixels();
    g.ksl = nd.ksl; g.ksp = nd.ksp;
    g.nb16 = nd.nb16; g.ns = slices(mid.c); g.cout = mid.c;
    g.act1 = nd.act1; g.act2 = MGI_ACT_NONE;
    return nd.tile.ks == 8 ? launch_gemm_pipe_k8(g, false, st) : launch_gemm_pipe(g, nd.tile.bm, nd.tile.bn, st);
}

hipError_t launch_fcsoftmax_node(const mgi_plan &p, const Node &nd, const Bases &B, void *y, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    // FC + softmax: one FC launch whose last workgroup per row tile
    // runs the softmax, or (split) the FC into the logits scratch and
    // the softmax kernel
    const Shape lg = p.bufs[nd.scratch].shape;
    float *logits = (float *)buf_ptr(p, nd.scratch, B);
    GemmParams q{};
    q.bf16 = bf;
    q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
    q.w = (const h8 *)(wbase + nd.w_off);
    q.bias = (const float *)(wbase + nd.b_off);
    q.y = logits;
    q.M = (int)lg.pixels();
    q.Min = (int)p.bufs[nd.in[0]].shape.pixels();
    q.ksl = nd.ksl; q.ksp = nd.ksp;
    q.nb16 = nd.nb16; q.ns = slices(lg.c); q.cout = lg.c;
    q.act1 = nd.act1; q.act2 = nd.act2;
    if (!nd.split) {
        q.sm_y = (float *)y;
        q.sm_cnt = (int *)(B.ws + nd.cnt_off);
        return launch_fc(q, nd.tile.wm, nd.tile.pf, st);
    }
    LaunchEvents &ev = launch_events();
    const LaunchEvents saved = ev;
    ev.stop = nullptr;
    hipError_t e = launch_fc(q, nd.tile.wm, nd.tile.pf, st);
    ev.start = nullptr;
    ev.stop = saved.stop;
    if (e == hipSuccess) e = launch_softmax(logits, (float *)y, q.M, q.cout, st);
    ev = saved;
    return e;
}

hipError_t launch_irb_node(const mgi_plan &p, const Node &nd, const Bases &B, void *y, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const Shape os = p.bufs[nd.out].shape;
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    const Shape d = nd.dw_out;
    if (nd.mode == 0) {
        IrbParams q{};
        q.bf16 = bf;
        q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
        q.w = (const h8 *)(wbase + nd.w_off);
        q.bias = (const float *)(wbase + nd.b_off);
        q.M = (int)nd.dw_in.pixels();
        q.ksl = nd.ksl; q.ksp = nd.ksp; q.nb16 = nd.nb16; q.act1 = nd.act1;
        q.dw_w = (const h8 *)(wbase + nd.dw_w_off);
        q.dw_b = (const float *)(wbase + nd.dw_b_off);
        q.ns = slices(d.c); q.act2 = nd.dw_act;
        q.pw = (const h8 *)(wbase + nd.pj_w_off);
        q.pbias = (const float *)(wbase + nd.pj_b_off);
        q.pksp = nd.pj_ksp; q.pnb16 = nd.pj_nb16; q.pact1 = nd.pj_act1; q.pact2 = nd.pj_act2;
        q.res = nd.residual >= 0 ? (const h8 *)buf_ptr(p, nd.residual, B) : nullptr;
        q.y = (h8 *)y;
        q.ps = slices(os.c); q.MO = (int)os.pixels();
        q.N = nd.dw_in.n; q.H = nd.dw_in.h; q.W = nd.dw_in.w; q.OH = d.h; q.OW = d.w;
        q.S = nd.dw_conv.stride_h; q.pt = nd.dw_conv.pad_t; q.pl = nd.dw_conv.pad_l;
        return launch_irb(q, nd.pwdw_cfg, st);
    }
    // split forms: the expansion and depthwise into the depthwise
    // scratch (one fused kernel, or the GEMM and the depthwise kernel),
    // then the projection GEMM; a timed run stamps the first kernel's
    // start and the last one's end
    LaunchEvents &ev = launch_events();
    const LaunchEvents saved = ev;
    void *d2 = buf_ptr(p, nd.scratch2, B);
    hipError_t e;
    ev.stop = nullptr;
    if (nd.mode == 1) {
        e = launch_node_pwdw(p, nd, B, d2, slices(d.c), bf, st);
    } else {
        e = launch_node_expand(p, nd, B, bf, st);
        ev.start = nullptr;
        if (e == hipSuccess) e = launch_split_dw(p, nd, buf_ptr(p, nd.scratch, B), d2, bf, st);
    }
    ev.start = nullptr;
    ev.stop = saved.stop;
    if (e == hipSuccess) {
        GemmParams g{};
        g.bf16 = bf;
        g.x = (const h8 *)d2;
        g.w = (const h8 *)(wbase + nd.pj_w_off);
        g.bias = (const float *)(wbase + nd.pj_b_off);
        g.res = nd.residual >= 0 ? (const h8 *)buf_ptr(p, nd.residual, B) : nullptr;
        g.y = y;
        g.M = g.Min = (int)os.pixels();
        g.ksl = nd.pj_ksl; g.ksp = nd.pj_ksp;
        g.nb16 = nd.pj_nb16; g.ns = slices(os.c); g.cout = os.c;
        g.act1 = nd.pj_act1; g.act2 = nd.pj_act2;
        e = launch_gemm_tile(g, nd.pj_tile, st);
    }
    ev = saved;
    return e;
}

hipError_t launch_pwdw_node(const mgi_plan &p, const Node &nd, const Bases &B, void *y, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const Shape os = p.bufs[nd.out].shape;
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    if (nd.split) {
        // the pointwise GEMM into the scratch tensor, then the depthwise
        // kernel; a timed run stamps the first kernel's start and the
        // second one's end
        LaunchEvents &ev = launch_events();
        const LaunchEvents saved = ev;
        const Shape mid = nd.dw_in;
        void *sp = buf_ptr(p, nd.scratch, B);
        GemmParams g{};
        g.bf16 = bf;
        g.x = (const h8 *)buf_ptr(p, nd.in[0], B);
        g.w = (const h8 *)(wbase + nd.w_off);
        g.bias = (const float *)(wbase + nd.b_off);
        g.y = sp;
        g.M = g.Min = (int)mid.pixels();
        g.ksl = nd.ksl; g.ksp = nd.ksp;
        g.nb16 = nd.nb16; g.ns = slices(mid.c); g.cout = mid.c;
        g.act1 = nd.act1; g.act2 = MGI_ACT_NONE;
        ev.stop = nullptr;
        hipError_t e = nd.tile.ks == 8 ? launch_gemm_pipe_k8(g, false, st)
                                       : launch_gemm_pipe(g, nd.tile.bm, nd.tile.bn, st);
        ev.start = nullptr;
        ev.stop = saved.stop;
        if (e == hipSuccess) e = launch_split_dw(p, nd, sp, y, bf, st);
        ev = saved;
        return e;
    }
    PwDwParams q{};
    q.bf16 = bf;
    q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
    q.w = (const h8 *)(wbase + nd.w_off);
    q.bias = (const float *)(wbase + nd.b_off);
    q.M = (int)nd.dw_in.pixels();
    q.ksl = nd.ksl; q.ksp = nd.ksp; q.nb16 = nd.nb16; q.act1 = nd.act1;
    q.dw_w = (const h8 *)(wbase + nd.dw_w_off);
    q.dw_b = (const float *)(wbase + nd.dw_b_off);
    q.y = (h8 *)y;
    q.N = nd.dw_in.n; q.H = nd.dw_in.h; q.W = nd.dw_in.w; q.OH = os.h; q.OW = os.w;
    q.S = nd.dw_conv.stride_h; q.pt = nd.dw_conv.pad_t; q.pl = nd.dw_conv.pad_l;
    q.act2 = nd.dw_act;
    q.ns = slices(os.c);
    return launch_pwdw(q, nd.pwdw_cfg, st);
}

hipError_t launch_gemmpool_node(const mgi_plan &p, const Node &nd, const Bases &B, void *y, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    // pointwise GEMM + global average pool: the pooled GEMM kernel,
    // or (split) the GEMM into the scratch tensor and the pool kernel
    const Shape mid = nd.dw_in;
    GemmParams g{};
    g.bf16 = bf;
    g.x = (const h8 *)buf_ptr(p, nd.in[0], B);
    g.w = (const h8 *)(wbase + nd.w_off);
    g.bias = (const float *)(wbase + nd.b_off);
    g.M = g.Min = (int)mid.pixels();
    g.ksl = nd.ksl; g.ksp = nd.ksp;
    g.nb16 = nd.nb16; g.ns = slices(mid.c); g.cout = mid.c;
    g.act1 = nd.act1; g.act2 = MGI_ACT_NONE;
    if (!nd.split) {
        g.y = y;
        g.hw = mid.h * mid.w;
        g.nimg = mid.n;
        if (nd.tile.slab) return launch_gemm_xs(g, nd.tile.wm, nd.tile.bn, nd.tile.pf, true, st);
        if (nd.tile.ks == 8) return launch_gemm_pipe_k8(g, true, st);
        return launch_gemm_pool(g, nd.tile.bm, nd.tile.bn, st);
    }
    LaunchEvents &ev = launch_events();
    const LaunchEvents saved = ev;
    void *sp = buf_ptr(p, nd.scratch, B);
    g.y = sp;
    ev.stop = nullptr;
    hipError_t e = launch_gemm_pipe(g, nd.tile.bm, nd.tile.bn, st);
    ev.start = nullptr;
    ev.stop = saved.stop;
    if (e == hipSuccess)
        e = launch_gap((const h8 *)sp, (h8 *)y, (const h8 *)(wbase + p.zero_off), mid.n, mid.h * mid.w,
                       slices(mid.c), bf, st);
    ev = saved;
    return e;
}

hipError_t launch_stemdw_node(const mgi_plan &p, const Node &nd, const Bases &B, void *y, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    const Buf &ib = p.bufs[nd.in[0]];
    const bool fp16_in = ib.in_dtype == MGI_DTYPE_FP16;
    if (nd.split) {
        // the stem kernel into the scratch tensor, then the depthwise
        // kernel (timed as one: first kernel's start, second's end)
        LaunchEvents &ev = launch_events();
        const LaunchEvents saved = ev;
        const Shape mid = nd.dw_in;
        void *sp = buf_ptr(p, nd.scratch, B);
        StemParams q{};
        q.bf16 = bf;
        q.x = buf_ptr(p, nd.in[0], B);
        q.w = (const h8 *)(wbase + nd.w_off);
        q.bias = (const float *)(wbase + nd.b_off);
        q.res = nullptr;
        q.y = (h8 *)sp;
        q.N = ib.shape.n; q.H = ib.shape.h; q.W = ib.shape.w; q.C = ib.shape.c;
        q.OH = mid.h; q.OW = mid.w; q.M = (int)mid.pixels();
        q.KH = nd.conv.kh; q.KW = nd.conv.kw; q.K = nd.conv.kh * nd.conv.kw * ib.shape.c;
        q.sh = nd.conv.stride_h; q.sw = nd.conv.stride_w;
        q.dh = nd.conv.dil_h; q.dw = nd.conv.dil_w;
        q.pt = nd.conv.pad_t; q.pl = nd.conv.pad_l;
        q.nb16 = nd.nb16; q.ns = slices(mid.c);
        q.act1 = nd.act1; q.act2 = MGI_ACT_NONE;
        ev.stop = nullptr;
        hipError_t e = launch_stem(q, fp16_in, st);
        ev.start = nullptr;
        ev.stop = saved.stop;
        if (e == hipSuccess) e = launch_split_dw(p, nd, sp, y, bf, st);
        ev = saved;
        return e;
    }
    StemDwParams q{};
    stemdw_shape(p, nd, q);
    q.bf16 = bf;
    q.x = buf_ptr(p, nd.in[0], B);
    q.w = (const h8 *)(wbase + nd.w_off);
    q.bias = (const float *)(wbase + nd.b_off);
    q.dw_w = (const h8 *)(wbase + nd.dw_w_off);
    q.dw_b = (const float *)(wbase + nd.dw_b_off);
    q.y = (h8 *)y;
    return launch_stemdw(q, nd.pwdw_cfg, fp16_in, st);
}

hipError_t launch_dwpw_node(const mgi_plan &p, const Node &nd, const Bases &B, void *y, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const Shape os = p.bufs[nd.out].shape;
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    const Buf &ib = p.bufs[nd.in[0]];
    DwPwParams q{};
    q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
    q.dww = (const h8 *)(wbase + nd.dw_w_off);
    q.dwb = (const float *)(wbase + nd.dw_b_off);
    q.zero = (const h8 *)(wbase + p.zero_off);
    q.N = ib.shape.n; q.H = ib.shape.h; q.W = ib.shape.w; q.OH = os.h; q.OW = os.w;
    q.sh = nd.dw_conv.stride_h; q.sw = nd.dw_conv.stride_w;
    q.pt = nd.dw_conv.pad_t; q.pl = nd.dw_conv.pad_l; q.act = nd.dw_act;
    GemmParams &g = q.g;
    g.bf16 = bf;
    g.w = (const h8 *)(wbase + nd.w_off);
    g.bias = (const float *)(wbase + nd.b_off);
    g.res = nd.residual >= 0 ? (const h8 *)buf_ptr(p, nd.residual, B) : nullptr;
    g.y = y;
    g.M = (int)os.pixels();
    g.Min = g.M;
    g.ksl = nd.ksl; g.ksp = nd.ksp;
    g.nb16 = nd.nb16; g.ns = slices(os.c); g.cout = os.c;
    g.act1 = nd.act1; g.act2 = nd.act2;
    DwPwTile t;
    if (!dwpw_tile(os.h, os.w, q.sh, os.n, t, nd.tile.bm > 0 ? nd.tile.bm : 128))
        return hipErrorInvalidValue;
    return launch_dwpw(q, t, st);
}

hipError_t launch_node(const mgi_plan &p, const Node &nd, const Bases &B, hipStream_t st) {
    const char *wbase = static_cast<const char *>(p.dev_w);
    const Buf &ob = p.bufs[nd.out];
    const Shape os = ob.shape;
    void *y = buf_ptr(p, nd.out, B);
    const bool bf = p.opt.dtype == MGI_DTYPE_BF16;
    switch (nd.kind) {
        case NodeKind::Ingest: {
            const Buf &ib = p.bufs[nd.in[0]];
            return launch_ingest(buf_ptr(p, nd.in[0], B), ib.in_dtype == MGI_DTYPE_FP16, (h8 *)y,
                                 (int)ib.shape.pixels(), ib.shape.c, bf, st);
        }
        case NodeKind::Stem: {
            const Buf &ib = p.bufs[nd.in[0]];
            StemParams q{};
            q.bf16 = bf;
            q.x = buf_ptr(p, nd.in[0], B);
            q.w = (const h8 *)(wbase + nd.w_off);
            q.bias = (const float *)(wbase + nd.b_off);
            q.res = nd.residual >= 0 ? (const h8 *)buf_ptr(p, nd.residual, B) : nullptr;
            q.y = (h8 *)y;
            q.N = ib.shape.n; q.H = ib.shape.h; q.W = ib.shape.w; q.C = ib.shape.c;
            q.OH = os.h; q.OW = os.w; q.M = (int)os.pixels();
            q.KH = nd.conv.kh; q.KW = nd.conv.kw; q.K = nd.conv.kh * nd.conv.kw * ib.shape.c;
            q.sh = nd.conv.stride_h; q.sw = nd.conv.stride_w;
            q.dh = nd.conv.dil_h; q.dw = nd.conv.dil_w;
            q.pt = nd.conv.pad_t; q.pl = nd.conv.pad_l;
            q.nb16 = nd.nb16; q.ns = slices(os.c);
            q.act1 = nd.act1; q.act2 = nd.act2;
            return launch_stem(q, ib.in_dtype == MGI_DTYPE_FP16, st);
        }
        case NodeKind::FcSoftmax:
            return launch_fcsoftmax_node(p, nd, B, y, st);
        case NodeKind::Gemm:
        case NodeKind::FC: {
            const Buf &ib = p.bufs[nd.in[0]];
            GemmParams q{};
            q.bf16 = bf;
            q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
            q.w = (const h8 *)(wbase + nd.w_off);
            q.bias = (const float *)(wbase + nd.b_off);
            q.res = nd.residual >= 0 ? (const h8 *)buf_ptr(p, nd.residual, B) : nullptr;
            q.y = y;
            q.M = (int)os.pixels();
            q.Min = (int)ib.shape.pixels();
            q.ksl = nd.ksl; q.ksp = nd.ksp;
            q.nb16 = nd.nb16; q.ns = slices(os.c); q.cout = os.c;
            q.act1 = nd.act1; q.act2 = nd.act2;
            q.H = ib.shape.h; q.W = ib.shape.w; q.OH = os.h; q.OW = os.w;
            q.sin = slices(ib.shape.c); q.kw = nd.conv.kw;
            q.sh = nd.conv.stride_h; q.sw = nd.conv.stride_w;
            q.dh = nd.conv.dil_h; q.dw = nd.conv.dil_w;
            q.pt = nd.conv.pad_t; q.pl = nd.conv.pad_l;
            if (nd.kind == NodeKind::FC) return launch_fc(q, nd.tile.wm, nd.tile.pf, st);
            if (nd.tile.pipe && nd.tile.ks == 8) return launch_gemm_pipe_k8(q, false, st);
            if (nd.tile.pipe) return launch_gemm_pipe(q, nd.tile.bm, nd.tile.bn, st);
            if (nd.tile.slab) return launch_gemm_xs(q, nd.tile.wm, nd.tile.bn, nd.tile.pf, false, st);
            return launch_gemm(q, nd.tile.bm, nd.tile.bn, nd.taps, nd.kind == NodeKind::FC, st);
        }
        case NodeKind::DwPw:
            return launch_dwpw_node(p, nd, B, y, st);
        case NodeKind::Irb:
            return launch_irb_node(p, nd, B, y, st);
        case NodeKind::PwDw:
            return launch_pwdw_node(p, nd, B, y, st);
        case NodeKind::GemmPool:
            return launch_gemmpool_node(p, nd, B, y, st);
        case NodeKind::StemDw:
            return launch_stemdw_node(p, nd, B, y, st);
        case NodeKind::Depthwise: {
            const Buf &ib = p.bufs[nd.in[0]];
            DwParams q{};
            q.bf16 = bf;
            q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
            q.w = (const h8 *)(wbase + nd.w_off);
            q.bias = (const float *)(wbase + nd.b_off);
            q.zero = (const h8 *)(wbase + p.zero_off);
            q.y = (h8 *)y;
            q.N = ib.shape.n; q.H = ib.shape.h; q.W = ib.shape.w; q.S = slices(ib.shape.c);
            q.OH = os.h; q.OW = os.w; q.KH = nd.conv.kh; q.KW = nd.conv.kw;
            q.sh = nd.conv.stride_h; q.sw = nd.conv.stride_w;
            q.dh = nd.conv.dil_h; q.dw = nd.conv.dil_w;
            q.pt = nd.conv.pad_t; q.pl = nd.conv.pad_l;
            q.act = nd.act1;
            return launch_depthwise(q, nd.dw_rows, st);
        }
        case NodeKind::Add:
            return launch_add((const h8 *)buf_ptr(p, nd.in[0], B), (const h8 *)buf_ptr(p, nd.in[1], B),
                              (h8 *)y, (size_t)slices(os.c) * os.pixels(), nd.act1, bf, st);
        case NodeKind::Act:
            return launch_act((const h8 *)buf_ptr(p, nd.in[0], B), (h8 *)y,
                              (size_t)slices(os.c) * os.pixels(), nd.act1, bf, st);
        case NodeKind::Gap: {
            const Buf &ib = p.bufs[nd.in[0]];
            return launch_gap((const h8 *)buf_ptr(p, nd.in[0], B), (h8 *)y,
                              (const h8 *)(wbase + p.zero_off), ib.shape.n,
                              ib.shape.h * ib.shape.w, slices(ib.shape.c), bf, st);
        }
        case NodeKind::Softmax:
            return launch_softmax((const float *)buf_ptr(p, nd.in[0], B), (float *)y,
                                  (int)os.pixels(), os.c, st);
        case NodeKind::Pad: {
            const Buf &ib = p.bufs[nd.in[0]];
            return launch_pad((const h8 *)buf_ptr(p, nd.in[0], B), (h8 *)y, ib.shape.n,
                              slices(ib.shape.c), ib.shape.h, ib.shape.w, os.h, os.w, nd.conv.pad_t,
                              nd.conv.pad_l, st);
        }
        case NodeKind::Concat: {
            ConcatParams q{};
            q.nin = (int)nd.in.size();
            int off = 0;
            for (int k = 0; k < q.nin; ++k) {
                q.src[k] = (const h8 *)buf_ptr(p, nd.in[k], B);
                q.coff[k] = off;
                off += p.bufs[nd.in[k]].shape.c;
            }
            q.coff[q.nin] = off;
            q.M = (int)os.pixels(); q.S = slices(os.c); q.C = os.c;
            q.y = (h8 *)y;
            return launch_concat(q, st);
        }
        case NodeKind::Resize:
        case NodeKind::ResizeArgmax: {
            const Buf &ib = p.bufs[nd.in[0]];
            ResizeParams q{};
            q.x = (const h8 *)buf_ptr(p, nd.in[0], B);
            q.y = y;
            q.N = ib.shape.n; q.H = ib.shape.h; q.W = ib.shape.w;
            q.S = slices(ib.shape.c); q.C = ib.shape.c;
            q.OH = os.h; q.OW = os.w;
            q.align_corners = nd.align_corners;
            q.bf16 = bf;
            return launch_resize(q, nd.kind == NodeKind::ResizeArgmax, st);
        }
        case NodeKind::Argmax: {
            const Buf &ib = p.bufs[nd.in[0]];
            return launch_argmax((const h8 *)buf_ptr(p, nd.in[0], B), (int *)y,
                                 (int)ib.shape.pixels(), slices(ib.shape.c), ib.shape.c, bf, st);
        }
        case NodeKind::Export: {
            const Buf &ib = p.bufs[nd.in[0]];
            return launch_export((const h8 *)buf_ptr(p, nd.in[0], B), (float *)y,
                                 (int)ib.shape.pixels(), ib.shape.c, bf, st);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace

namespace {

void release_graph(mgi_plan &p) {
    if (p.graph_exec) (void)hipGraphExecDestroy(static_cast<hipGraphExec_t>(p.graph_exec));
    if (p.graph) (void)hipGraphDestroy(static_cast<hipGraph_t>(p.graph));
    p.graph_exec = nullptr;
    p.graph = nullptr;
    p.graph_outputs.clear();
}

}  // namespace

mgi_plan::~mgi_plan() { release_graph(*this); }

extern "C" mgi_status mgi_plan_destroy(mgi_plan *p) {
    MGI_ABI_TRY
    delete p;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_destroy")
}

extern "C" mgi_status mgi_plan_bind(mgi_plan *p, void *dev_workspace, void *dev_weights,
                                    void *stream) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_bind: null plan");
    if (!dev_workspace || !dev_weights)
        return fail(MGI_ERR_WORKSPACE, "mgi_plan_bind: workspace and weight buffers are required");
    if (((uintptr_t)dev_workspace & 255) || ((uintptr_t)dev_weights & 255))
        return fail(MGI_ERR_WORKSPACE, "mgi_plan_bind: buffers must be 256-byte aligned");
    if (p->bound && p->weights.empty())
        return fail(MGI_ERR_STATE, "mgi_plan_bind: plan already bound");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (!p->weights.empty()) {
        hipError_t e = hipMemcpyAsync(dev_weights, p->weights.data(), p->weights.size(),
                                      hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return hip_fail(e, "mgi_plan_bind: weight upload");
        e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "mgi_plan_bind: weight upload");
    }
    if (p->state_bytes) {   // counters start at zero; runs leave them at zero
        hipError_t e = hipMemsetAsync(static_cast<char *>(dev_workspace) + p->state_off, 0,
                                      p->state_bytes, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "mgi_plan_bind: state region");
    }
    std::vector<uint8_t>().swap(p->weights);
    p->dev_ws = dev_workspace;
    p->dev_w = dev_weights;
    p->bound = true;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_bind")
}

namespace {

// Enqueues every node of a bound plan on `stream`, with the arena and state
// region at `ws` (the bound workspace, or the no-allocation workspace).
mgi_status run_plan(mgi_plan *p, const void *const *dev_inputs, void *const *dev_outputs,
                    void *stream, void *const *start_ev, void *const *stop_ev, const char *who,
                    char *ws = nullptr) {
    if (!p) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null plan");
    if (!p->bound) return fail(MGI_ERR_STATE, std::string(who) + ": plan is not bound");
    if (!p->input_bufs.empty() && !dev_inputs)
        return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null input array");
    if (!dev_outputs) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null output array");
    for (size_t i = 0; i < p->input_bufs.size(); ++i)
        if (!dev_inputs[i]) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null input pointer");
    for (size_t i = 0; i < p->output_bufs.size(); ++i)
        if (!dev_outputs[i]) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null output pointer");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (!ws) ws = static_cast<char *>(p->dev_ws);
    Bases B{ws, dev_inputs, dev_outputs};
    LaunchEvents &ev = launch_events();
    for (size_t i = 0; i < p->nodes.size(); ++i) {
        ev.start = start_ev ? static_cast<hipEvent_t>(start_ev[i]) : nullptr;
        ev.stop = stop_ev ? static_cast<hipEvent_t>(stop_ev[i]) : nullptr;
        hipError_t e = launch_node(*p, p->nodes[i], B, st);
        ev.start = ev.stop = nullptr;
        if (e != hipSuccess)
            return hip_fail(e, (std::string(who) + ": node " + std::to_string(i) + " (" +
                                p->nodes[i].kname + ")").c_str());
    }
    p->last_outputs.assign(dev_outputs, dev_outputs + p->output_bufs.size());
    p->last_ws = ws;
    return MGI_OK;
}

// ---------------------------------------------------------------------------
// the no-allocation workspace: one array per device, placed by the code
// object loader when the library's kernels are loaded on that device, never
// allocated or freed by the library.  Host code must not use the array's name
// as a device address (on the host it names a stand-in): the address is
// looked up once per device with hipGetSymbolAddress and kept here.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[MGI_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's array, looked up on the first call
// on that device.
mgi_status noalloc_workspace(char **out, const char *who) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, who);
    if (dev < 0 || dev >= kMaxDevices)
        return fail(MGI_ERR_UNSUPPORTED, std::string(who) + ": device index " + std::to_string(dev) +
                                             " beyond the " + std::to_string(kMaxDevices) + " supported");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, (std::string(who) + ": workspace address").c_str());
        if (!ptr || ((uintptr_t)ptr & 255))
            return fail(MGI_ERR_WORKSPACE, std::string(who) + ": workspace address not 256-byte aligned");
        g_scratch_ptr[dev] = ptr;
    }
    *out = static_cast<char *>(g_scratch_ptr[dev]);
    return MGI_OK;
}

}  // namespace

extern "C" mgi_status mgi_plan_run(mgi_plan *p, const void *const *dev_inputs,
                                   void *const *dev_outputs, void *stream) {
    MGI_ABI_TRY
    return run_plan(p, dev_inputs, dev_outputs, stream, nullptr, nullptr, "mgi_plan_run");
    MGI_ABI_CATCH("mgi_plan_run")
}

extern "C" mgi_status mgi_plan_run_noalloc(mgi_plan *p, const void *const *dev_inputs,
                                           void *const *dev_outputs, void *stream) {
    MGI_ABI_TRY
    const char *who = "mgi_plan_run_noalloc";
    if (!p) return fail(MGI_ERR_INVALID_ARG, std::string(who) + ": null plan");
    if (!p->bound) return fail(MGI_ERR_STATE, std::string(who) + ": plan is not bound");
    if (p->workspace_bytes > (size_t)MGI_NOALLOC_WORKSPACE_BYTES)
        return fail(MGI_ERR_WORKSPACE,
                    std::string(who) + ": the plan needs a workspace of " + std::to_string(p->workspace_bytes) +
                        " bytes, more than the " + std::to_string((size_t)MGI_NOALLOC_WORKSPACE_BYTES) +
                        " bytes of the no-allocation workspace; run it with mgi_plan_run");
    char *ws = nullptr;
    mgi_status s = noalloc_workspace(&ws, who);
    if (s != MGI_OK) return s;
    // the array holds whatever the previous call on this device left there:
    // the state region (arrival counters) must start at zero
    if (p->state_bytes) {
        hipError_t e = launch_zero_words(reinterpret_cast<unsigned *>(ws + p->state_off),
                                         p->state_bytes / sizeof(unsigned), static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return hip_fail(e, (std::string(who) + ": state region").c_str());
    }
    return run_plan(p, dev_inputs, dev_outputs, stream, nullptr, nullptr, who, ws);
    MGI_ABI_CATCH("mgi_plan_run_noalloc")
}

extern "C" mgi_status mgi_plan_run_timed(mgi_plan *p, const void *const *dev_inputs,
                                         void *const *dev_outputs, void *stream,
                                         void *const *start_events, void *const *stop_events) {
    MGI_ABI_TRY
    if (!start_events || !stop_events)
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_run_timed: null event array");
    return run_plan(p, dev_inputs, dev_outputs, stream, start_events, stop_events,
                    "mgi_plan_run_timed");
    MGI_ABI_CATCH("mgi_plan_run_timed")
}

// The launch list of one run is recorded once through stream capture on a
// stream of the library's own (the caller's stream may be the null stream,
// which cannot be captured), instantiated, and then replayed with a single
// graph launch: the per-kernel launch cost of the eager loop, which dominates
// at batch 1, is paid once at capture.  No node issues a memset or copy, so
// the graph holds kernel nodes only.
extern "C" mgi_status mgi_plan_capture(mgi_plan *p, const void *const *dev_inputs,
                                       void *const *dev_outputs) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_capture: null plan");
    if (!p->bound) return fail(MGI_ERR_STATE, "mgi_plan_capture: plan is not bound");
    release_graph(*p);
    hipStream_t cs = nullptr;
    hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
    if (e != hipSuccess) return hip_fail(e, "mgi_plan_capture: stream");
    e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
        (void)hipStreamDestroy(cs);
        return hip_fail(e, "mgi_plan_capture: begin capture");
    }
    const mgi_status st = run_plan(p, dev_inputs, dev_outputs, cs, nullptr, nullptr, "mgi_plan_capture");
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(cs, &g);
    (void)hipStreamDestroy(cs);
    if (st != MGI_OK) {
        if (g) (void)hipGraphDestroy(g);
        return st;
    }
    if (e != hipSuccess) return hip_fail(e, "mgi_plan_capture: end capture");
    hipGraphExec_t ge = nullptr;
    e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        (void)hipGraphDestroy(g);
        return hip_fail(e, "mgi_plan_capture: instantiate");
    }
    p->graph = g;
    p->graph_exec = ge;
    p->graph_outputs.assign(dev_outputs, dev_outputs + p->output_bufs.size());
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_capture")
}

extern "C" mgi_status mgi_plan_replay(mgi_plan *p, void *stream) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_replay: null plan");
    if (!p->graph_exec) return fail(MGI_ERR_STATE, "mgi_plan_replay: nothing captured");
    hipError_t e = hipGraphLaunch(static_cast<hipGraphExec_t>(p->graph_exec),
                                  static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "mgi_plan_replay");
    p->last_outputs = p->graph_outputs;
    p->last_ws = p->dev_ws;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_replay")
}

// Plan-time tuning, the counterpart of choosing work-group sizes by
// measurement (Sec. 4.2): every node with more than one candidate
// configuration is launched reps + 1 times per candidate on the plan's own
// buffers (after one full run has filled them), each launch timestamped on the
// device; the one with the lowest median over the timed launches (the first
// launch being a warm-up) is kept, a later candidate replacing an earlier one
// only when more than 2% faster.  Candidates compute identical results, so tuning changes
// speed only.  A captured graph holds the old configurations and is released.
extern "C" mgi_status mgi_plan_autotune(mgi_plan *p, const void *const *dev_inputs,
                                        void *const *dev_outputs, void *stream, int reps) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_autotune: null plan");
    if (reps < 1 || reps > 1000) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_autotune: reps in 1..1000");
    mgi_status s = run_plan(p, dev_inputs, dev_outputs, stream, nullptr, nullptr, "mgi_plan_autotune");
    if (s != MGI_OK) return s;
    release_graph(*p);
    hipStream_t st = static_cast<hipStream_t>(stream);
    // one start/stop pair per run, so that a candidate's runs go back to
    // back (as in steady operation) and are read after one synchronisation
    std::vector<hipEvent_t> evs(2 * (size_t)(reps + 1), nullptr);
    hipError_t e = hipSuccess;
    for (size_t k = 0; k < evs.size() && e == hipSuccess; ++k) e = hipEventCreate(&evs[k]);
    auto destroy = [&]() {
        for (hipEvent_t x : evs)
            if (x) (void)hipEventDestroy(x);
    };
    if (e != hipSuccess) {
        destroy();
        return hip_fail(e, "mgi_plan_autotune: events");
    }
    Bases B{static_cast<char *>(p->dev_ws), dev_inputs, dev_outputs};
    LaunchEvents &ev = launch_events();
    mgi_status result = MGI_OK;
    std::vector<float> times;
    for (size_t ni = 0; ni < p->nodes.size() && result == MGI_OK; ++ni) {
        Node &nd = p->nodes[ni];
        if (nd.cfgs.size() < 2) continue;
        int best = 0;
        float best_ms = 3.0e38f;
        for (size_t c = 0; c < nd.cfgs.size() && result == MGI_OK; ++c) {
            nd.apply((int)c);
            bool usable = true;
            for (int r = 0; r <= reps && usable && result == MGI_OK; ++r) {
                // the whole plan runs, so that the node meets its input as it
                // does in a run (just written by its producer), and only the
                // node's kernels are timestamped
                for (size_t j = 0; j < p->nodes.size(); ++j) {
                    ev.start = j == ni ? evs[2 * r] : nullptr;
                    ev.stop = j == ni ? evs[2 * r + 1] : nullptr;
                    e = launch_node(*p, p->nodes[j], B, st);
                    ev.start = ev.stop = nullptr;
                    if (e == hipSuccess) continue;
                    if (j != ni) result = hip_fail(e, "mgi_plan_autotune: run");
                    else usable = false;   // configuration not launchable for this shape
                    e = hipSuccess;
                    break;
                }
            }
            if (result != MGI_OK) break;
            // drain what was queued (also after an unusable configuration)
            e = hipStreamSynchronize(st);
            if (e != hipSuccess) {
                result = hip_fail(e, "mgi_plan_autotune: run");
                break;
            }
            if (!usable) continue;
            times.clear();
            for (int r = 1; r <= reps && e == hipSuccess; ++r) {
                float ms = 0.0f;
                e = hipEventElapsedTime(&ms, evs[2 * r], evs[2 * r + 1]);
                times.push_back(ms);
            }
            if (e != hipSuccess) {
                result = hip_fail(e, "mgi_plan_autotune: timing");
                break;
            }
            // median of the runs after the first (which meets cold caches);
            // a later candidate must be more than 2% faster to replace an
            // earlier one, so that run-to-run noise does not flip the choice
            // (candidates are listed fused forms first, the split form of a
            // fused node, which moves more bytes, last)
            std::sort(times.begin(), times.end());
            const float med = times[times.size() / 2];
            if (med < best_ms * 0.98f) {
                best_ms = med;
                best = (int)c;
            }
        }
        nd.apply(best);
    }
    destroy();
    return result;
    MGI_ABI_CATCH("mgi_plan_autotune")
}

extern "C" mgi_status mgi_plan_node_config(const mgi_plan *p, int i, int *config, int *n_configs,
                                           const char **name) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_node_config: null plan");
    if (i < 0 || i >= (int)p->nodes.size())
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_node_config: node index out of range");
    const Node &nd = p->nodes[i];
    if (config) *config = nd.cfgs.empty() ? 0 : nd.cfg;
    if (n_configs) *n_configs = nd.cfgs.empty() ? 1 : (int)nd.cfgs.size();
    if (name) *name = nd.cfgs.empty() ? nd.kname : nd.cfgs[nd.cfg].name.c_str();
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_node_config")
}

extern "C" mgi_status mgi_plan_set_node_config(mgi_plan *p, int i, int config) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_set_node_config: null plan");
    if (i < 0 || i >= (int)p->nodes.size())
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_set_node_config: node index out of range");
    Node &nd = p->nodes[i];
    const int n = nd.cfgs.empty() ? 1 : (int)nd.cfgs.size();
    if (config < 0 || config >= n)
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_set_node_config: configuration out of range");
    if (!nd.cfgs.empty()) nd.apply(config);
    release_graph(*p);
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_set_node_config")
}

extern "C" mgi_status mgi_plan_read_node(mgi_plan *p, int i, void *dev_dst, void *stream) {
    MGI_ABI_TRY
    if (!p || !dev_dst) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_read_node: null pointer");
    if (i < 0 || i >= (int)p->nodes.size())
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_read_node: node index out of range");
    if (!p->opt.materialize_all)
        return fail(MGI_ERR_STATE, "mgi_plan_read_node: plan was finalized without materialize_all");
    if (!p->bound || p->last_outputs.size() != p->output_bufs.size())
        return fail(MGI_ERR_STATE, "mgi_plan_read_node: no run has been enqueued");
    hipStream_t st = static_cast<hipStream_t>(stream);
    const Node &nd = p->nodes[i];
    const Buf &b = p->bufs[nd.out];
    Bases B{static_cast<char *>(p->last_ws ? p->last_ws : p->dev_ws), nullptr, p->last_outputs.data()};
    if (b.loc == Loc::Input) return fail(MGI_ERR_STATE, "mgi_plan_read_node: input buffer");
    void *src = buf_ptr(*p, nd.out, B);
    hipError_t e;
    if (b.layout == Layout::C8) {
        e = launch_export((const h8 *)src, (float *)dev_dst, (int)b.shape.pixels(), b.shape.c,
                          p->opt.dtype == MGI_DTYPE_BF16, st);
    } else {
        e = hipMemcpyAsync(dev_dst, src, b.bytes, hipMemcpyDeviceToDevice, st);
    }
    if (e != hipSuccess) return hip_fail(e, "mgi_plan_read_node");
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_read_node")
}

extern "C" mgi_status mgi_plan_read_node_raw(mgi_plan *p, int i, void *dev_dst, size_t *bytes, void *stream) {
    MGI_ABI_TRY
    if (!p || !bytes) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_read_node_raw: null pointer");
    if (i < 0 || i >= (int)p->nodes.size())
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_read_node_raw: node index out of range");
    const Node &nd = p->nodes[i];
    const Buf &b = p->bufs[nd.out];
    if (b.layout != Layout::C8 || b.loc != Loc::Arena)
        return fail(MGI_ERR_UNSUPPORTED, "mgi_plan_read_node_raw: node output is not stored sliced");
    *bytes = b.bytes;
    if (!dev_dst) return MGI_OK;
    if (!p->opt.materialize_all)
        return fail(MGI_ERR_STATE, "mgi_plan_read_node_raw: plan was finalized without materialize_all");
    if (!p->bound || p->last_outputs.size() != p->output_bufs.size())
        return fail(MGI_ERR_STATE, "mgi_plan_read_node_raw: no run has been enqueued");
    const char *src = static_cast<const char *>(p->last_ws ? p->last_ws : p->dev_ws) + b.offset;
    hipError_t e = hipMemcpyAsync(dev_dst, src, b.bytes, hipMemcpyDeviceToDevice, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "mgi_plan_read_node_raw");
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_read_node_raw")
}

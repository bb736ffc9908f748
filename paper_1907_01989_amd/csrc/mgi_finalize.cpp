// Graph finalisation: fusion, node list, buffer planning, weight packing.
//
// Pure host code: no HIP call is made here, so every step runs and is tested
// on a machine without a GPU.
//
// Fusion (Sec. 3.2, first technique): an element-wise operator whose input is
// produced by an expensive operator, and used by nothing else, becomes part of
// that operator's epilogue:
//   conv / depthwise / fc / add  + activation       -> act1 (or act2 after a residual)
//   conv (any window)            + add(other)       -> residual epilogue, act2 = add's act
//   resize_bilinear              + argmax           -> one resize-argmax pass
// A fused node takes the place of the last operator it absorbed, so every
// operand it reads has been produced by then.
//
// Kernel specialisation (Sec. 3.2, fourth technique): a 1x1 stride-1
// convolution runs the plain pointwise GEMM; other windows run the same GEMM
// with an implicit-im2col loader; a convolution that reads a graph input with
// a small window (kh*kw*cin <= 32, the network stem) reads the NHWC input
// directly and needs no layout conversion (Sec. 3.2, input conversion to the
// sliced layout is skipped).
#include <algorithm>
#include <cstring>
#include <new>

#include "kernels.h"
#include "mgi_internal.h"

namespace mgi {

void stemdw_shape(const mgi_plan &p, const Node &nd, kern::StemDwParams &q) {
    const Shape x = p.bufs[nd.in[0]].shape;
    const mgi_conv_desc &c = nd.conv, &d = nd.dw_conv;
    q.N = x.n; q.H = x.h; q.W = x.w; q.C = x.c;
    q.SH = nd.dw_in.h; q.SW = nd.dw_in.w;
    q.KH = c.kh; q.KW = c.kw; q.K = c.kh * c.kw * x.c;
    q.sh = c.stride_h; q.sw = c.stride_w; q.dh = c.dil_h; q.dw = c.dil_w;
    q.pt = c.pad_t; q.pl = c.pad_l;
    q.nb16 = nd.nb16; q.act1 = nd.act1;
    q.OH = nd.dw_out.h; q.OW = nd.dw_out.w; q.S = d.stride_h;
    q.dpt = d.pad_t; q.dpl = d.pad_l;
    q.ns = (nd.dw_out.c + 7) / 8; q.act2 = nd.dw_act;
    q.fp16_in = p.bufs[nd.in[0]].in_dtype == MGI_DTYPE_FP16;
}

namespace {

inline int slices(int c) { return (c + 7) / 8; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

uint16_t f32_to_f16_bits(float f) {
    _Float16 h = (_Float16)f;  // round to nearest even
    uint16_t b;
    std::memcpy(&b, &h, 2);
    return b;
}

// bf16: the upper half of the fp32 pattern, rounded to nearest even (NaN
// kept quiet)
uint16_t f32_to_bf16_bits(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

struct Group {
    int head = -1;          // heavy op
    int last = -1;          // last absorbed op (position and output tensor)
    int n = 1;
    int act1 = MGI_ACT_NONE, act2 = MGI_ACT_NONE;
    int residual_tensor = -1;
    bool resize_argmax = false;
};

// Choose the GEMM tile for an (M x cout x K) problem: the largest tile that
// still gives two workgroups per compute unit (256 CUs), else the smallest.
GemmTile pick_tile(size_t M, int cout) {
    GemmTile t;
    int npad = ((cout + 15) / 16) * 16;
    t.bn = npad <= 32 ? 32 : (npad <= 64 ? 64 : 128);
    size_t ntiles = (npad + t.bn - 1) / t.bn;
    const int bms[3] = {128, 64, 32};
    t.bm = 32;
    for (int bm : bms) {
        size_t tiles = ((M + bm - 1) / bm) * ntiles;
        if (tiles >= 512) { t.bm = bm; break; }
    }
    return t;
}

// Pipelined pointwise kernel (K >= 64, at least 64 output channels): a
// 128 x 128 tile when there are at least 512 channels, else 128 x 64, as long
// as that still gives 384 workgroups (1.5 per CU); otherwise the shape with
// the most workgroups.  Measured on the MobileNet shapes: 128-channel tiles
// pay off only when many channels share one activation read.
// Candidate kernel configurations of a node for the autotuner; the first is
// the configuration finalize picked.  Every candidate accumulates each output
// in the same order (K ascending in steps of 32 for the GEMMs, taps in window
// order for depthwise), so they differ in speed only.
std::string tile_name(const GemmTile &t) {
    if (t.pipe) return "pipe" + std::to_string(t.bm) + "x" + std::to_string(t.bn) + (t.ks == 8 ? "k8" : "");
    if (t.slab)
        return "slab" + std::to_string(4 * t.wm) + "x" + std::to_string(t.bn) + "p" + std::to_string(t.pf);
    return "lds" + std::to_string(t.bm) + "x" + std::to_string(t.bn);
}

void pick_pipe_tile(GemmTile &t, size_t M, int npad);

// Candidate tiles of a pointwise or implicit-GEMM node: the finalize-time
// tile first, then pipelined, two-K-step and weight-slab tiles that fit.
void add_gemm_configs(Node &nd, size_t M) {
    auto push = [&](const GemmTile &t) {
        for (const Node::Config &c : nd.cfgs)
            if (c.tile.pipe == t.pipe && c.tile.slab == t.slab && (t.slab || c.tile.bm == t.bm) &&
                c.tile.ks == t.ks && c.tile.bn == t.bn && c.tile.wm == t.wm && c.tile.pf == t.pf)
                return;
        nd.cfgs.push_back({t, 0, tile_name(t)});
    };
    push(nd.tile);
    const int npad = nd.nb16 * 16;
    if (!nd.taps) {
        const int pipes[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
        for (auto &pb : pipes) {
            if (pb[1] > 64 && npad <= 64) continue;
            GemmTile t;
            t.pipe = true;
            t.bm = pb[0];
            t.bn = pb[1];
            push(t);
        }
        if (nd.ksp % 8 == 0) {            // two K-steps per ring stage
            GemmTile t;
            t.pipe = true;
            t.ks = 8;
            push(t);
        }
        const int slabs[5][2] = {{32, 32}, {16, 32}, {32, 64}, {16, 64}, {16, 16}};
        for (auto &sb : slabs) {
            if (sb[1] > 32 && npad <= 32) continue;
            const size_t lds = kern::gemm_xs_lds_bytes(nd.ksp, sb[0], sb[1]);
            // where the grid is less than one workgroup per compute unit (a
            // batch of one; v2's 7x7 projections at batch 64), activations 8
            // K-steps ahead (the K loop waits on memory latency) and slabs up
            // to the whole LDS (one workgroup per compute unit costs nothing
            // there)
            const size_t tiles = (M + 4 * sb[0] - 1) / (4 * sb[0]) * (size_t)((npad + sb[1] - 1) / sb[1]);
            const bool few = nd.ksp >= 32 && tiles < 256;
            if (lds > (few ? 160 * 1024 : 65536) || (sb[1] == 16 && !few)) continue;   // 16 channels: p8 only
            GemmTile t;
            t.slab = true;
            t.wm = sb[0];
            t.bn = sb[1];
            if (lds <= 65536 && sb[1] > 16) {
                t.pf = nd.ksp >= 8 ? 2 : 1;
                push(t);
            }
            if (few) {
                t.pf = 8;
                push(t);
            }
        }
    }
    const int ldss[5][2] = {{128, 128}, {64, 128}, {32, 128}, {64, 64}, {128, 64}};
    for (auto &lb : ldss) {
        if (lb[1] > 64 && npad <= 64) continue;
        GemmTile t;
        t.bm = lb[0];
        t.bn = lb[1];
        push(t);
    }
}

void add_pwdw_configs(Node &nd) {
    // channels per workgroup of the fused pointwise + depthwise kernel, and
    // the two separate kernels through the scratch tensor (pipelined GEMM
    // tile by the pointwise rule, depthwise rows by the depthwise rule);
    // the split form first when the fused kernel would not fill the GPU
    const Shape &s = nd.dw_in;
    const int nf = kern::pwdw_configs(s.n, s.h, s.w, nd.dw_out.h, nd.dw_out.w, nd.dw_conv.stride_h,
                                      nd.dw_conv.pad_t, nd.dw_conv.pad_l, nd.ksp, nd.nb16, -1, nullptr, nullptr);
    for (int c = 0; c < nf; ++c) {
        const char *name = "";
        kern::pwdw_configs(s.n, s.h, s.w, nd.dw_out.h, nd.dw_out.w, nd.dw_conv.stride_h, nd.dw_conv.pad_t,
                           nd.dw_conv.pad_l, nd.ksp, nd.nb16, c, nullptr, &name);
        Node::Config fc{GemmTile{}, 0, name, false, c};
        nd.cfgs.push_back(fc);
    }
    GemmTile t;
    pick_pipe_tile(t, nd.dw_in.pixels(), nd.nb16 * 16);
    const int dwr = nd.dw_conv.stride_h == 1 ? 4 : 2;
    const Node::Config split{t, dwr, "split_" + tile_name(t), true, 0};
    nd.cfgs.insert(nd.fused_default ? nd.cfgs.end() : nd.cfgs.begin(), Node::Config(split));
    if (nd.ksp % 8 == 0) {                // the GEMM with two K-steps per ring stage
        GemmTile t8;
        t8.pipe = true;
        t8.ks = 8;
        nd.cfgs.push_back(Node::Config{t8, dwr, "split_" + tile_name(t8), true, 0});
    }
    nd.apply(0);
}

void add_irb_configs(Node &nd) {
    // the block kernel's configurations; the fused pointwise -> depthwise
    // kernel's configurations, each followed by the projection GEMM; the
    // three separate kernels.  The block kernel first when it fills the
    // GPU, else the form the pointwise -> depthwise node would have taken.
    // The projection GEMM of the split forms: the weight-slab tile for at
    // most 32 output channels (it streams the wide input once), else the
    // pipelined tile by the pointwise rule.
    const Shape &s = nd.dw_in, &d = nd.dw_out;
    {
        const int npad = nd.pj_nb16 * 16;
        const size_t slab_lds = (size_t)2 * nd.pj_ksp * 256 + (size_t)4 * 2 * 2 * 1024;
        GemmTile t;
        if (npad <= 32 && slab_lds <= 65536) {
            t.slab = true;
            t.wm = 32;
            t.bn = 32;
            t.pf = nd.pj_ksp >= 8 ? 2 : 1;
        } else if (npad >= 64) {
            pick_pipe_tile(t, d.pixels(), npad);
        } else {
            t = pick_tile(d.pixels(), npad);
        }
        nd.pj_tile = t;
    }
    const int st = nd.dw_conv.stride_h, pt = nd.dw_conv.pad_t, pl = nd.dw_conv.pad_l;
    std::vector<Node::Config> blk, two, three;
    const int nb = kern::irb_configs(s.n, s.h, s.w, d.h, d.w, st, pt, pl, nd.ksp, nd.nb16, nd.pj_nb16, -1,
                                     nullptr, nullptr);
    for (int c = 0; c < nb; ++c) {
        const char *name = "";
        kern::irb_configs(s.n, s.h, s.w, d.h, d.w, st, pt, pl, nd.ksp, nd.nb16, nd.pj_nb16, c, &name, nullptr);
        blk.push_back(Node::Config{GemmTile{}, 0, name, false, c, 0});
    }
    const int nf = kern::pwdw_configs(s.n, s.h, s.w, d.h, d.w, st, pt, pl, nd.ksp, nd.nb16, -1, nullptr, nullptr);
    for (int c = 0; c < nf; ++c) {
        const char *name = "";
        kern::pwdw_configs(s.n, s.h, s.w, d.h, d.w, st, pt, pl, nd.ksp, nd.nb16, c, nullptr, &name);
        two.push_back(Node::Config{GemmTile{}, 0, std::string(name) + "+" + tile_name(nd.pj_tile), true, c, 1});
    }
    GemmTile t;
    pick_pipe_tile(t, s.pixels(), nd.nb16 * 16);
    three.push_back(Node::Config{t, st == 1 ? 4 : 2, "split3_" + tile_name(t), true, 0, 2});
    std::vector<Node::Config> order;
    auto add = [&](const std::vector<Node::Config> &v) { order.insert(order.end(), v.begin(), v.end()); };
    if (nd.irb_default) {
        add(blk); add(two); add(three);
    } else if (nd.fused_default) {
        add(two); add(blk); add(three);
    } else {
        add(three); add(two); add(blk);
    }
    nd.cfgs = order;
    nd.apply(0);
}

void add_stemdw_configs(const mgi_plan &p, Node &nd) {
    // band heights of the fused stem + depthwise kernel, and the two
    // separate kernels through the scratch tensor (first when the fused
    // kernel would not fill the GPU)
    kern::StemDwParams q{};
    stemdw_shape(p, nd, q);
    const int nf = kern::stemdw_configs(q, -1, nullptr, nullptr);
    for (int c = 0; c < nf; ++c) {
        const char *name = "";
        kern::stemdw_configs(q, c, nullptr, &name);
        nd.cfgs.push_back(Node::Config{GemmTile{}, 0, name, false, c});
    }
    const Node::Config split{GemmTile{}, 4, "split", true, 0};
    nd.cfgs.insert(nd.fused_default ? nd.cfgs.end() : nd.cfgs.begin(), Node::Config(split));
    nd.apply(0);
}

void add_fc_configs(Node &nd, size_t M) {
    // images per workgroup (16 * fm) and K-steps per load batch; 16 images
    // and 8 steps first (the most workgroups, one load latency per wave:
    // fastest on v1 b64, 5.6 us against 8.2 us for 64 images and 4 steps)
    const int fm0 = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
    const int opts[6][2] = {{1, 8}, {2, 8}, {4, 8}, {1, 4}, {2, 4}, {4, 4}};
    for (auto &o : opts) {
        if (o[0] > fm0) continue;
        bool dup = false;
        for (const Node::Config &c : nd.cfgs) dup = dup || (c.tile.wm == o[0] && c.tile.pf == o[1]);
        if (dup) continue;
        GemmTile t;
        t.wm = o[0];
        t.pf = o[1];
        nd.cfgs.push_back({t, 0, "fc" + std::to_string(16 * o[0]) + "k" + std::to_string(o[1])});
    }
    if (nd.kind == NodeKind::FcSoftmax) {
        // FC into the logits, then the softmax kernel: first when there
        // is more than one tile of 16 rows (each arriving workgroup's L2
        // write-back costs more than the softmax launch it saves once
        // the grid has a few hundred workgroups: 16.1 us fused against
        // 10.6 us split for 64 rows of 1000 classes, 7.2 against 9.6 us
        // for one row)
        Node::Config split = nd.cfgs[0];
        split.name = "split_" + split.name;
        split.split = true;
        nd.cfgs.insert(M > 16 ? nd.cfgs.begin() : nd.cfgs.end(), split);
    }
    nd.apply(0);
}

void add_pool_configs(Node &nd) {
    // tiles of the pooled GEMM (M-tiles of whole images), and the GEMM
    // then the pool kernel through the scratch tensor (first when the
    // fused kernel would not fill the GPU)
    const int hw = nd.dw_in.h * nd.dw_in.w, npad = nd.nb16 * 16;
    const int tiles[4][2] = {{128, 64}, {128, 128}, {64, 128}, {64, 64}};
    for (auto &tb : tiles) {
        if (hw > tb[0] || (tb[1] > 64 && npad <= 64)) continue;
        GemmTile t;
        t.pipe = true;
        t.bm = tb[0];
        t.bn = tb[1];
        nd.cfgs.push_back({t, 0, "pool" + std::to_string(tb[0]) + "x" + std::to_string(tb[1])});
    }
    if (nd.ksp % 8 == 0) {
        GemmTile t;
        t.pipe = true;
        t.ks = 8;
        nd.cfgs.push_back({t, 0, "pool64x64k8"});
    }
    // weight-slab tiles of one 64-row image group (planes of at most 64
    // pixels) for grids of few workgroups: the slab loads in one round and
    // the activations stream 8 K-steps ahead
    const size_t per = (size_t)std::max(1, 64 / hw), groups = ((size_t)nd.dw_in.n + per - 1) / per;
    for (int bn : {16, 32, 64}) {
        if (hw > 64) break;   // (a pooled node's planes have at most 64 pixels)
        const size_t lds = kern::gemm_xs_lds_bytes(nd.ksp, 16, bn);
        if (groups * (size_t)((npad + bn - 1) / bn) >= 128 || nd.ksp < 32 || lds > 160 * 1024) continue;
        GemmTile ts;
        ts.slab = true;
        ts.wm = 16;
        ts.bn = bn;
        ts.pf = 8;
        nd.cfgs.push_back({ts, 0, "poolslab64x" + std::to_string(bn) + "p8"});
    }
    GemmTile t;
    pick_pipe_tile(t, nd.dw_in.pixels(), npad);
    const Node::Config split{t, 0, "split_" + tile_name(t), true, 0};
    nd.cfgs.insert(nd.fused_default ? nd.cfgs.end() : nd.cfgs.begin(), Node::Config(split));
    nd.apply(0);
}

void add_dwpw_configs(Node &nd) {
    // band heights for the fused depthwise + pointwise kernel: up to 128
    // or up to 64 pixels per workgroup
    for (int px : {128, 64}) {
        GemmTile t;
        t.bm = px;
        nd.cfgs.push_back({t, 0, "band" + std::to_string(px)});
    }
}

// rows per thread of the 3x3 depthwise kernel (stride 1 or 2, dilation 1 or 2)
void add_depthwise_configs(Node &nd) {
    if (nd.conv.kh != 3 || nd.conv.kw != 3 || nd.conv.stride_h != nd.conv.stride_w ||
        nd.conv.dil_h != nd.conv.dil_w || nd.conv.stride_h > 2 || nd.conv.dil_h > 2)
        return;
    const int rows[2][3] = {{4, 2, 8}, {2, 1, 4}};
    for (int r : rows[nd.conv.stride_h - 1]) nd.cfgs.push_back({GemmTile{}, r, "rows" + std::to_string(r)});
    nd.dw_rows = nd.cfgs[0].dw_rows;
}

// the node's candidate configurations, in preference order (the first is
// the one a plan runs before any autotuning)
void add_configs(const mgi_plan &p, Node &nd, size_t M) {
    switch (nd.kind) {
        case NodeKind::Gemm: add_gemm_configs(nd, M); break;
        case NodeKind::PwDw: add_pwdw_configs(nd); break;
        case NodeKind::Irb: add_irb_configs(nd); break;
        case NodeKind::StemDw: add_stemdw_configs(p, nd); break;
        case NodeKind::FC:
        case NodeKind::FcSoftmax: add_fc_configs(nd, M); break;
        case NodeKind::GemmPool: add_pool_configs(nd); break;
        case NodeKind::DwPw: add_dwpw_configs(nd); break;
        case NodeKind::Depthwise: add_depthwise_configs(nd); break;
        default: break;
    }
}

// Depthwise -> pointwise fusion (Sec. 3.2's fusion extended to the
// depthwise-separable pair): a 3x3 depthwise node (stride 1 or 2, dilation 1)
// whose output only feeds one pointwise GEMM with at most 320 output channels
// becomes part of that GEMM's node, when whole output rows tile the image
// (a band of rows of at most 128 pixels) into at least 256 workgroups; the
// intermediate buffer is dropped.
void fuse_dw_into_pw(mgi_plan &p) {
    std::vector<int> readers(p.bufs.size(), 0), producer(p.bufs.size(), -1);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &nd = p.nodes[i];
        for (int b : nd.in) readers[b]++;
        if (nd.residual >= 0) readers[nd.residual]++;
        producer[nd.out] = (int)i;
    }
    std::vector<char> drop(p.nodes.size(), 0);
    for (Node &pw : p.nodes) {
        if (pw.kind != NodeKind::Gemm || pw.taps || pw.in.empty()) continue;
        const int mid = pw.in[0];
        if (readers[mid] != 1 || p.bufs[mid].loc != Loc::Arena || producer[mid] < 0) continue;
        Node &dw = p.nodes[producer[mid]];
        const mgi_conv_desc &c = dw.conv;
        if (dw.kind != NodeKind::Depthwise || c.kh != 3 || c.kw != 3 || c.stride_h != c.stride_w ||
            c.stride_h > 2 || c.dil_h != 1 || c.dil_w != 1)
            continue;
        if (kern::dwpw_blocks(pw.nb16) == 0) continue;
        const Shape os = p.bufs[pw.out].shape;
        kern::DwPwTile t;
        if (!kern::dwpw_tile(os.h, os.w, c.stride_h, os.n, t) || (size_t)os.n * t.nbands < 256) continue;
        pw.kind = NodeKind::DwPw;
        pw.kname = "dw_pw";
        pw.dw_op = dw.op;
        pw.dw_conv = dw.conv;
        pw.dw_act = dw.act1;
        pw.in[0] = dw.in[0];
        pw.n_fused += dw.n_fused;
        pw.tile = GemmTile{};
        pw.tile.bm = 128;
        p.bufs[mid].dead = true;
        drop[producer[mid]] = 1;
    }
    std::vector<Node> kept;
    for (size_t i = 0; i < p.nodes.size(); ++i)
        if (!drop[i]) kept.push_back(std::move(p.nodes[i]));
    p.nodes.swap(kept);
}

// Pointwise -> depthwise fusion (Sec. 3.2's fusion of a cheap operator into
// the expensive one, extended to the pair inside a MobileNet stage): a 1x1
// pointwise GEMM node without residual whose output only feeds one 3x3
// depthwise node (dilation 1, stride 1 or 2) becomes a single node producing
// the depthwise output, when the planes fit the fused kernel's whole-image
// tiles or bands (pwdw_configs).  The intermediate tensor stays planned as the
// node's scratch, so the node can also run as the two separate kernels; the
// fused kernel is its default configuration when it gets at least 128
// workgroups (or `always`): with fewer, the separate kernels, which split
// the work finer, finish first.
void fuse_pw_into_dw(mgi_plan &p, bool always) {
    std::vector<int> readers(p.bufs.size(), 0), producer(p.bufs.size(), -1);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &nd = p.nodes[i];
        for (int b : nd.in) readers[b]++;
        if (nd.residual >= 0) readers[nd.residual]++;
        producer[nd.out] = (int)i;
    }
    std::vector<char> drop(p.nodes.size(), 0);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &dw = p.nodes[i];
        const mgi_conv_desc &c = dw.conv;
        if (dw.kind != NodeKind::Depthwise || dw.in.size() != 1 || c.kh != 3 || c.kw != 3 ||
            c.stride_h != c.stride_w || c.stride_h > 2 || c.dil_h != 1 || c.dil_w != 1)
            continue;
        const int mid = dw.in[0];
        if (readers[mid] != 1 || p.bufs[mid].loc != Loc::Arena || producer[mid] < 0) continue;
        Node &pw = p.nodes[producer[mid]];
        if (pw.kind != NodeKind::Gemm || pw.taps || pw.residual >= 0 || pw.in.size() != 1) continue;
        const Shape in = p.bufs[mid].shape, out = p.bufs[dw.out].shape;
        kern::PwDwGeom geo{};
        if (kern::pwdw_configs(in.n, in.h, in.w, out.h, out.w, c.stride_h, c.pad_t, c.pad_l, pw.ksp, pw.nb16, 0, &geo,
                               nullptr) == 0)
            continue;
        pw.fused_default = always || (size_t)geo.groups * ((pw.nb16 + geo.nbt - 1) / geo.nbt) >= 128;
        pw.kind = NodeKind::PwDw;
        pw.kname = "pw_dw";
        pw.dw_op = dw.op;
        pw.dw_conv = dw.conv;
        pw.dw_act = dw.act1;
        pw.dw_in = in;
        pw.dw_out = out;
        pw.out = dw.out;
        pw.out_tensor = dw.out_tensor;
        pw.n_fused += dw.n_fused;
        pw.tile = GemmTile{};
        pw.scratch = mid;
        drop[i] = 1;
    }
    std::vector<Node> kept;
    for (size_t i = 0; i < p.nodes.size(); ++i)
        if (!drop[i]) kept.push_back(std::move(p.nodes[i]));
    p.nodes.swap(kept);
}

// Projection fusion (MobileNet-v2's inverted residual block as one node): a
// 1x1 stride-1 GEMM node that alone reads the output of a fused pointwise ->
// depthwise node joins it, when its residual (if any) is produced before that
// node, it has at most 320 output channels and the block kernel (irb.hip)
// covers the shapes.  The depthwise output stays planned as the node's second
// scratch tensor, so the node can also run as the fused pointwise ->
// depthwise kernel plus the projection GEMM, or as three kernels; the block
// kernel is the default configuration when it gets at least 256 workgroups
// (or `always`).
void fuse_proj_into_pwdw(mgi_plan &p, bool always) {
    std::vector<int> readers(p.bufs.size(), 0), producer(p.bufs.size(), -1), reader(p.bufs.size(), -1);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &nd = p.nodes[i];
        for (int b : nd.in) {
            readers[b]++;
            reader[b] = (int)i;
        }
        if (nd.residual >= 0) readers[nd.residual]++;
        producer[nd.out] = (int)i;
    }
    std::vector<char> drop(p.nodes.size(), 0);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        Node &b = p.nodes[i];
        if (b.kind != NodeKind::PwDw) continue;
        const int mid = b.out;
        if (readers[mid] != 1 || p.bufs[mid].loc != Loc::Arena || reader[mid] < 0) continue;
        const Node &pj = p.nodes[reader[mid]];
        const mgi_conv_desc &c = pj.conv;
        if (pj.kind != NodeKind::Gemm || pj.taps || pj.in.size() != 1 || c.kh != 1 || c.kw != 1 || c.stride_h != 1 ||
            c.stride_w != 1 || pj.nb16 > 20)
            continue;
        if (pj.residual >= 0 && producer[pj.residual] >= (int)i) continue;
        const Shape &s = b.dw_in, &d = b.dw_out;
        if (pj.ksl != (d.c + 7) / 8) continue;
        int groups = 0;
        if (kern::irb_configs(s.n, s.h, s.w, d.h, d.w, b.dw_conv.stride_h, b.dw_conv.pad_t, b.dw_conv.pad_l, b.ksp,
                              b.nb16, pj.nb16, 0, nullptr, &groups) == 0)
            continue;
        b.irb_default = always || groups >= 256;
        b.kind = NodeKind::Irb;
        b.kname = "irb";
        b.pj_op = pj.op;
        b.pj_ksl = pj.ksl;
        b.pj_ksp = pj.ksp;
        b.pj_nb16 = pj.nb16;
        b.pj_act1 = pj.act1;
        b.pj_act2 = pj.act2;
        b.residual = pj.residual;
        b.scratch2 = mid;
        b.out = pj.out;
        b.out_tensor = pj.out_tensor;
        b.n_fused += pj.n_fused;
        drop[reader[mid]] = 1;
    }
    std::vector<Node> kept;
    for (size_t i = 0; i < p.nodes.size(); ++i)
        if (!drop[i]) kept.push_back(std::move(p.nodes[i]));
    p.nodes.swap(kept);
}

// The stem and a 3x3 depthwise convolution at stride 1 that alone reads its
// output become one node (kernel in stemdw.hip), the same pattern as above
// for the network's first layer pair; the stem output stays a planned scratch
// tensor for the split configuration.
void fuse_stem_into_dw(mgi_plan &p, bool always) {
    std::vector<int> readers(p.bufs.size(), 0), producer(p.bufs.size(), -1);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &nd = p.nodes[i];
        for (int b : nd.in) readers[b]++;
        if (nd.residual >= 0) readers[nd.residual]++;
        producer[nd.out] = (int)i;
    }
    std::vector<char> drop(p.nodes.size(), 0);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &dw = p.nodes[i];
        const mgi_conv_desc &c = dw.conv;
        if (dw.kind != NodeKind::Depthwise || dw.in.size() != 1 || c.kh != 3 || c.kw != 3 ||
            c.stride_h != 1 || c.stride_w != 1 || c.dil_h != 1 || c.dil_w != 1)
            continue;
        const int mid = dw.in[0];
        if (readers[mid] != 1 || p.bufs[mid].loc != Loc::Arena || producer[mid] < 0) continue;
        Node &sn = p.nodes[producer[mid]];
        if (sn.kind != NodeKind::Stem || sn.residual >= 0 || sn.in.size() != 1) continue;
        Node t = sn;
        t.kind = NodeKind::StemDw;
        t.dw_conv = dw.conv;
        t.dw_act = dw.act1;
        t.dw_in = p.bufs[mid].shape;
        t.dw_out = p.bufs[dw.out].shape;
        kern::StemDwParams q{};
        stemdw_shape(p, t, q);
        kern::StemDwGeom geo{};
        if (kern::stemdw_configs(q, 0, &geo, nullptr) == 0) continue;
        t.fused_default = always || (size_t)q.N * geo.nbands >= 128;
        t.kname = "stem_dw";
        t.dw_op = dw.op;
        t.out = dw.out;
        t.out_tensor = dw.out_tensor;
        t.n_fused += dw.n_fused;
        t.scratch = mid;
        sn = std::move(t);
        drop[i] = 1;
    }
    std::vector<Node> kept;
    for (size_t i = 0; i < p.nodes.size(); ++i)
        if (!drop[i]) kept.push_back(std::move(p.nodes[i]));
    p.nodes.swap(kept);
}

// A pointwise GEMM whose output only a global average pool reads (planes of
// at most 64 pixels) becomes one node (GemmPool): the pooled GEMM kernel
// (gemm.hip, pool_epilogue) writes the means directly; the GEMM output stays
// a planned scratch tensor for the split configuration (GEMM, then pool).
void fuse_pool_into_pw(mgi_plan &p, bool always) {
    std::vector<int> readers(p.bufs.size(), 0), producer(p.bufs.size(), -1);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &nd = p.nodes[i];
        for (int b : nd.in) readers[b]++;
        if (nd.residual >= 0) readers[nd.residual]++;
        producer[nd.out] = (int)i;
    }
    std::vector<char> drop(p.nodes.size(), 0);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &gp = p.nodes[i];
        if (gp.kind != NodeKind::Gap || gp.in.size() != 1) continue;
        const int mid = gp.in[0];
        if (readers[mid] != 1 || p.bufs[mid].loc != Loc::Arena || producer[mid] < 0) continue;
        Node &pw = p.nodes[producer[mid]];
        if (pw.kind != NodeKind::Gemm || pw.taps || pw.residual >= 0 || pw.in.size() != 1 ||
            pw.act2 != MGI_ACT_NONE || gp.act1 != MGI_ACT_NONE)
            continue;
        const Shape in = p.bufs[mid].shape;
        if (in.h * in.w > 64 || pw.ksp % 4 != 0) continue;
        const int hw = in.h * in.w, ipt = 128 / hw;
        pw.fused_default = always || (size_t)((in.n + ipt - 1) / ipt) * ((pw.nb16 * 16 + 63) / 64) >= 128;
        pw.kind = NodeKind::GemmPool;
        pw.kname = "pw_pool";
        pw.dw_in = in;
        pw.dw_out = p.bufs[gp.out].shape;
        pw.out = gp.out;
        pw.out_tensor = gp.out_tensor;
        pw.n_fused += gp.n_fused;
        pw.tile = GemmTile{};
        pw.scratch = mid;
        drop[i] = 1;
    }
    std::vector<Node> kept;
    for (size_t i = 0; i < p.nodes.size(); ++i)
        if (!drop[i]) kept.push_back(std::move(p.nodes[i]));
    p.nodes.swap(kept);
}

// FC -> softmax fusion: a softmax whose input is the logits of an FC node and
// nothing else reads them joins that node; the FC kernel's workgroups count
// themselves in per row tile and the last one runs the tile's softmax.  The
// logits stay planned as the node's scratch (written, then read by the last
// workgroup; the split form runs the softmax kernel over them), or stay in
// the caller's buffer when they are a graph output themselves.
void fuse_softmax_into_fc(mgi_plan &p) {
    std::vector<int> readers(p.bufs.size(), 0), producer(p.bufs.size(), -1);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &nd = p.nodes[i];
        for (int b : nd.in) readers[b]++;
        if (nd.residual >= 0) readers[nd.residual]++;
        producer[nd.out] = (int)i;
    }
    std::vector<char> drop(p.nodes.size(), 0);
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        const Node &sm = p.nodes[i];
        if (sm.kind != NodeKind::Softmax || sm.in.size() != 1) continue;
        const int mid = sm.in[0];
        const Loc loc = p.bufs[mid].loc;
        if (readers[mid] != 1 || (loc != Loc::Arena && loc != Loc::Output) || producer[mid] < 0) continue;
        Node &fc = p.nodes[producer[mid]];
        if (fc.kind != NodeKind::FC) continue;
        fc.kind = NodeKind::FcSoftmax;
        fc.kname = "fc_softmax";
        fc.out = sm.out;
        fc.out_tensor = sm.out_tensor;
        fc.n_fused += sm.n_fused;
        fc.scratch = mid;
        drop[i] = 1;
    }
    std::vector<Node> kept;
    for (size_t i = 0; i < p.nodes.size(); ++i)
        if (!drop[i]) kept.push_back(std::move(p.nodes[i]));
    p.nodes.swap(kept);
}

void pick_pipe_tile(GemmTile &t, size_t M, int npad) {
    const int cand[3][2] = {{128, 128}, {128, 64}, {64, 64}};
    size_t best_tiles = 0;
    int best = 2;
    for (int c = 0; c < 3; ++c) {
        const int bm = cand[c][0], bn = cand[c][1];
        if (bn == 128 && npad < 512) continue;
        const size_t tiles = ((M + bm - 1) / bm) * (size_t)((npad + bn - 1) / bn);
        if (tiles >= 384) { best = c; break; }
        if (tiles > best_tiles) { best_tiles = tiles; best = c; }
    }
    t.pipe = true;
    t.slab = false;
    t.bm = cand[best][0];
    t.bn = cand[best][1];
}

}  // namespace

namespace {

// Graph transformations before fusion (Sec. 3.1), on a copy of the graph:
//  - identity removal: an activation NONE, a one-input concatenation or a
//    resize to the input's own size forwards its input to its consumers.
//    Identities applied directly to a graph input are kept: they are where the
//    input is converted to the sliced layout;
//  - PAD merge: a zero PAD whose consumers are all convolutions (full or
//    depthwise) is folded into their padding: a convolution over a zero-padded
//    tensor equals the convolution with the pads added.
// Graph outputs are never rewritten away.  Tensor ids are unchanged; ops left
// without consumers are dropped afterwards as dead.
void clean_graph(mgi_graph &g) {
    const int nops = (int)g.ops.size();
    std::vector<char> is_output(nops, 0);
    for (int t : g.outputs) is_output[t] = 1;
    std::vector<int> alias(nops);
    for (int i = 0; i < nops; ++i) alias[i] = i;
    for (int i = 0; i < nops; ++i) {
        GOp &op = g.ops[i];
        for (int &t : op.in) t = alias[t];
        if (is_output[i] || op.in.empty() || g.ops[op.in[0]].kind == OpKind::Input) continue;
        const Shape &x = g.ops[op.in[0]].out;
        const bool identity =
            (op.kind == OpKind::Activation && op.act == MGI_ACT_NONE) ||
            (op.kind == OpKind::Concat && op.in.size() == 1) ||
            (op.kind == OpKind::ResizeBilinear && op.oh == x.h && op.ow == x.w) ||
            (op.kind == OpKind::Pad && op.pads[0] == 0 && op.pads[1] == 0 && op.pads[2] == 0 &&
             op.pads[3] == 0);
        if (identity) alias[i] = op.in[0];
    }
    std::vector<std::vector<int>> consumers(nops);
    for (int i = 0; i < nops; ++i)
        if (alias[i] == i)
            for (int t : g.ops[i].in) consumers[t].push_back(i);
    for (int i = 0; i < nops; ++i) {
        const GOp &pd = g.ops[i];
        if (pd.kind != OpKind::Pad || alias[i] != i || is_output[i] || consumers[i].empty()) continue;
        bool all_conv = true;
        for (int c : consumers[i]) {
            const OpKind k = g.ops[c].kind;
            all_conv = all_conv && (k == OpKind::Conv2d || k == OpKind::Depthwise);
        }
        if (!all_conv) continue;
        for (int c : consumers[i]) {
            GOp &cv = g.ops[c];
            cv.conv.pad_t += pd.pads[0];
            cv.conv.pad_b += pd.pads[1];
            cv.conv.pad_l += pd.pads[2];
            cv.conv.pad_r += pd.pads[3];
            cv.in[0] = pd.in[0];
        }
    }
}

// Ops that some graph output depends on; graph inputs are always kept.
std::vector<char> live_ops(const mgi_graph &g) {
    std::vector<char> live(g.ops.size(), 0);
    std::vector<int> stack(g.outputs.begin(), g.outputs.end());
    while (!stack.empty()) {
        const int t = stack.back();
        stack.pop_back();
        if (live[t]) continue;
        live[t] = 1;
        for (int u : g.ops[t].in) stack.push_back(u);
    }
    for (int t : g.inputs) live[t] = 1;
    return live;
}


mgi_status build_plan_impl(const mgi_graph &g, const mgi_options &o, mgi_plan &p);

}  // namespace

mgi_status build_plan(const mgi_graph &g, const mgi_options &o, mgi_plan &p) {
    if (g.outputs.empty()) return fail(MGI_ERR_STATE, "mgi_graph_finalize: no output marked");
    if (!o.fuse) return build_plan_impl(g, o, p);
    mgi_graph gc = g;
    clean_graph(gc);
    return build_plan_impl(gc, o, p);
}

namespace {

mgi_status check_options(const mgi_options &o) {
    if (o.planner != MGI_PLANNER_NAIVE && o.planner != MGI_PLANNER_GREEDY && o.planner != MGI_PLANNER_MCFP)
        return fail(MGI_ERR_UNSUPPORTED, "mgi_graph_finalize: unknown planner");
    if (o.dtype != MGI_DTYPE_FP16 && o.dtype != MGI_DTYPE_BF16)
        return fail(MGI_ERR_UNSUPPORTED, "mgi_graph_finalize: storage is fp16 or bf16");
    if (o.fuse_pwdw < 0 || o.fuse_pwdw > 2)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_finalize: fuse_pwdw is 0, 1 or 2");
    if (o.fuse_stemdw < 0 || o.fuse_stemdw > 2)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_finalize: fuse_stemdw is 0, 1 or 2");
    if (o.fuse_pool < 0 || o.fuse_pool > 2)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_finalize: fuse_pool is 0, 1 or 2");
    if (o.fuse_softmax < 0 || o.fuse_softmax > 1)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_finalize: fuse_softmax is 0 or 1");
    if (o.fuse_irb < 0 || o.fuse_irb > 2)
        return fail(MGI_ERR_INVALID_ARG, "mgi_graph_finalize: fuse_irb is 0, 1 or 2");
    return MGI_OK;
}

// Element-wise operator fusion (Sec. 3.2): an activation or an add whose
// operand is the private output of a convolution (or of another fusible
// group), and an argmax of a resize, join that group; every other live
// operator starts its own.  Groups come back in execution order (the
// position of the last absorbed operator).
std::vector<Group> group_operators(const mgi_graph &g, const mgi_options &o, const std::vector<char> &live) {
    const int nops = (int)g.ops.size();
    std::vector<char> is_output(nops, 0);
    for (int t : g.outputs) is_output[t] = 1;
    std::vector<std::vector<int>> consumers(nops);
    for (int i = 0; i < nops; ++i)
        if (live[i])
            for (int t : g.ops[i].in) consumers[t].push_back(i);
    std::vector<int> group_of(nops, -1);
    std::vector<Group> groups;
    auto single_private_use = [&](int t) {
        return consumers[t].size() == 1 && !is_output[t];
    };
    for (int i = 0; i < nops; ++i) {
        const GOp &op = g.ops[i];
        if (op.kind == OpKind::Input || !live[i]) continue;
        if (o.fuse && op.kind == OpKind::Activation) {
            int t = op.in[0];
            int gi = group_of[t];
            if (gi >= 0 && groups[gi].last == t && single_private_use(t)) {
                Group &G = groups[gi];
                OpKind hk = g.ops[G.head].kind;
                bool ok_kind = hk == OpKind::Conv2d || hk == OpKind::Depthwise ||
                               hk == OpKind::FC || hk == OpKind::Add;
                int &slot = (G.residual_tensor >= 0) ? G.act2 : G.act1;
                if (ok_kind && !G.resize_argmax && slot == MGI_ACT_NONE) {
                    slot = op.act;
                    G.last = i;
                    G.n++;
                    group_of[i] = gi;
                    continue;
                }
            }
        }
        if (o.fuse && op.kind == OpKind::Add) {
            bool fused = false;
            for (int side = 0; side < 2 && !fused; ++side) {
                int t = op.in[side], other = op.in[1 - side];
                if (t == other) break;
                int gi = group_of[t];
                if (gi < 0 || groups[gi].last != t || !single_private_use(t)) continue;
                Group &G = groups[gi];
                if (g.ops[G.head].kind != OpKind::Conv2d || G.residual_tensor >= 0) continue;
                G.residual_tensor = other;
                G.act2 = op.act;
                G.last = i;
                G.n++;
                group_of[i] = gi;
                fused = true;
            }
            if (fused) continue;
        }
        if (o.fuse && op.kind == OpKind::Argmax) {
            int t = op.in[0];
            int gi = group_of[t];
            if (gi >= 0 && groups[gi].last == t && single_private_use(t) &&
                g.ops[groups[gi].head].kind == OpKind::ResizeBilinear && groups[gi].n == 1) {
                Group &G = groups[gi];
                G.resize_argmax = true;
                G.last = i;
                G.n++;
                group_of[i] = gi;
                continue;
            }
        }
        Group G;
        G.head = i;
        G.last = i;
        if (op.kind == OpKind::Conv2d || op.kind == OpKind::Depthwise || op.kind == OpKind::Add ||
            op.kind == OpKind::Activation)
            G.act1 = op.act;
        group_of[i] = (int)groups.size();
        groups.push_back(G);
    }
    std::stable_sort(groups.begin(), groups.end(), [](const Group &a, const Group &b) { return a.last < b.last; });
    return groups;
}


// Buffers and nodes for the operator groups: every graph input gets a buffer
// read in place, every group one node (lower), graph outputs an fp32 / int32
// buffer of the caller.
struct Lowering {
    const mgi_graph &g;
    mgi_plan &p;
    std::vector<int> c8_buf;     // graph tensor -> C8 (or other) buffer holding it
    std::vector<int> flat_buf;   // graph tensor -> F32 / I32 buffer
    std::vector<int> in_buf;     // graph input tensor -> NHWC_IN buffer
    std::vector<int> out_index;  // graph tensor -> graph output index

    Lowering(const mgi_graph &g_, mgi_plan &p_)
        : g(g_), p(p_), c8_buf(g_.ops.size(), -1), flat_buf(g_.ops.size(), -1), in_buf(g_.ops.size(), -1),
          out_index(g_.ops.size(), -1) {
        for (size_t k = 0; k < g.outputs.size(); ++k) out_index[g.outputs[k]] = (int)k;
    }
    void add_inputs();
    int new_buf(Layout L, const Shape &s, int tensor);
    int add_node(Node &&nd) {
        p.nodes.push_back(std::move(nd));
        return (int)p.nodes.size() - 1;
    }
    int need_c8(int t);
    mgi_status lower_conv(const Group &G, const GOp &op, const Shape &out_shape, Node &nd);
    mgi_status lower_other(const Group &G, const GOp &op, const Shape &out_shape, Node &nd);
    mgi_status lower(const Group &G);
    mgi_status bind_outputs();
};

void Lowering::add_inputs() {
    p.input_bufs.clear();
    p.input_shapes.clear();
    p.input_dtypes.clear();
    for (size_t k = 0; k < g.inputs.size(); ++k) {
        int t = g.inputs[k];
        Buf b;
        b.layout = Layout::NHWC_IN;
        b.shape = g.ops[t].out;
        b.in_dtype = g.ops[t].in_dtype;
        b.bytes = b.shape.elems() * (b.in_dtype == MGI_DTYPE_FP16 ? 2 : 4);
        b.loc = Loc::Input;
        b.index = (int)k;
        b.graph_tensor = t;
        in_buf[t] = (int)p.bufs.size();
        p.input_bufs.push_back(in_buf[t]);
        p.input_shapes.push_back(b.shape);
        p.input_dtypes.push_back(b.in_dtype);
        p.bufs.push_back(b);
    }

}

int Lowering::new_buf(Layout L, const Shape &s, int tensor) {
    Buf b;
    b.layout = L;
    b.shape = s;
    if (L == Layout::C8) b.bytes = (size_t)slices(s.c) * 8 * s.pixels() * 2;
    else b.bytes = s.elems() * 4;
    b.graph_tensor = tensor;
    if (tensor >= 0 && out_index[tensor] >= 0 && L != Layout::C8) {
        b.loc = Loc::Output;
        b.index = out_index[tensor];
    }
    p.bufs.push_back(b);
    return (int)p.bufs.size() - 1;
}

// a C8 view of graph tensor t, converting a graph input on first use
int Lowering::need_c8(int t) {
    if (c8_buf[t] >= 0) return c8_buf[t];
    if (g.ops[t].kind == OpKind::Input) {
        Node nd;
        nd.kind = NodeKind::Ingest;
        nd.kname = "ingest";
        nd.op = t;
        nd.out_tensor = -1;
        nd.n_fused = 0;
        nd.in = {in_buf[t]};
        nd.out = new_buf(Layout::C8, g.ops[t].out, -1);
        const int ob = nd.out;
        add_node(std::move(nd));
        c8_buf[t] = ob;
        return ob;
    }
    return -1;
}

// A convolution group: the stem kernel when it reads a graph input through a
// window of at most 32 values, otherwise a GEMM (pointwise) or implicit GEMM
// over the sliced input, with the residual operand of a fused add.
mgi_status Lowering::lower_conv(const Group &G, const GOp &op, const Shape &out_shape, Node &nd) {
    const Shape x = g.ops[op.in[0]].out;
    const mgi_conv_desc &d = op.conv;
    nd.conv = d;
    const bool from_input = g.ops[op.in[0]].kind == OpKind::Input;
    // LDS for a one-row band of the stem kernel (graph inputs up to a few
    // thousand pixels wide); wider inputs take the sliced path
    const int ow = out_shape.w;
    const int rs = std::max(((ow - 1) * d.stride_w + (d.kw - 1) * d.dil_w + 1) * x.c,
                            (x.w + d.pad_l) * x.c);
    const size_t band1 = (size_t)((d.kh - 1) * d.dil_h + 1) * (rs + 7) * 2;
    if (from_input && d.kh * d.kw * x.c <= 32 && d.cout <= 64 && band1 + kern::kStemStageBytes <= 65536) {
        nd.kind = NodeKind::Stem;
        nd.kname = "conv_stem";
        nd.in = {in_buf[op.in[0]]};
        nd.ksl = 4;
        nd.ksp = 4;
    } else {
        int xb = need_c8(op.in[0]);
        if (xb < 0) return fail(MGI_ERR_UNSUPPORTED, "conv2d input has no sliced form");
        nd.kind = NodeKind::Gemm;
        nd.in = {xb};
        nd.taps = !(d.kh == 1 && d.kw == 1 && d.stride_h == 1 && d.stride_w == 1 &&
                    d.pad_t == 0 && d.pad_b == 0 && d.pad_l == 0 && d.pad_r == 0);
        nd.kname = nd.taps ? "conv_igemm" : "pw_gemm";
        nd.ksl = d.kh * d.kw * slices(x.c);
        nd.ksp = (nd.ksl + 3) / 4 * 4;
    }
    nd.nb16 = (d.cout + 15) / 16;
    nd.tile = pick_tile(out_shape.pixels(), d.cout);
    if (nd.kind == NodeKind::Gemm && !nd.taps && nd.ksl >= 8 && nd.nb16 * 16 >= 64) {
        pick_pipe_tile(nd.tile, out_shape.pixels(), nd.nb16 * 16);
    } else if (nd.kind == NodeKind::Gemm && !nd.taps) {
        // weight-slab kernel: 128 x 32 tiles, two K steps of
        // prefetch when there are at least two; the slab (32
        // channels x all K) plus the epilogue tiles fit 64 KiB
        // up to K = 768
        const size_t slab = (size_t)2 * nd.ksp * 256 + 16384;
        if (slab <= 65536) {
            nd.tile.slab = true;
            nd.tile.wm = 32;
            nd.tile.bn = 32;
            nd.tile.pf = nd.ksp >= 8 ? 2 : 1;
        }
    }
    if (G.residual_tensor >= 0) {
        int rb = need_c8(G.residual_tensor);
        if (rb < 0) rb = c8_buf[G.residual_tensor];
        if (rb < 0) return fail(MGI_ERR_UNSUPPORTED, "residual operand has no sliced form");
        nd.residual = rb;
    }
    nd.out = new_buf(Layout::C8, out_shape, G.last);
    c8_buf[G.last] = nd.out;
    return MGI_OK;
}

// One node for an operator group (Sec. 3.2: the element-wise operators a
// group absorbed run in the head operator's epilogue), plus an export node
// when the group's output is a graph output kept in sliced form.
// Groups headed by a fully-connected layer, softmax, concatenation, resize,
// argmax or padding.
mgi_status Lowering::lower_other(const Group &G, const GOp &op, const Shape &out_shape, Node &nd) {
    switch (op.kind) {
        case OpKind::FC: {
            int xb = need_c8(op.in[0]);
            if (xb < 0) xb = c8_buf[op.in[0]];
            if (xb < 0)
                return fail(MGI_ERR_UNSUPPORTED, "fc input must come from a sliced tensor");
            const Shape x = g.ops[op.in[0]].out;
            nd.kind = NodeKind::FC;
            nd.kname = "fc_gemm";
            nd.in = {xb};
            nd.ksl = slices(x.c);
            nd.ksp = (nd.ksl + 3) / 4 * 4;
            nd.nb16 = (op.cout + 15) / 16;
            nd.conv.cout = op.cout;
            nd.tile = pick_tile(out_shape.pixels(), op.cout);
            nd.out = new_buf(Layout::F32, out_shape, G.last);
            flat_buf[G.last] = nd.out;
            return MGI_OK;
        }
        case OpKind::Softmax: {
            int t = op.in[0];
            int xb = flat_buf[t];
            if (xb < 0) {
                int cb = need_c8(t);
                if (cb < 0) cb = c8_buf[t];
                if (cb < 0) return fail(MGI_ERR_UNSUPPORTED, "softmax input unavailable");
                Node ex;
                ex.kind = NodeKind::Export;
                ex.kname = "export";
                ex.out_tensor = -1;
                ex.n_fused = 0;
                ex.in = {cb};
                ex.out = new_buf(Layout::F32, g.ops[t].out, -1);
                xb = ex.out;
                add_node(std::move(ex));
            }
            nd.kind = NodeKind::Softmax;
            nd.kname = "softmax";
            nd.in = {xb};
            nd.out = new_buf(Layout::F32, out_shape, G.last);
            flat_buf[G.last] = nd.out;
            return MGI_OK;
        }
        case OpKind::Concat: {
            nd.kind = NodeKind::Concat;
            nd.kname = "concat";
            for (int t : op.in) {
                int b = need_c8(t);
                if (b < 0) b = c8_buf[t];
                if (b < 0) return fail(MGI_ERR_UNSUPPORTED, "concat operand is not sliced");
                nd.in.push_back(b);
            }
            nd.out = new_buf(Layout::C8, out_shape, G.last);
            c8_buf[G.last] = nd.out;
            return MGI_OK;
        }
        case OpKind::ResizeBilinear: {
            int xb = need_c8(op.in[0]);
            if (xb < 0) xb = c8_buf[op.in[0]];
            if (xb < 0) return fail(MGI_ERR_UNSUPPORTED, "resize input is not sliced");
            nd.in = {xb};
            nd.align_corners = op.align_corners;
            if (G.resize_argmax) {
                nd.kind = NodeKind::ResizeArgmax;
                nd.kname = "resize_argmax";
                nd.out = new_buf(Layout::I32, out_shape, G.last);
                flat_buf[G.last] = nd.out;
            } else {
                nd.kind = NodeKind::Resize;
                nd.kname = "resize_bilinear";
                nd.out = new_buf(Layout::C8, out_shape, G.last);
                c8_buf[G.last] = nd.out;
            }
            return MGI_OK;
        }
        case OpKind::Argmax: {
            int xb = need_c8(op.in[0]);
            if (xb < 0) xb = c8_buf[op.in[0]];
            if (xb < 0) return fail(MGI_ERR_UNSUPPORTED, "argmax input is not sliced");
            nd.kind = NodeKind::Argmax;
            nd.kname = "argmax";
            nd.in = {xb};
            nd.out = new_buf(Layout::I32, out_shape, G.last);
            flat_buf[G.last] = nd.out;
            return MGI_OK;
        }
        case OpKind::Pad: {
            int xb = need_c8(op.in[0]);
            if (xb < 0) xb = c8_buf[op.in[0]];
            if (xb < 0) return fail(MGI_ERR_UNSUPPORTED, "pad input is not sliced");
            nd.kind = NodeKind::Pad;
            nd.kname = "pad";
            nd.in = {xb};
            nd.conv.pad_t = op.pads[0];
            nd.conv.pad_l = op.pads[2];
            nd.out = new_buf(Layout::C8, out_shape, G.last);
            c8_buf[G.last] = nd.out;
            return MGI_OK;
        }
        default:
            break;
    }
    return MGI_OK;
}

mgi_status Lowering::lower(const Group &G) {
    const GOp &op = g.ops[G.head];
    const Shape out_shape = g.ops[G.last].out;
    Node nd;
    nd.op = G.head;
    nd.out_tensor = G.last;
    nd.n_fused = G.n;
    nd.act1 = G.act1;
    nd.act2 = G.act2;
    switch (op.kind) {
        case OpKind::Conv2d: {
            const mgi_status st = lower_conv(G, op, out_shape, nd);
            if (st != MGI_OK) return st;
            break;
        }
        case OpKind::Depthwise: {
            int xb = need_c8(op.in[0]);
            if (xb < 0) return fail(MGI_ERR_UNSUPPORTED, "depthwise input has no sliced form");
            nd.kind = NodeKind::Depthwise;
            nd.kname = "dw_conv";
            nd.conv = op.conv;
            nd.in = {xb};
            nd.out = new_buf(Layout::C8, out_shape, G.last);
            c8_buf[G.last] = nd.out;
            break;
        }
        case OpKind::Add:
        case OpKind::Activation: {
            nd.kind = op.kind == OpKind::Add ? NodeKind::Add : NodeKind::Act;
            nd.kname = op.kind == OpKind::Add ? "add" : "activation";
            for (int t : op.in) {
                int b = need_c8(t);
                if (b < 0) b = c8_buf[t];
                if (b < 0) return fail(MGI_ERR_UNSUPPORTED, "element-wise operand is not sliced");
                nd.in.push_back(b);
            }
            nd.out = new_buf(Layout::C8, out_shape, G.last);
            c8_buf[G.last] = nd.out;
            break;
        }
        case OpKind::GlobalAvgPool: {
            int xb = need_c8(op.in[0]);
            if (xb < 0) xb = c8_buf[op.in[0]];
            if (xb < 0) return fail(MGI_ERR_UNSUPPORTED, "pool input is not sliced");
            nd.kind = NodeKind::Gap;
            nd.kname = "global_avgpool";
            nd.in = {xb};
            nd.out = new_buf(Layout::C8, out_shape, G.last);
            c8_buf[G.last] = nd.out;
            break;
        }
        case OpKind::FC:
        case OpKind::Softmax:
        case OpKind::Concat:
        case OpKind::ResizeBilinear:
        case OpKind::Argmax:
        case OpKind::Pad: {
            const mgi_status st = lower_other(G, op, out_shape, nd);
            if (st != MGI_OK) return st;
            break;
        }
        case OpKind::Input:
            break;
    }
    add_node(std::move(nd));
    // a sliced tensor that is a graph output is exported right away
    const int t = G.last;
    if (out_index[t] >= 0 && c8_buf[t] >= 0 && p.bufs[c8_buf[t]].layout == Layout::C8 &&
        flat_buf[t] < 0) {
        Node ex;
        ex.kind = NodeKind::Export;
        ex.kname = "export";
        ex.out_tensor = -1;
        ex.n_fused = 0;
        ex.in = {c8_buf[t]};
        Buf b;
        b.layout = Layout::F32;
        b.shape = g.ops[t].out;
        b.bytes = b.shape.elems() * 4;
        b.loc = Loc::Output;
        b.index = out_index[t];
        b.graph_tensor = t;
        p.bufs.push_back(b);
        ex.out = (int)p.bufs.size() - 1;
        flat_buf[t] = ex.out;
        add_node(std::move(ex));
    }
    return MGI_OK;
}

mgi_status Lowering::bind_outputs() {
    // outputs
    p.output_bufs.assign(g.outputs.size(), -1);
    p.output_tensor = g.outputs;
    p.output_shapes.clear();
    p.output_dtypes.clear();
    for (size_t k = 0; k < g.outputs.size(); ++k) {
        int t = g.outputs[k];
        int b = flat_buf[t];
        if (b < 0 || p.bufs[b].loc != Loc::Output)
            return fail(MGI_ERR_UNSUPPORTED, "output tensor " + std::to_string(t) +
                                                 " was fused away or cannot be exported");
        p.output_bufs[k] = b;
        Shape s = g.ops[t].out;
        p.output_shapes.push_back(s);
        p.output_dtypes.push_back(p.bufs[b].layout == Layout::I32 ? MGI_DTYPE_INT32 : MGI_DTYPE_FP32);
    }

    return MGI_OK;
}

// First and last node of every buffer (the lifetimes the planner shares
// memory by, Sec. 5).
void compute_lifetimes(mgi_plan &p) {
    for (size_t i = 0; i < p.nodes.size(); ++i) {
        Node &nd = p.nodes[i];
        p.bufs[nd.out].producer = (int)i;
        for (int b : nd.in) p.bufs[b].last_use = (int)i;
        if (nd.residual >= 0) p.bufs[nd.residual].last_use = (int)i;
        if (nd.scratch >= 0) p.bufs[nd.scratch].producer = p.bufs[nd.scratch].last_use = (int)i;
        if (nd.scratch2 >= 0) p.bufs[nd.scratch2].producer = p.bufs[nd.scratch2].last_use = (int)i;
    }

}

// Offsets of the arena buffers (the planner the options name, Sec. 5), then
// the state region behind the arena.
void plan_memory(mgi_plan &p, const mgi_options &o) {
    std::vector<int> arena;
    std::vector<size_t> sizes;
    std::vector<int> first, last;
    for (size_t b = 0; b < p.bufs.size(); ++b) {
        if (p.bufs[b].loc != Loc::Arena || p.bufs[b].dead) continue;
        arena.push_back((int)b);
        sizes.push_back(p.bufs[b].bytes);
        first.push_back(p.bufs[b].producer);
        last.push_back(p.bufs[b].last_use);
    }
    PlanResult naive = plan_naive(sizes);
    PlanResult pr = o.materialize_all                   ? naive
                    : o.planner == MGI_PLANNER_GREEDY ? plan_greedy(sizes, first, last)
                    : o.planner == MGI_PLANNER_MCFP   ? plan_mcfp(sizes, first, last)
                                                      : naive;
    p.mem_naive = 0;
    for (size_t s : sizes) p.mem_naive += s;
    p.mem_planned = 0;
    std::vector<size_t> obj_off(pr.object_size.size());
    size_t off = 0;
    for (size_t k = 0; k < pr.object_size.size(); ++k) {
        p.mem_planned += pr.object_size[k];
        obj_off[k] = off;
        off = align256(off + pr.object_size[k]);
    }
    p.n_objects = (int)pr.object_size.size();
    for (size_t i = 0; i < arena.size(); ++i) p.bufs[arena[i]].offset = obj_off[pr.object_of[i]];
    // state region: arrival counters of fused FC -> softmax nodes, one per
    // tile of 16 rows (the finest row tiling of the FC kernel)
    p.state_off = off;
    size_t state = 0;
    for (Node &nd : p.nodes) {
        if (nd.kind != NodeKind::FcSoftmax) continue;
        nd.cnt_off = p.state_off + state;
        state = align256(state + ((p.bufs[nd.out].shape.pixels() + 15) / 16) * sizeof(int));
    }
    p.state_bytes = state;
    p.workspace_bytes = std::max<size_t>(p.state_off + state, 256);

}

// The packed weight blob, uploaded by mgi_plan_bind.
void pack_weights(const mgi_graph &g, mgi_plan &p, const mgi_options &o) {
    auto to_bits = o.dtype == MGI_DTYPE_BF16 ? f32_to_bf16_bits : f32_to_f16_bits;
    // GEMM weights (A operand of v_mfma_f32_16x16x32_f16): for output block nb
    // (16 channels) and K slice ks (8 inputs), 16 rows x 8 halves, contiguous:
    //   packed[((nb * ksp + ks) * 16 + row) * 8 + j] = W[nb*16 + row][k(ks, j)]
    // so one wave's fragment for (nb, four slices) is 1 KiB of consecutive
    // 16-byte lane loads.  K order for an implicit GEMM: tap-major
    // (ky, kx), then input channel slices; for the stem: k = (ky*kw + kx)*cin + ci.
    std::vector<uint8_t> &blob = p.weights;
    blob.clear();
    auto reserve = [&](size_t bytes) {
        size_t o2 = align256(blob.size());
        blob.resize(o2 + align256(bytes), 0);
        return o2;
    };
    p.zero_off = reserve(256);  // zeroed block read by kernels for out-of-range taps
    for (Node &nd : p.nodes) {
        const GOp &op = g.ops[nd.op >= 0 ? nd.op : 0];
        if (nd.kind == NodeKind::DwPw) {
            // depthwise taps of the absorbed op, laid out as for a depthwise node
            const GOp &dop = g.ops[nd.dw_op];
            const int c = dop.out.c, S = slices(c);
            nd.dw_w_off = reserve((size_t)S * 9 * 8 * 2);
            uint16_t *wp = reinterpret_cast<uint16_t *>(blob.data() + nd.dw_w_off);
            for (int ch = 0; ch < c; ++ch)
                for (int t = 0; t < 9; ++t)
                    wp[((size_t)(ch / 8) * 9 + t) * 8 + ch % 8] = to_bits(dop.w[(size_t)ch * 9 + t]);
            nd.dw_b_off = reserve((size_t)S * 8 * 4);
            float *bp = reinterpret_cast<float *>(blob.data() + nd.dw_b_off);
            for (int ch = 0; ch < c; ++ch) bp[ch] = dop.b[ch];
        }
        if (nd.kind == NodeKind::PwDw || nd.kind == NodeKind::StemDw || nd.kind == NodeKind::Irb) {
            // depthwise taps of the absorbed op laid out as for a depthwise
            // node, [S][9][8], biases fp32; channels past c are zero
            const GOp &dop = g.ops[nd.dw_op];
            const int c = dop.out.c, cp = nd.nb16 * 16;
            nd.dw_w_off = reserve((size_t)(cp / 8) * 9 * 8 * 2);
            uint16_t *wp = reinterpret_cast<uint16_t *>(blob.data() + nd.dw_w_off);
            for (int ch = 0; ch < c; ++ch)
                for (int t = 0; t < 9; ++t)
                    wp[((size_t)(ch / 8) * 9 + t) * 8 + ch % 8] = to_bits(dop.w[(size_t)ch * 9 + t]);
            nd.dw_b_off = reserve((size_t)cp * 4);
            float *bp = reinterpret_cast<float *>(blob.data() + nd.dw_b_off);
            for (int ch = 0; ch < c; ++ch) bp[ch] = dop.b[ch];
        }
        if (nd.kind == NodeKind::Gemm || nd.kind == NodeKind::Stem || nd.kind == NodeKind::FC ||
            nd.kind == NodeKind::DwPw || nd.kind == NodeKind::PwDw || nd.kind == NodeKind::StemDw ||
            nd.kind == NodeKind::GemmPool || nd.kind == NodeKind::FcSoftmax || nd.kind == NodeKind::Irb) {
            const Shape x = g.ops[op.in[0]].out;
            const int cin = x.c;
            const bool fc = nd.kind == NodeKind::FC || nd.kind == NodeKind::FcSoftmax;
            const int cout = fc ? op.cout : op.conv.cout;
            const int kh = fc ? 1 : op.conv.kh;
            const int kw = fc ? 1 : op.conv.kw;
            const int sin = slices(cin);
            nd.w_bytes = (size_t)nd.nb16 * nd.ksp * 16 * 8 * 2;
            nd.w_off = reserve(nd.w_bytes);
            uint16_t *wp = reinterpret_cast<uint16_t *>(blob.data() + nd.w_off);
            for (int co = 0; co < cout; ++co) {
                const int nb = co / 16, row = co % 16;
                for (int ky = 0; ky < kh; ++ky)
                    for (int kx = 0; kx < kw; ++kx)
                        for (int ci = 0; ci < cin; ++ci) {
                            int ks, j;
                            if (nd.kind == NodeKind::Stem || nd.kind == NodeKind::StemDw) {
                                const int k = kern::stem_kpos(ky, kx, ci, kh, kw, cin, op.conv.dil_w);
                                ks = k / 8;
                                j = k % 8;
                            } else {
                                ks = (ky * kw + kx) * sin + ci / 8;
                                j = ci % 8;
                            }
                            float v = op.w[(((size_t)co * kh + ky) * kw + kx) * cin + ci];
                            wp[(((size_t)nb * nd.ksp + ks) * 16 + row) * 8 + j] = to_bits(v);
                        }
            }
            nd.b_bytes = (size_t)nd.nb16 * 16 * 4;
            nd.b_off = reserve(nd.b_bytes);
            float *bp = reinterpret_cast<float *>(blob.data() + nd.b_off);
            for (int co = 0; co < cout; ++co) bp[co] = op.b[co];
            if (nd.kind == NodeKind::Irb) {
                // the projection: a 1x1 GEMM over the depthwise output, same layout
                const GOp &pop = g.ops[nd.pj_op];
                const int pin = g.ops[pop.in[0]].out.c, pco = pop.conv.cout;
                nd.pj_w_off = reserve((size_t)nd.pj_nb16 * nd.pj_ksp * 16 * 8 * 2);
                uint16_t *qp = reinterpret_cast<uint16_t *>(blob.data() + nd.pj_w_off);
                for (int co = 0; co < pco; ++co)
                    for (int ci = 0; ci < pin; ++ci)
                        qp[(((size_t)(co / 16) * nd.pj_ksp + ci / 8) * 16 + co % 16) * 8 + ci % 8] =
                            to_bits(pop.w[(size_t)co * pin + ci]);
                nd.pj_b_off = reserve((size_t)nd.pj_nb16 * 16 * 4);
                float *pb = reinterpret_cast<float *>(blob.data() + nd.pj_b_off);
                for (int co = 0; co < pco; ++co) pb[co] = pop.b[co];
            }
        } else if (nd.kind == NodeKind::Depthwise) {
            // fp16 taps per slice: [S][kh*kw][8], bias fp32 [S*8]; padded channels 0
            const int c = op.out.c, S = slices(c), taps = op.conv.kh * op.conv.kw;
            nd.w_bytes = (size_t)S * taps * 8 * 2;
            nd.w_off = reserve(nd.w_bytes);
            uint16_t *wp = reinterpret_cast<uint16_t *>(blob.data() + nd.w_off);
            for (int ch = 0; ch < c; ++ch)
                for (int t = 0; t < taps; ++t)
                    wp[((size_t)(ch / 8) * taps + t) * 8 + ch % 8] =
                        to_bits(op.w[(size_t)ch * taps + t]);
            nd.b_bytes = (size_t)S * 8 * 4;
            nd.b_off = reserve(nd.b_bytes);
            float *bp = reinterpret_cast<float *>(blob.data() + nd.b_off);
            for (int ch = 0; ch < c; ++ch) bp[ch] = op.b[ch];
        }
    }
    p.weight_bytes = std::max<size_t>(blob.size(), 256);
}

mgi_status build_plan_impl(const mgi_graph &g, const mgi_options &o, mgi_plan &p) {
    if (g.outputs.empty()) return fail(MGI_ERR_STATE, "mgi_graph_finalize: no output marked");
    mgi_status st = check_options(o);
    if (st != MGI_OK) return st;
    const std::vector<Group> groups = group_operators(g, o, live_ops(g));
    p.bufs.clear();
    p.nodes.clear();
    Lowering L(g, p);
    L.add_inputs();
    for (const Group &G : groups)
        if ((st = L.lower(G)) != MGI_OK) return st;
    if ((st = L.bind_outputs()) != MGI_OK) return st;
    // node-level fusion passes, then each node's kernel configurations
    if (o.fuse && o.fuse_pwdw) fuse_pw_into_dw(p, o.fuse_pwdw == 2);
    if (o.fuse && o.fuse_pwdw && o.fuse_irb) fuse_proj_into_pwdw(p, o.fuse_irb == 2);
    if (o.fuse && o.fuse_stemdw) fuse_stem_into_dw(p, o.fuse_stemdw == 2);
    if (o.fuse && o.fuse_pool) fuse_pool_into_pw(p, o.fuse_pool == 2);
    if (o.fuse && o.fuse_softmax) fuse_softmax_into_fc(p);
    if (o.fuse && o.fuse_dwpw) fuse_dw_into_pw(p);
    for (Node &nd : p.nodes) add_configs(p, nd, p.bufs[nd.out].shape.pixels());
    compute_lifetimes(p);
    plan_memory(p, o);
    pack_weights(g, p, o);
    p.opt = o;
    return MGI_OK;
}

}  // namespace

}  // namespace mgi

using namespace mgi;

extern "C" mgi_status mgi_graph_finalize(const mgi_graph *g, const mgi_options *o, mgi_plan **p) {
    MGI_ABI_TRY
    if (!g || !o || !p) return fail(MGI_ERR_INVALID_ARG, "mgi_graph_finalize: null pointer");
    *p = nullptr;
    mgi_plan *plan = new (std::nothrow) mgi_plan();
    if (!plan) return fail(MGI_ERR_OOM_HOST, "mgi_graph_finalize: out of host memory");
    mgi_status s;
    try {
        s = build_plan(*g, *o, *plan);
    } catch (const std::bad_alloc &) {
        s = fail(MGI_ERR_OOM_HOST, "mgi_graph_finalize: out of host memory");
    } catch (...) {
        delete plan;   // (the wrapper below turns the exception into a status)
        throw;
    }
    if (s != MGI_OK) {
        delete plan;
        return s;
    }
    *p = plan;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_graph_finalize")
}

extern "C" mgi_status mgi_plan_workspace_bytes(const mgi_plan *p, size_t *bytes) {
    MGI_ABI_TRY
    if (!p || !bytes) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_workspace_bytes: null pointer");
    *bytes = p->workspace_bytes;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_workspace_bytes")
}

extern "C" mgi_status mgi_plan_weight_bytes(const mgi_plan *p, size_t *bytes) {
    MGI_ABI_TRY
    if (!p || !bytes) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_weight_bytes: null pointer");
    *bytes = p->weight_bytes;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_weight_bytes")
}

extern "C" mgi_status mgi_plan_memory_report(const mgi_plan *p, size_t *naive, size_t *planned,
                                             int *n_objects) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_memory_report: null plan");
    if (naive) *naive = p->mem_naive;
    if (planned) *planned = p->mem_planned;
    if (n_objects) *n_objects = p->n_objects;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_memory_report")
}

extern "C" mgi_status mgi_plan_num_io(const mgi_plan *p, int *n_inputs, int *n_outputs) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_num_io: null plan");
    if (n_inputs) *n_inputs = (int)p->input_bufs.size();
    if (n_outputs) *n_outputs = (int)p->output_bufs.size();
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_num_io")
}

extern "C" mgi_status mgi_plan_io_info(const mgi_plan *p, int is_output, int index, int *n, int *h,
                                       int *w, int *c, int *dtype, size_t *bytes) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_io_info: null plan");
    const auto &shapes = is_output ? p->output_shapes : p->input_shapes;
    const auto &types = is_output ? p->output_dtypes : p->input_dtypes;
    if (index < 0 || index >= (int)shapes.size())
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_io_info: index out of range");
    const Shape s = shapes[index];
    if (n) *n = s.n;
    if (h) *h = s.h;
    if (w) *w = s.w;
    if (c) *c = s.c;
    if (dtype) *dtype = types[index];
    if (bytes) *bytes = s.elems() * (types[index] == MGI_DTYPE_FP16 ? 2 : 4);
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_io_info")
}

extern "C" mgi_status mgi_plan_node_count(const mgi_plan *p, int *count) {
    MGI_ABI_TRY
    if (!p || !count) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_node_count: null pointer");
    *count = (int)p->nodes.size();
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_node_count")
}

extern "C" mgi_status mgi_plan_node_info(const mgi_plan *p, int i, const char **kind,
                                         int *tensor_id, int *n, int *h, int *w, int *c,
                                         int *n_fused) {
    MGI_ABI_TRY
    if (!p) return fail(MGI_ERR_INVALID_ARG, "mgi_plan_node_info: null plan");
    if (i < 0 || i >= (int)p->nodes.size())
        return fail(MGI_ERR_INVALID_ARG, "mgi_plan_node_info: node index out of range");
    const Node &nd = p->nodes[i];
    const Shape s = p->bufs[nd.out].shape;
    if (kind) *kind = nd.kname;
    if (tensor_id) *tensor_id = nd.out_tensor;
    if (n) *n = s.n;
    if (h) *h = s.h;
    if (w) *w = s.w;
    if (c) *c = s.c;
    if (n_fused) *n_fused = nd.n_fused;
    return MGI_OK;
    MGI_ABI_CATCH("mgi_plan_node_info")
}
